#!/usr/bin/env python3
"""Synaptic-event throughput of libspk on one MI355X.

A step is one simulation timestep of the whole hot path: delivery of every
event arriving at the step into LDS, the update of every neuron with spike
compaction, and the filing of the new spikes' events by arrival step.  The
default workload is the 3-billion-synapse one-GPU network (2 000 000 LIF
neurons, fan-out 1 500, delays 1..20 steps) with the external Poisson drive
that keeps it active (without drive every neuron decays to rest and no
synaptic event happens).

    python bench.py [--steps K] [--warmup W] [--config 4] [--acc f32|fixed]
                    [--mode auto|graph|persistent] [--format auto|full|compact]

Prints one JSON line (the last line of stdout).  Timing: a fixed number of
settling steps (past the start-up transient and every pending delay, run
whatever --warmup says), W untimed warm-up steps, then exactly K steps (one
persistent-kernel launch, or graph replays) between HIP events on the
network's stream, bracketed by torch.cuda.synchronize().  `value` counts the
events of the spikes emitted inside the timed window (the rows read there);
the events delivered in the window are reported beside it.  For the
persistent kernel the same launch is also timed by the library's own HIP
events around it, which gives the dominant kernel's duration for the
roofline figure over the same window; the graph path times a second pass
with each step's kernels launched on their own.  The CPU oracle is timed on
a bounded sample (reduced neuron count, same per-neuron statistics).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.join(ROOT, "tests"))

PEAK_HBM_GBS = 8000.0  # MI355X HBM3E, published
METRIC = "synaptic events delivered/sec on 1 MI355X; % of HBM roofline"
WORKLOAD_NAMES = {
    0: "C0: 1,000 LIF, Bernoulli p=0.02, delay 1",
    1: "C1: 250,000 LIF, Bernoulli p=0.02 (1.25e9 synapses), delay 1",
    2: "C2: 100,000 LIF, in-degree 8,000 exc + 2,000 inh (1e9 synapses), delay 15, Poisson drive",
    3: "C3: 1,000,000 Bernoulli sources, fan-out 1,000 (1e9 synapses), dt 1 ms",
    4: "C4: 2,000,000 LIF, fan-out 1,500 (3e9 synapses), delays 1-20 steps",
}


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=4500)
    ap.add_argument("--warmup", type=int, default=500)
    ap.add_argument("--config", type=int, default=4, choices=range(5))
    ap.add_argument("--rate", type=float, default=10.0, help="source rate (Hz) for config 3")
    ap.add_argument("--acc", choices=["f32", "fixed"], default="f32")
    ap.add_argument("--delivery", choices=["auto", "direct", "binned"], default="auto")
    ap.add_argument("--mode", choices=["auto", "graph", "persistent"], default="auto",
                    help="how steps are launched (spk_params.step_mode)")
    ap.add_argument("--format", choices=["auto", "full", "compact", "procedural"], default="auto",
                    help="synapse storage (spk_params.syn_format)")
    ap.add_argument("--seed", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target duration of the timed oracle sample")
    ap.add_argument("--setup", action="store_true",
                    help="setup-time study instead of the step benchmark: create Synth networks "
                         "(density 5%%) of growing size and C2/C4, print one JSON line")
    ap.add_argument("--probe-copy", type=int, default=0, metavar="BYTES",
                    help="only run the library's copy kernel on BYTES (counter calibration)")
    return ap.parse_args()


def workload(args):
    import inputs as I
    acc = I.ACC_FIXED if args.acc == "fixed" else I.ACC_F32
    cfg = I.config(args.config, driven=True, seed=args.seed, rate_hz=args.rate, acc_mode=acc)
    cfg["delivery"] = {"auto": 0, "direct": 1, "binned": 2}[args.delivery]
    cfg["step_mode"] = {"auto": 0, "graph": 1, "persistent": 2}[args.mode]
    cfg["syn_format"] = {"auto": 0, "full": 1, "compact": 2, "procedural": 3}[args.format]
    return cfg


def algorithmic_bytes(n, kind, events, spikes, steps, split=False):
    """Bytes the hot path must move per the method, over `steps` steps with
    `events` synaptic events (rows read) and `spikes` spikes in total: per
    event one synapse record read once (8 B for a 32-bit target + 32-bit
    weight; also given at 4 B, the record stored where the network has
    per-population weights and only target and delay are kept, as the paper's
    adjacency list does; 0 B where synapses are generated, not stored), 10 B
    per LIF neuron and step (V read + write,
    refractory counter read + write; 8 B for a source neuron, which has no
    counter), 8 B per spike (ID written once, read once).  Accumulators are
    on chip and cost nothing.  Returns {bytes per event: total bytes}, or
    with split=True ({bytes per event: event bytes}, neuron and spike bytes)."""
    per_neuron = 8 if kind == 1 else 10
    neu = per_neuron * float(n) * steps + 8.0 * spikes
    ev = {8: 8.0 * events, 4: 4.0 * events, 0: 0.0}  # (0: procedural synapses, none read)
    if split:
        return ev, neu
    return {b: v + neu for b, v in ev.items()}


SETTLE_MS = 30.0


def settle_steps(cfg):
    """Steps every run makes untimed before its warm-up, whatever --warmup
    says: 30 ms of biological time and at least twice the longest delay.
    Every neuron starts at a random V below threshold and the drive fires a
    burst in the first milliseconds whose events arrive over the next delays;
    after that the network is in its steady state, so that the timed window
    measures steady-state throughput."""
    return max(2 * int(cfg["delay_max"]), int(round(SETTLE_MS / cfg["dt_ms"])))


STEP_SOURCES = ("spk_internal.h", "spk_dev.h", "spk_step.hip", "spk_run.hip", "spk_run_batch.hip", "spk_proc.hip",
                "spk_runtime.hip")


def step_source_sha():
    """Hash of the sources of the step kernels (counter summaries are valid
    only for the code they were taken on)."""
    h = hashlib.sha256()
    for name in STEP_SOURCES:
        with open(os.path.join(ROOT, "paper_2102_04681_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def workload_tag(config, rate):
    """Short name of a workload in profiles/ (the source network carries its rate)."""
    return f"c{config}" + (f"r{rate:g}" if config == 3 else "")


def measured_traffic(tag, acc, kernel, steps_per_launch):
    """HBM bytes per launch from the committed counter summary (calibrated
    FETCH_SIZE + WRITE_SIZE per step of the kernel, times the steps of one
    launch), or None when the summary is missing or the step kernels changed
    since it was taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{tag}_{acc}.json")
    try:
        with open(path) as f:
            d = json.load(f)
    except OSError:
        return None
    if d.get("source_sha") != step_source_sha():
        return None
    k = d.get("kernels", {}).get(kernel)
    if not k:
        return None
    return k["hbm_bytes_per_step"] * steps_per_launch


def cpu_baseline(cfg, seconds):
    """The oracle (single-threaded C, unchanged) on a bounded sample of the
    workload: the same per-neuron statistics at a neuron count whose network
    the oracle builds in seconds; only its step loop is timed."""
    import oracle
    import inputs as I
    n_full = cfg["n"]
    n = min(n_full, 20000)
    sample = dict(cfg)
    sample["n"] = n
    if cfg["conn_kind"] == I.BERNOULLI and cfg["p"] * n_full > 0:
        sample["p"] = min(1.0, cfg["p"] * n_full / n)  # keep the expected in-degree
    if cfg["conn_kind"] == I.FIXED_IN:
        ne = round(cfg["frac_exc"] * n)
        sample["k_in_exc"] = min(cfg["k_in_exc"], ne)
        sample["k_in_inh"] = min(cfg["k_in_inh"], n - ne)
    net = oracle.Net(sample)
    net.run(200)  # initial transient
    events, steps, t0 = 0, 0, time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        r = net.run(100)
        events += int(r["events"].sum())
        steps += 100
    dt = time.perf_counter() - t0
    desc = (f"oracle step loop (single thread), {steps} steps of the same workload at n={n} "
            f"(fan-in, fan-out, weights, delays and drive unchanged), network build and the "
            f"first 200 steps excluded")
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), model)
    except OSError:
        pass
    return {"value": events / dt, "unit": "events/s", "cores": 1, "kind": "oracle",
            "sample": desc, "steps": steps, "seconds": round(dt, 2),
            "wall_per_bio_time": round(dt / (steps * cfg["dt_ms"] * 1e-3), 2),
            "cpu_model": model, "host_cpus": os.cpu_count()}


SETUP_SYNTH_N = (10_000, 20_000, 50_000, 100_000, 200_000, 300_000)


def setup_study(stream, seed):
    """Setup time as a function of network size (Sec. IV-C): Synth networks of
    density 5 % and the C2 and C4 networks, created on the GPU.  Reports the
    wall time of the creating call and the GPU time of the generation
    kernels (rows counted, drawn, grouped) and of the accumulator-range pass."""
    import torch
    import inputs as I
    from paper_2102_04681_amd import spk
    cases = [(f"synth n={n:,}", I.synth(n, 0.05, seed=seed)) for n in SETUP_SYNTH_N]
    cases += [("C2", I.config(2, driven=True, seed=seed)), ("C4", I.config(4, driven=True, seed=seed))]
    points = []
    for name, cfg in cases:
        net = spk.Net(cfg, stream=stream, max_steps=1)
        st = net.stats()
        nnz = int(st["nnz"])
        points.append({"network": name, "n": cfg["n"], "synapses": nnz,
                       "setup_ms": round(st["setup_ms"], 2), "gen_ms": round(st["gen_ms"], 3),
                       "range_ms": round(st["range_ms"], 3),
                       "gen_synapses_per_ms": round(nnz / st["gen_ms"]) if st["gen_ms"] > 0 else None,
                       "setup_synapses_per_ms": round(nnz / st["setup_ms"]) if st["setup_ms"] > 0 else None})
        print(f"[setup] {name}: {nnz:,} synapses, create {st['setup_ms']:.1f} ms, generation kernels "
              f"{st['gen_ms']:.2f} ms, range pass {st['range_ms']:.2f} ms", file=sys.stderr, flush=True)
        del net
        torch.cuda.synchronize()
    synth = [p_ for p_ in points if p_["network"].startswith("synth")]
    best = max(synth, key=lambda p_: p_["synapses"])
    return {"metric": "setup: synapses generated per ms (GPU generation kernels), Synth density 5%",
            "value": best["gen_synapses_per_ms"], "unit": "synapses/ms", "n_gpus": 1,
            "higher_is_better": True, "data": "synthetic", "seed": seed,
            "config": {"workload": f"Synth density 5%, n={best['n']:,}"}, "points": points}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one MI355X: the simulated network is one GPU's share and "
              "there is no multi-GPU path (run with --gpus 1).", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2102_04681_amd import spk

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    stream = torch.cuda.Stream()
    torch.cuda.set_stream(stream)

    if args.setup:
        print(json.dumps(setup_study(stream, args.seed)))
        return

    if args.probe_copy:
        cfg = workload(args)
        cfg["n"] = 1000
        g = spk.Net(dict(cfg, conn_kind=0, p=0.0), stream=stream, max_steps=1)
        ms = g.hbm_copy(args.probe_copy, reps=20)
        print(json.dumps({"probe": "copy", "bytes": args.probe_copy, "reps": 20,
                          "GB/s": 2 * args.probe_copy * 20 / (ms * 1e-3) / 1e9}))
        return

    cfg = workload(args)
    W, K = args.warmup, args.steps
    S = settle_steps(cfg)
    t_create = time.perf_counter()
    net = spk.Net(cfg, stream=stream, max_steps=S + W + 2 * K)
    torch.cuda.synchronize()
    t_create = time.perf_counter() - t_create
    st = net.stats()
    persistent = st["step_mode"] == spk.SPK_STEP_PERSISTENT
    bpe = float(st["bytes_per_synapse"])
    print(f"[bench] {WORKLOAD_NAMES[args.config]}: nnz={st['nnz']} tiles={st['tiles']}x{st['tile_width']} "
          f"delivery={'direct' if st['delivery'] == 1 else 'binned'} "
          f"steps={'persistent' if persistent else 'graph'} batch={st['batch_steps']} bytes/synapse={bpe:g} "
          f"create={t_create:.2f}s settle={S} warmup={W} timed={K}", file=sys.stderr, flush=True)

    net.step(S)  # past the start-up transient and every pending delay
    net.step(W)
    torch.cuda.synchronize()
    # The persistent kernel runs all K steps in one launch: HIP events around
    # that launch (on the network's stream) time the dominant kernel over the
    # same window the wall clock times.
    if persistent:
        net.set_profiling(True)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    net.step(K)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    t0 = S + W
    emitted = float(net.events(t0, K).astype(float).sum())
    delivered = float(net.delivered(t0, K).astype(float).sum())
    spikes = float(net.spike_counts(t0, K).astype(float).sum())
    # events whose rows were read inside the timed window
    value = emitted / (ms * 1e-3)
    ms_step = ms / K

    if persistent:
        km = net.kernel_ms()
        net.set_profiling(False)
        assert km["run_launches"] == 1 and km["steps"] == K
        kernels = {"k_run": (km["run_ms"], algorithmic_bytes(cfg["n"], cfg["neuron_kind"], emitted, spikes, K))}
        win_ev, win_sp = emitted, spikes
        spl = K
    else:  # graph path: a second pass with each step's kernels launched and timed on their own
        net.set_profiling(True)
        net.step(K)
        km = net.kernel_ms()
        net.set_profiling(False)
        nsteps = km["steps"]
        win_ev = float(net.events(t0 + K, K).astype(float).sum())
        win_sp = float(net.spike_counts(t0 + K, K).astype(float).sum())
        ev_b, neu_b = algorithmic_bytes(cfg["n"], cfg["neuron_kind"], win_ev, win_sp, nsteps, split=True)
        if st["delivery"] == 2:  # push kernel reads the fired rows; tile kernel updates the neurons
            kernels = {"k_push": (km["push_ms"] / nsteps, {b: v / nsteps for b, v in ev_b.items()}),
                       "k_tile": (km["tile_ms"] / nsteps, {b: neu_b / nsteps for b in ev_b})}
        else:     # tile kernel does both
            kernels = {"k_tile": (km["tile_ms"] / nsteps, {b: (v + neu_b) / nsteps for b, v in ev_b.items()})}
        spl = 1
    # measured bandwidths of this device: a streaming read (what a synapse
    # stream can reach) and the library's copy kernel (1 GiB each)
    read_gbs = (1 << 30) * 10 / (net.hbm_read(1 << 30, reps=10) * 1e-3) / 1e9
    copy_gbs = 2 * (1 << 30) * 10 / (net.hbm_copy(1 << 30, reps=10) * 1e-3) / 1e9
    dom = max(kernels, key=lambda k: kernels[k][0])
    dom_ms, dom_bytes = kernels[dom]
    achieved = dom_bytes[8] / (dom_ms * 1e-3) / 1e9
    achieved_rec = dom_bytes[bpe] / (dom_ms * 1e-3) / 1e9
    traffic = measured_traffic(workload_tag(args.config, args.rate), args.acc, dom, spl)
    roofline = {
        "bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
        "frac": round(achieved / PEAK_HBM_GBS, 4),
        "traffic": None if traffic is None else round(traffic),
        "kernel": dom, "kernel_us": round(dom_ms * 1e3, 2), "steps_per_launch": spl,
        "bytes_per_event": 8.0,
        "kernel_alg_bytes": round(dom_bytes[8]),
        "stored_record_bytes_per_event": bpe,
        "achieved_stored_record": round(achieved_rec, 1),
        "frac_stored_record": round(achieved_rec / PEAK_HBM_GBS, 4),
        "events_only_frac": round(value * 8.0 / (PEAK_HBM_GBS * 1e9), 4),
        "per_launch_us": {k: round(v[0] * 1e3, 2) for k, v in kernels.items()},
        "probe_read_GBs": round(read_gbs, 1), "frac_vs_read_probe": round(achieved / read_gbs, 4),
        "probe_copy_GBs": round(copy_gbs, 1),
    }

    rate_hz = spikes / (cfg["n"] * K * cfg["dt_ms"] * 1e-3)
    name = WORKLOAD_NAMES[args.config]
    if args.config == 3:
        name += f", {args.rate:g} Hz"
    out = {
        "metric": METRIC, "value": value, "unit": "events/s", "n_gpus": 1, "steps": K,
        "warmup": W, "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32" if args.acc == "f32" else "i32",
        "data": "synthetic",
        "config": {
            "workload": name + (", Poisson drive at twice threshold rate"
                                if cfg["ext_lambda"] and args.config != 2 else ""),
            "n_neurons": cfg["n"], "synapses": int(st["nnz"]), "dt_ms": cfg["dt_ms"],
            "delivery": "direct" if st["delivery"] == 1 else "binned",
            "steps": "one persistent launch" if persistent else "HIP graphs of 32 steps",
            "batch_steps": st["batch_steps"],
            "synapse_bytes": bpe,
            "accumulation": "exact int64 fixed point, rounded once to fp32" if args.acc == "f32"
                            else f"int32 fixed point 2^-{cfg['fixed_shift']}",
            "settle_steps": S,
            "mean_rate_hz": round(rate_hz, 3),
            "events_emitted_per_step": round(emitted / K, 1),
            "events_delivered_per_step": round(delivered / K, 1),
            "seed": args.seed, "parallelism": "1 GPU",
        },
        "roofline": roofline,
        "wall_per_bio_time": round(ms_step / cfg["dt_ms"], 4),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, args.cpu_seconds)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
