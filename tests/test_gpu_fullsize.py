"""GPU parity at the full benchmark sizes, in the configurations bench.py times.

Workload: 2,000,000 LIF neurons, fixed out-degree 1,500 (3.0e9 synapses),
delays 1..20 steps, external Poisson drive at twice the threshold rate,
fp32 accumulation, binned delivery, steps run by the persistent kernel (as
bench.py times them) and replayed from HIP graphs.  The oracle cannot
simulate this network step by step in test time, so it checks sampled
outputs it can compute one by one:

  - sampled rows, generated lazily by the oracle, equal the library's rows;
  - after 300 steps, the input of sampled neurons at the next step is the
    sum of the synapses of every spike of the previous 20 steps (oracle
    rows) whose delay makes them arrive then; the library sums exactly and
    rounds once, so the same exact sum fed to the oracle's single-neuron
    update must reproduce the library's membrane potential, refractory
    counter and spike decision bit for bit;
  - events delivered at that step = synapses of those spikes with the
    arriving delay; events emitted = 1,500 per spike.
"""
import sys

import numpy as np
import pytest

import inputs as I
import oracle

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def spk_full():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2102_04681_amd import spk as mod
    mod.lib()
    return mod


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("step_mode", [2, 1], ids=["persist", "graph"])
def test_full_size_bench_configuration_sampled(spk_full, step_mode):
    spk = spk_full
    cfg = I.config(4, driven=True, step_mode=step_mode)
    n, K, dmax = cfg["n"], cfg["k_out"], cfg["delay_max"]
    T0 = 300
    _say(f"[full] create n={n} k_out={K}")
    g = spk.Net(cfg, max_steps=T0 + 1, raster_capacity=4_000_000)
    st = g.stats()
    assert st["step_mode"] == step_mode
    assert st["nnz"] == n * K
    assert st["delivery"] == spk.SPK_DELIVERY_BINNED
    s64 = int(st["fixed_shift"])
    o = oracle.Net(cfg, build_csr=False)
    rng = np.random.default_rng(7)

    # 1. sampled rows
    rows = rng.choice(n, 48, replace=False).astype(np.uint32)
    offs, col, w, d = g.export_rows(rows)
    for k, s in enumerate(rows):
        ot, ow, od = o.row(int(s), cap=K)
        a, b = int(offs[k]), int(offs[k + 1])
        gi = np.lexsort((w[a:b].view(np.uint32), d[a:b], col[a:b]))
        oi = np.lexsort((ow.view(np.uint32), od, ot))
        assert np.array_equal(col[a:b][gi], ot[oi]), f"row {s}: targets"
        assert np.array_equal(d[a:b][gi], od[oi]), f"row {s}: delays"
        assert np.array_equal(w[a:b][gi].view(np.uint32), ow[oi].view(np.uint32)), f"row {s}: weights"
    _say("[full] rows ok")

    # 2. run as the benchmark does, then one more step
    g.step(T0)
    V0, R0 = g.state()
    g.step(1)
    V1, R1 = g.state()
    offs_r, ids = g.raster()
    t = T0
    spiked_t = set(ids[int(offs_r[t]):int(offs_r[t + 1])].tolist())
    assert 0 < len(spiked_t) < n // 10, "the driven network should fire sparsely"

    # 3. exact input of sampled neurons at step t from the oracle's rows
    targets = np.unique(rng.choice(n, 256, replace=False)).astype(np.uint32)
    pos = {int(x): k for k, x in enumerate(targets)}
    tmask = np.zeros(n, dtype=bool)
    tmask[targets] = True
    acc = np.zeros(len(targets), dtype=np.int64)       # units of 2^-s64
    delivered = 0
    for dd in range(1, dmax + 1):
        ts = t - dd
        src = ids[int(offs_r[ts]):int(offs_r[ts + 1])]
        for s in src:
            ot, ow, od = o.row(int(s), cap=K)
            m = od == dd
            delivered += int(m.sum())
            hit = tmask[ot] & m
            for tg, wv in zip(ot[hit], ow[hit]):
                acc[pos[int(tg)]] += int(np.rint(np.ldexp(np.float64(wv), s64)))
    _say(f"[full] inputs of {len(targets)} neurons from {int(offs_r[t] - offs_r[t - dmax])} spikes")
    assert int(g.delivered(t, 1)[0]) == delivered
    assert int(g.events(t - 1, 1)[0]) == K * int(offs_r[t] - offs_r[t - 1])

    # 4. the oracle's update with that input reproduces the library bit for bit
    for k, i in enumerate(targets):
        isyn = np.float32(np.ldexp(np.float64(acc[k]), -s64))
        v, r, sp = o.update_one(t, int(i), float(V0[i]), int(R0[i]), isyn_f=float(isyn))
        assert np.float32(v).view(np.uint32) == V1[i].view(np.uint32), f"neuron {i}: V {v} vs {V1[i]}"
        assert r == int(R1[i]), f"neuron {i}: refractory counter"
        assert sp == (int(i) in spiked_t), f"neuron {i}: spike decision"
    _say("[full] sampled update ok")


def test_full_size_delay15_batch_sampled(spk_full):
    """The 1e9-synapse network with delay 15 (100,000 LIF, in-degree 8,000
    excitatory + 2,000 inhibitory, Poisson drive, fp32 accumulation) in the
    configuration bench.py --config 2 times: the persistent kernel in batches
    of 8 steps.  After 300 steps, one more batch; for sampled
    neurons the oracle draws the in-synapses (its per-target generator), sums
    the weights of those whose source fired 15 steps earlier exactly, and
    runs its single-neuron update for each step: every spike decision of the batch
    and the final state must equal the library's bit for bit."""
    spk = spk_full
    cfg = I.config(2, driven=True)
    n, D, d = cfg["n"], 8, cfg["delay_min"]
    T0 = 300
    _say(f"[full c2] create n={n}")
    g = spk.Net(cfg, max_steps=T0 + D, raster_capacity=2_000_000)
    st = g.stats()
    assert st["step_mode"] == spk.SPK_STEP_PERSISTENT
    assert st["delivery"] == spk.SPK_DELIVERY_BINNED and st["batch_steps"] == D
    assert st["nnz"] == n * (cfg["k_in_exc"] + cfg["k_in_inh"])
    s64 = int(st["fixed_shift"])
    g.step(T0)
    V0, R0 = g.state()
    g.step(D)
    V1, R1 = g.state()
    offs, ids = g.raster()
    spikes = [set(ids[int(offs[t]):int(offs[t + 1])].tolist()) for t in range(T0 + D)]
    fired = np.zeros((D, n), dtype=bool)  # fired[k, s]: s spiked at step T0 + k - 15
    for k in range(D):
        fired[k, ids[int(offs[T0 + k - d]):int(offs[T0 + k - d + 1])]] = True
    assert 0 < sum(len(spikes[t]) for t in range(T0, T0 + D)) < n
    # every synapse has delay 15: events arriving at t are those emitted at t - 15
    dl, ev = g.delivered(T0, D), g.events(T0 - d, D)
    assert np.array_equal(dl, ev)

    o = oracle.Net(cfg, build_csr=False)
    rng = np.random.default_rng(11)
    targets = rng.choice(n, 256, replace=False).astype(np.uint32)
    for i in targets:
        src, w, dd = o.in_row(int(i))
        assert (dd == d).all()
        units = np.rint(np.ldexp(w.astype(np.float64), s64)).astype(np.int64)
        v, r = float(V0[i]), int(R0[i])
        for t in range(T0, T0 + D):
            acc = int(units[fired[t - T0, src]].sum())
            isyn = np.float32(np.ldexp(np.float64(acc), -s64))
            v, r, sp = o.update_one(t, int(i), v, r, isyn_f=float(isyn))
            assert sp == (int(i) in spikes[t]), f"neuron {i}: spike decision at step {t}"
        assert np.float32(v).view(np.uint32) == V1[i].view(np.uint32), f"neuron {i}: V {v} vs {V1[i]}"
        assert r == int(R1[i]), f"neuron {i}: refractory counter"
    _say("[full c2] sampled batch ok")
