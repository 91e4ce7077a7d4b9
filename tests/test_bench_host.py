"""Host-side checks of bench.py's contract (no GPU needed).

  - a request for more than one GPU ends with a message and exit status 2,
    before anything touches a device;
  - the roofline's `traffic` comes from the committed counter summary only
    while the step kernels' sources are the ones the counters were taken on;
  - the algorithmic bytes per step of the 3e9-synapse workload (4 B per
    event, 10 B per LIF neuron, 8 B per spike) add up to the figure the
    profiles quote for it.
"""
import json
import os
import subprocess
import sys

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one MI355X" in r.stderr and r.stdout == ""


@pytest.mark.parametrize("config,rate", [(2, 10.0), (4, 10.0), (1, 10.0), (3, 10.0), (3, 50.0)])
def test_traffic_is_used_only_for_the_sources_it_was_taken_on(config, rate, monkeypatch):
    tag = bench.workload_tag(config, rate)
    with open(os.path.join(ROOT, "profiles", f"traffic_{tag}_f32.json")) as f:
        d = json.load(f)
    per_step = d["kernels"]["k_run"]["hbm_bytes_per_step"]
    monkeypatch.setattr(bench, "step_source_sha", lambda: d["source_sha"])
    assert bench.measured_traffic(tag, "f32", "k_run", 1000) == per_step * 1000
    assert bench.measured_traffic(tag, "f32", "k_tile", 1000) is None
    monkeypatch.setattr(bench, "step_source_sha", lambda: "0" * 16)
    assert bench.measured_traffic(tag, "f32", "k_run", 1000) is None


def test_step_source_hash_covers_every_step_kernel_source():
    csrc = os.path.join(ROOT, "paper_2102_04681_amd", "csrc")
    kernels = {f for f in os.listdir(csrc) if f.endswith(".hip") and f != "spk_gen.hip"}
    assert kernels <= set(bench.STEP_SOURCES)
    assert len(bench.step_source_sha()) == 16


def test_algorithmic_bytes_of_the_3e9_synapse_workload():
    # per step at 10 Hz: 2,000 spikes x 1,500 events; 8 B per event (a 32-bit
    # target and a 32-bit weight read once), 10 B per LIF neuron (V and the
    # refractory counter read and written), 8 B per spike
    steps, rate = 500, 10.0
    spikes = 2_000_000 * rate * 1e-4 * steps  # dt = 0.1 ms
    events = spikes * 1500
    b = bench.algorithmic_bytes(2_000_000, 0, events, spikes, steps)
    other = 10.0 * 2_000_000 * steps + 8.0 * spikes
    assert b[8] == pytest.approx(8.0 * events + other)
    assert b[4] == pytest.approx(4.0 * events + other)
    assert b[8] / steps == pytest.approx(44.0e6, rel=1e-3)  # 24 MB of events + 20 MB of neurons
    ev, neu = bench.algorithmic_bytes(1_000_000, 1, 10.0, 2.0, 3, split=True)
    assert ev == {8: 80.0, 4: 40.0, 0: 0.0} and neu == 8.0 * 1_000_000 * 3 + 16.0


def test_settle_steps_cover_transient_and_delays():
    import inputs as I
    assert bench.settle_steps(I.config(4, driven=True)) == 300
    assert bench.settle_steps(I.config(3)) == 30
    assert bench.settle_steps(I.config(0, delay_max=200)) == 400
