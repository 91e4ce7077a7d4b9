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


@pytest.mark.parametrize("config", [2, 4])
def test_traffic_is_used_only_for_the_sources_it_was_taken_on(config, monkeypatch):
    with open(os.path.join(ROOT, "profiles", f"traffic_c{config}_f32.json")) as f:
        d = json.load(f)
    per_step = d["kernels"]["k_run"]["hbm_bytes_per_step"]
    monkeypatch.setattr(bench, "step_source_sha", lambda: d["source_sha"])
    assert bench.measured_traffic(config, "f32", "k_run", 1000) == per_step * 1000
    assert bench.measured_traffic(config, "f32", "k_tile", 1000) is None
    monkeypatch.setattr(bench, "step_source_sha", lambda: "0" * 16)
    assert bench.measured_traffic(config, "f32", "k_run", 1000) is None


def test_step_source_hash_covers_every_step_kernel_source():
    csrc = os.path.join(ROOT, "paper_2102_04681_amd", "csrc")
    kernels = {f for f in os.listdir(csrc) if f.endswith(".hip") and f != "spk_gen.hip"}
    assert kernels <= set(bench.STEP_SOURCES)
    assert len(bench.step_source_sha()) == 16


def test_algorithmic_bytes_of_the_3e9_synapse_workload():
    with open(os.path.join(ROOT, "profiles", "traffic_c4_f32.json")) as f:
        k = json.load(f)["kernels"]["k_run"]
    steps, events = 500, k["events_per_step"] * 500
    spikes = 2_000_000 * k["mean_rate_hz"] * 1e-4 * steps  # dt = 0.1 ms
    ev_bytes, other = bench.algorithmic_bytes(2_000_000, 0, events, spikes, 4.0, steps)
    assert ev_bytes == 4.0 * events
    assert other == pytest.approx(10.0 * 2_000_000 * steps + 8.0 * spikes)
    assert (ev_bytes + other) / steps == pytest.approx(32.3e6, rel=2e-3)
