"""Seeded synthetic inputs shared by the oracle side and the GPU side of the tests.

This module holds workload definitions (parameter dictionaries) and seeded
random inputs (spike sets, explicit adjacency lists).  It contains none of
the method's arithmetic: no connectivity generation, no neuron update, no
delivery.  Both ``oracle.Net`` and ``paper_2102_04681_amd.Net`` accept the
same parameter dictionaries.

Workloads stand in for the paper's benchmark models (Sec. IV: Vogels-Abbott,
Brunel, and the synthetic 'Synth' model of Sec. IV-B), whose exact
definitions the paper defers to other publications.  The five shapes below
are the ones this project measures:

  C0  1 000 LIF, 80/20 exc/inh, Bernoulli p=0.02, w +0.27 / -4.5 mV, delay 1
  C1  250 000 LIF, p=0.02, weights x 80/(0.02 N)
  C2  100 000 LIF, fixed in-degree 8 000 exc + 2 000 inh, J=0.1, g=5,
      delay 15 steps, Poisson drive at twice the threshold rate
  C3  1 000 000 Bernoulli sources (1/10/50 Hz), dt = 1 ms, fan-out 1 000,
      w ~ U[0, 1e-3)
  C4  2 000 000 LIF, fan-out 1 500, weights x 80/1500, delays 1..20 steps

Membrane parameters (all LIF workloads): tau_m 20 ms, V_rest = V_reset = -60,
V_th = -50 mV, 5 ms refractory, dt 0.1 ms, V0 ~ U[-60, -50).  With no
external drive these networks are silent (every V0 is below threshold and
decays towards V_rest), so each LIF workload also has a "driven" variant that
adds Brunel's external Poisson drive at twice the threshold rate:
lambda = 2 * theta * (dt/tau_m) / J events per step of weight J = w_exc,
theta = V_th - V_rest = 10 mV.
"""
from __future__ import annotations

import os

import numpy as np

LIF, SOURCE = 0, 1
BERNOULLI, FIXED_OUT, FIXED_IN, EXPLICIT = 0, 1, 2, 3
ACC_F32, ACC_FIXED = 0, 1

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

_MEMBRANE = dict(
    neuron_kind=LIF, frac_exc=0.8, dt_ms=0.1, tau_m_ms=20.0, t_ref_ms=5.0,
    v_rest=-60.0, v_th=-50.0, v_reset=-60.0, v0_lo=-60.0, v0_hi=-50.0, i_bias=0.0,
    p=0.0, k_out=0, k_in_exc=0, k_in_inh=0, w_uniform=0, w_lo=0.0, w_hi=0.0,
    delay_min=1, delay_max=1, ext_lambda=0.0, ext_w=0.0, src_rate_hz=0.0,
    acc_mode=ACC_F32, fixed_shift=20,
)


def _f32(x: float) -> float:
    return float(np.float32(x))


def drive_lambda(cfg: dict) -> float:
    """Brunel's external rate at twice threshold, per step, for weight w_exc."""
    theta = float(cfg["v_th"]) - float(cfg["v_rest"])
    return 2.0 * theta * (cfg["dt_ms"] / cfg["tau_m_ms"]) / _f32(cfg["w_exc"])


def config(index: int, driven: bool = False, seed: int = 1, rate_hz: float = 10.0,
           acc_mode: int = ACC_F32, **over) -> dict:
    """Workload C<index> as a parameter dictionary (see module docstring)."""
    c = dict(_MEMBRANE, seed=seed, acc_mode=acc_mode)
    if index == 0:
        c.update(n=1000, conn_kind=BERNOULLI, p=0.02, w_exc=0.27, w_inh=-4.5, steps=1000)
    elif index == 1:
        n = 250_000
        s = 80.0 / (0.02 * n)
        c.update(n=n, conn_kind=BERNOULLI, p=0.02, w_exc=_f32(0.27 * s), w_inh=_f32(-4.5 * s),
                 steps=10_000)
    elif index == 2:
        c.update(n=100_000, conn_kind=FIXED_IN, k_in_exc=8000, k_in_inh=2000, w_exc=0.1,
                 w_inh=-0.5, delay_min=15, delay_max=15, ext_lambda=1.0, ext_w=0.1,
                 steps=10_000)
    elif index == 3:
        c.update(n=1_000_000, neuron_kind=SOURCE, frac_exc=1.0, dt_ms=1.0, conn_kind=FIXED_OUT,
                 k_out=1000, w_uniform=1, w_lo=0.0, w_hi=1e-3, w_exc=0.0, w_inh=0.0,
                 src_rate_hz=rate_hz, steps=1000)
    elif index == 4:
        s = 80.0 / 1500.0
        c.update(n=2_000_000, conn_kind=FIXED_OUT, k_out=1500, w_exc=_f32(0.27 * s),
                 w_inh=_f32(-4.5 * s), delay_min=1, delay_max=20, steps=5000)
    else:
        raise ValueError(index)
    if driven and c["neuron_kind"] == LIF and c["ext_lambda"] == 0.0:
        c["ext_lambda"] = drive_lambda(c)
        c["ext_w"] = c["w_exc"]
    for k, v in over.items():
        c[k] = v
    for k in ("v_rest", "v_th", "v_reset", "v0_lo", "v0_hi", "i_bias", "w_exc", "w_inh",
              "w_lo", "w_hi", "ext_w"):
        c[k] = _f32(c[k])
    return c


def synth(n: int, density: float = 0.05, seed: int = 1, **over) -> dict:
    """The Synth shape of the setup-time study (Sec. IV-C): one intra-connected
    LIF population, Bernoulli connectivity of the given density, delay 1,
    weights scaled by 80/(density n) as in C1."""
    s = 80.0 / (density * n)
    c = dict(_MEMBRANE, seed=seed, n=n, frac_exc=1.0, conn_kind=BERNOULLI, p=density,
             w_exc=_f32(0.27 * s), w_inh=_f32(-4.5 * s), steps=1000)
    c.update(over)
    for k in ("v_rest", "v_th", "v_reset", "v0_lo", "v0_hi", "i_bias", "w_exc", "w_inh",
              "w_lo", "w_hi", "ext_w"):
        c[k] = _f32(c[k])
    return c


def scaled(index: int, n: int, driven: bool = True, **over) -> dict:
    """A reduced-size network with the per-neuron statistics of C<index>:
    Bernoulli p is rescaled to keep the expected in-degree when n is small
    enough, fixed degrees are clipped to n."""
    c = config(index, driven=driven, **over)
    full = c["n"]
    c["n"] = n
    if c["conn_kind"] == BERNOULLI:
        c["p"] = min(1.0, c["p"] * full / n) if index == 1 else c["p"]
    if c["conn_kind"] == FIXED_IN:
        ne = int(round(0.8 * n))
        c["k_in_exc"] = min(c["k_in_exc"], max(1, ne // 10))
        c["k_in_inh"] = min(c["k_in_inh"], max(1, (n - ne) // 10))
    for k, v in over.items():
        c[k] = v
    return c


def random_shape(seed: int) -> dict:
    """A seeded random network shape for broad parity sweeps: n in [40, 6000),
    Bernoulli, fixed out-degree or fixed in-degree connectivity, smallest
    delay 1-5 with 1 to 26 delay lists, weights scaled by 80 / (expected
    in-degree) as in C1 (at most 1x), and the driven variant's Poisson drive."""
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(40, 6000))
    kind = int(rng.choice([BERNOULLI, FIXED_OUT, FIXED_IN]))
    dmin = int(rng.integers(1, 6))
    dmax = dmin + int(rng.choice([0, 0, 3, 12, 25]))
    c = dict(_MEMBRANE, seed=int(seed), n=n, conn_kind=kind, delay_min=dmin, delay_max=dmax, steps=200)
    if kind == BERNOULLI:
        c["p"] = float(rng.uniform(0.002, 0.15))
        deg = c["p"] * n
    elif kind == FIXED_OUT:
        c["k_out"] = int(rng.integers(1, min(n, 400) + 1))
        deg = float(c["k_out"])
    else:
        ne = int(round(0.8 * n))
        c["k_in_exc"] = int(rng.integers(1, max(2, min(ne, 320))))
        c["k_in_inh"] = int(rng.integers(1, max(2, min(n - ne, 80))))
        deg = float(c["k_in_exc"] + c["k_in_inh"])
    sc = min(1.0, 80.0 / max(deg, 1.0))
    c["w_exc"], c["w_inh"] = _f32(0.27 * sc), _f32(-4.5 * sc)
    c["ext_w"] = c["w_exc"]
    c["ext_lambda"] = drive_lambda(c)
    for k in ("v_rest", "v_th", "v_reset", "v0_lo", "v0_hi", "i_bias", "w_lo", "w_hi"):
        c[k] = _f32(c[k])
    return c


def spike_set(n: int, count: int, seed: int, unique: bool = True) -> np.ndarray:
    """Seeded random spike IDs in [0, n)."""
    rng = np.random.default_rng(seed)
    if unique:
        return np.sort(rng.choice(n, size=min(count, n), replace=False)).astype(np.uint32)
    return rng.integers(0, n, size=count, dtype=np.uint32)


def random_csr(n: int, mean_deg: float, seed: int, delay_max: int = 1, w_scale: float = 1.0,
               max_deg: int | None = None):
    """Seeded random explicit adjacency list (rows unsorted, multapses possible)."""
    rng = np.random.default_rng(seed)
    deg = rng.poisson(mean_deg, size=n)
    if max_deg is not None:
        deg = np.minimum(deg, max_deg)
    row_ptr = np.zeros(n + 1, dtype=np.uint64)
    row_ptr[1:] = np.cumsum(deg)
    nnz = int(row_ptr[-1])
    col = rng.integers(0, n, size=nnz, dtype=np.uint32)
    w = (rng.standard_normal(nnz) * w_scale).astype(np.float32)
    delay = rng.integers(1, delay_max + 1, size=nnz).astype(np.uint8)
    return row_ptr, col, w, delay


def fig_adj():
    """The paper's Fig. 'adj' fixture as a dict (see tests/golden/fig_adj.txt)."""
    rows, out = [], {}
    with open(os.path.join(GOLDEN, "fig_adj.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].split()
            if not line:
                continue
            key, vals = line[0], line[1:]
            if key == "row":
                rows.append([int(v) for v in vals if v != "-"])
            else:
                out[key] = [int(v) for v in vals]
    n = len(rows)
    row_ptr = np.zeros(n + 1, dtype=np.uint64)
    row_ptr[1:] = np.cumsum([len(r) for r in rows])
    col = np.array([c for r in rows for c in r], dtype=np.uint32)
    out.update(rows=rows, n=n, row_ptr=row_ptr, col=col,
               w=np.ones(len(col), dtype=np.float32),
               delay=np.ones(len(col), dtype=np.uint8))
    return out


def explicit_params(n: int, **over) -> dict:
    """Parameters for a network given by an explicit adjacency list."""
    c = dict(_MEMBRANE, seed=1, n=n, conn_kind=EXPLICIT, w_exc=0.0, w_inh=0.0)
    c.update(over)
    for k in ("v_rest", "v_th", "v_reset", "v0_lo", "v0_hi", "i_bias", "w_exc", "w_inh",
              "w_lo", "w_hi", "ext_w"):
        c[k] = _f32(c[k])
    return c
