"""CPU oracle for the spike-transmission path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product (``paper_2102_04681_amd``)
never imports, links or runs anything here, and this package never imports
the product: the two share no code.

This module is argument marshalling (ctypes) around ``spk_oracle.c``; all
arithmetic lives in the C file, which follows the paper (arXiv 2102.04681)
section by section -- see the header of ``spk_oracle.c``.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "spk_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

OK, EINVAL, ENOMEM, EOVERFLOW = 0, -1, -2, -4
TAG = dict(CONN=1, TGT=2, SRC_E=3, SRC_I=4, W=5, DELAY=6, V0=7, POIS=8, BERN=9)


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no FMA contraction, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call([
            "gcc", "-O2", "-std=c99", "-D_DEFAULT_SOURCE", "-ffp-contract=off",
            "-fno-fast-math", "-Wall", "-Wextra", "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class Params(C.Structure):
    _fields_ = [
        ("seed", C.c_uint64), ("n", C.c_uint32), ("neuron_kind", C.c_uint32),
        ("frac_exc", C.c_double), ("dt_ms", C.c_double), ("tau_m_ms", C.c_double),
        ("t_ref_ms", C.c_double),
        ("v_rest", C.c_float), ("v_th", C.c_float), ("v_reset", C.c_float),
        ("v0_lo", C.c_float), ("v0_hi", C.c_float), ("i_bias", C.c_float),
        ("conn_kind", C.c_uint32), ("p", C.c_double), ("k_out", C.c_uint32),
        ("k_in_exc", C.c_uint32), ("k_in_inh", C.c_uint32),
        ("w_exc", C.c_float), ("w_inh", C.c_float), ("w_uniform", C.c_uint32),
        ("w_lo", C.c_float), ("w_hi", C.c_float),
        ("delay_min", C.c_uint32), ("delay_max", C.c_uint32),
        ("ext_lambda", C.c_double), ("ext_w", C.c_float), ("src_rate_hz", C.c_double),
        ("acc_mode", C.c_uint32), ("fixed_shift", C.c_int32),
    ]


class Derived(C.Structure):
    _fields_ = [
        ("n_exc", C.c_uint32), ("k", C.c_float), ("ref_steps", C.c_uint32),
        ("ring", C.c_uint32), ("conn_thr", C.c_uint64), ("src_thr", C.c_uint64),
        ("pois_len", C.c_uint32), ("ext_wq", C.c_int32), ("bias_q", C.c_int32),
        ("w_exc_q", C.c_int32), ("w_inh_q", C.c_int32), ("nnz", C.c_uint64),
        ("max_row", C.c_uint32),
    ]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        L = C.CDLL(_LIB)
        P, u64, u32, i32 = C.c_void_p, C.c_uint64, C.c_uint32, C.c_int
        L.orc_splitmix64.restype = u64
        L.orc_splitmix64.argtypes = [u64]
        L.orc_hash.restype = u64
        L.orc_hash.argtypes = [u64, u32, u64, u64]
        L.orc_hash_step.restype = u64
        L.orc_hash_step.argtypes = [u64, u32, u32, u32]
        L.orc_poisson_table.restype = i32
        L.orc_poisson_table.argtypes = [C.c_double, P, i32]
        L.orc_create.restype = i32
        L.orc_create.argtypes = [C.POINTER(Params), i32, C.POINTER(P)]
        L.orc_create_explicit.restype = i32
        L.orc_create_explicit.argtypes = [C.POINTER(Params), u32, P, P, P, P, C.POINTER(P)]
        L.orc_destroy.restype = None
        L.orc_destroy.argtypes = [P]
        L.orc_get_derived.restype = i32
        L.orc_get_derived.argtypes = [P, C.POINTER(Derived)]
        L.orc_nnz.restype = u64
        L.orc_nnz.argtypes = [P]
        L.orc_get_csr.restype = i32
        L.orc_get_csr.argtypes = [P, P, P, P, P]
        L.orc_row.restype = i32
        L.orc_row.argtypes = [P, u32, P, P, P, u64, C.POINTER(u64)]
        L.orc_in_row.restype = i32
        L.orc_in_row.argtypes = [P, u32, P, P, P, u64, C.POINTER(u64)]
        L.orc_deliver.restype = i32
        L.orc_deliver.argtypes = [P, P, u64, u32, P, P]
        L.orc_run.restype = i32
        L.orc_run.argtypes = [P, u64, P, P, P, P, u64, P]
        L.orc_pair.restype = i32
        L.orc_pair.argtypes = [P, u32, u32, C.POINTER(C.c_int), C.POINTER(C.c_float), C.POINTER(C.c_uint8)]
        L.orc_get_state.restype = i32
        L.orc_get_state.argtypes = [P, P, P]
        L.orc_step_index.restype = u64
        L.orc_step_index.argtypes = [P]
        L.orc_update_one.restype = i32
        L.orc_update_one.argtypes = [P, u64, u32, C.c_float, C.c_uint8, C.c_float, C.c_int64,
                                     C.POINTER(C.c_float), C.POINTER(C.c_uint8), C.POINTER(C.c_int)]
        L.orc_in_abs_sum_q.restype = i32
        L.orc_in_abs_sum_q.argtypes = [P, P]
        _lib = L
    return _lib


class OracleError(RuntimeError):
    def __init__(self, code, what):
        super().__init__(f"oracle {what} failed with status {code}")
        self.code = code


def _check(rc, what):
    if rc != OK:
        raise OracleError(rc, what)


def _ptr(a):
    return a.ctypes.data_as(C.c_void_p) if a is not None else None


def make_params(cfg: dict) -> Params:
    p = Params()
    for name, _ in Params._fields_:
        if name in cfg:
            setattr(p, name, cfg[name])
    return p


def splitmix64(z: int) -> int:
    return lib().orc_splitmix64(z)


def hash64(seed: int, tag: int, a: int, b: int) -> int:
    return lib().orc_hash(seed, tag, a, b)


def hash_step(seed: int, tag: int, i: int, t: int) -> int:
    return lib().orc_hash_step(seed, tag, i, t)


def poisson_table(lam: float, cap: int = 256) -> np.ndarray:
    thr = np.zeros(cap, dtype=np.uint64)
    L = lib().orc_poisson_table(lam, _ptr(thr), cap)
    _check(0 if L > 0 else L, "poisson_table")
    return thr[:L].copy()


class Net:
    """An oracle network (owned C object)."""

    def __init__(self, cfg: dict, build_csr: bool = True, csr=None):
        self.cfg = dict(cfg)
        self._p = make_params(cfg)
        h = C.c_void_p()
        if csr is None:
            _check(lib().orc_create(C.byref(self._p), 1 if build_csr else 0, C.byref(h)),
                   "create")
        else:
            row_ptr, col, w, delay = csr
            row_ptr = np.ascontiguousarray(row_ptr, dtype=np.uint64)
            col = np.ascontiguousarray(col, dtype=np.uint32)
            w = np.ascontiguousarray(w, dtype=np.float32)
            delay = None if delay is None else np.ascontiguousarray(delay, dtype=np.uint8)
            n = len(row_ptr) - 1
            _check(lib().orc_create_explicit(C.byref(self._p), n, _ptr(row_ptr), _ptr(col),
                                             _ptr(w), _ptr(delay), C.byref(h)), "create_explicit")
        self._h = h
        self.n = int(cfg["n"]) if csr is None else len(csr[0]) - 1

    def close(self):
        if self._h:
            lib().orc_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def derived(self) -> dict:
        d = Derived()
        _check(lib().orc_get_derived(self._h, C.byref(d)), "derived")
        return {name: getattr(d, name) for name, _ in Derived._fields_}

    @property
    def nnz(self) -> int:
        return int(lib().orc_nnz(self._h))

    def csr(self):
        nnz = self.nnz
        row_ptr = np.zeros(self.n + 1, dtype=np.uint64)
        col = np.zeros(max(nnz, 1), dtype=np.uint32)
        w = np.zeros(max(nnz, 1), dtype=np.float32)
        d = np.zeros(max(nnz, 1), dtype=np.uint8)
        _check(lib().orc_get_csr(self._h, _ptr(row_ptr), _ptr(col), _ptr(w), _ptr(d)), "get_csr")
        return row_ptr, col[:nnz], w[:nnz], d[:nnz]

    def row(self, s: int, cap: int | None = None):
        cap = cap or max(self.n, int(self.cfg.get("k_out", 0)), 1)
        tgt = np.zeros(cap, dtype=np.uint32)
        w = np.zeros(cap, dtype=np.float32)
        d = np.zeros(cap, dtype=np.uint8)
        L = C.c_uint64()
        _check(lib().orc_row(self._h, s, _ptr(tgt), _ptr(w), _ptr(d), cap, C.byref(L)), "row")
        L = L.value
        return tgt[:L].copy(), w[:L].copy(), d[:L].copy()

    def in_row(self, tgt: int):
        """Fixed in-degree: the in-synapses of target tgt (source, weight,
        delay) in draw order (Sec. III-B), without the CSR."""
        cap = int(self.cfg["k_in_exc"]) + int(self.cfg["k_in_inh"])
        src = np.zeros(max(cap, 1), dtype=np.uint32)
        w = np.zeros(max(cap, 1), dtype=np.float32)
        d = np.zeros(max(cap, 1), dtype=np.uint8)
        L = C.c_uint64()
        _check(lib().orc_in_row(self._h, tgt, _ptr(src), _ptr(w), _ptr(d), cap, C.byref(L)), "in_row")
        L = L.value
        return src[:L].copy(), w[:L].copy(), d[:L].copy()

    def deliver(self, spikes, delay: int = 0, fixed: bool = False):
        spikes = np.ascontiguousarray(spikes, dtype=np.uint32)
        out_f = np.zeros(self.n, dtype=np.float64)
        out_q = np.zeros(self.n, dtype=np.int64) if fixed else None
        _check(lib().orc_deliver(self._h, _ptr(spikes), len(spikes), delay, _ptr(out_f),
                                 _ptr(out_q)), "deliver")
        return (out_f, out_q) if fixed else out_f

    def run(self, n_steps: int, raster_cap: int | None = None):
        """Run n_steps; per-step spike counts, events emitted, events
        delivered (arriving), and the raster (offs, IDs ascending per step).
        A network made with build_csr=False generates each spike's row when
        it is delivered (Bernoulli and fixed out-degree)."""
        counts = np.zeros(n_steps, dtype=np.uint32)
        events = np.zeros(n_steps, dtype=np.uint64)
        delivered = np.zeros(n_steps, dtype=np.uint64)
        offs = np.zeros(n_steps + 1, dtype=np.uint64)
        cap = raster_cap if raster_cap is not None else n_steps * self.n
        raster = np.zeros(max(cap, 1), dtype=np.uint32)
        _check(lib().orc_run(self._h, n_steps, _ptr(counts), _ptr(events), _ptr(delivered), _ptr(raster),
                             cap, _ptr(offs)), "run")
        return dict(counts=counts, events=events, delivered=delivered, offs=offs,
                    raster=raster[:int(offs[-1])].copy())

    def pair(self, s: int, tgt: int):
        """Bernoulli networks: (connected, weight, delay) of the pair s -> tgt."""
        c, w, d = C.c_int(), C.c_float(), C.c_uint8()
        _check(lib().orc_pair(self._h, s, tgt, C.byref(c), C.byref(w), C.byref(d)), "pair")
        return bool(c.value), np.float32(w.value), int(d.value)

    def state(self):
        v = np.zeros(self.n, dtype=np.float32)
        ref = np.zeros(self.n, dtype=np.uint8)
        _check(lib().orc_get_state(self._h, _ptr(v), _ptr(ref)), "state")
        return v, ref

    @property
    def t(self) -> int:
        return int(lib().orc_step_index(self._h))

    def update_one(self, t, i, v, ref, isyn_f=0.0, isyn_q=0):
        vo, ro, sp = C.c_float(), C.c_uint8(), C.c_int()
        _check(lib().orc_update_one(self._h, t, i, v, ref, isyn_f, isyn_q, C.byref(vo),
                                    C.byref(ro), C.byref(sp)), "update_one")
        return vo.value, ro.value, bool(sp.value)

    def in_abs_sum_q(self):
        out = np.zeros(self.n, dtype=np.int64)
        _check(lib().orc_in_abs_sum_q(self._h, _ptr(out)), "in_abs_sum_q")
        return out
