"""ctypes binding of libspk (include/spk.h).

Argument marshalling only: every step of the simulation runs in the HIP
kernels of libspk.so.  There is no fallback path; if the library is not
built (``python -m paper_2102_04681_amd._build``) or cannot be loaded,
``lib()`` raises.

``Net`` accepts the same parameter dictionary keys as the fields of
``spk_params``; ``stream`` may be a ``torch.cuda.Stream`` (its HIP stream is
used) or an integer handle; ``None`` lets the library create its own stream.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libspk.so")

SPK_OK, SPK_EINVAL, SPK_ENOMEM, SPK_EHIP, SPK_EOVERFLOW, SPK_ESTATE = 0, -1, -2, -3, -4, -5
SPK_ABI_VERSION = 5
SPK_LIF, SPK_SOURCE = 0, 1
SPK_CONN_BERNOULLI, SPK_CONN_FIXED_OUT, SPK_CONN_FIXED_IN, SPK_CONN_EXPLICIT = 0, 1, 2, 3
SPK_ACC_F32, SPK_ACC_FIXED = 0, 1
SPK_DELIVERY_AUTO, SPK_DELIVERY_DIRECT, SPK_DELIVERY_BINNED = 0, 1, 2
SPK_FORMAT_AUTO, SPK_FORMAT_FULL, SPK_FORMAT_COMPACT, SPK_FORMAT_PROCEDURAL = 0, 1, 2, 3
SPK_STEP_AUTO, SPK_STEP_GRAPH, SPK_STEP_PERSISTENT = 0, 1, 2

EXPORTED = [
    "spk_preset", "spk_create", "spk_create_from_csr", "spk_step", "spk_sync",
    "spk_read_spike_counts", "spk_read_events", "spk_read_delivered", "spk_read_raster",
    "spk_read_state", "spk_debug_deliver", "spk_export_rows", "spk_poisson_table", "spk_stats",
    "spk_set_profiling", "spk_read_kernel_ms", "spk_hbm_copy", "spk_hbm_read", "spk_deliver_noalloc",
    "spk_destroy", "spk_last_error",
    "spk_abi_version",
]


class spk_params(C.Structure):
    _fields_ = [
        ("abi_version", C.c_uint32), ("n", C.c_uint32), ("seed", C.c_uint64),
        ("neuron_kind", C.c_uint32), ("conn_kind", C.c_uint32),
        ("frac_exc", C.c_double), ("dt_ms", C.c_double), ("tau_m_ms", C.c_double),
        ("t_ref_ms", C.c_double),
        ("v_rest", C.c_float), ("v_th", C.c_float), ("v_reset", C.c_float),
        ("v0_lo", C.c_float), ("v0_hi", C.c_float), ("i_bias", C.c_float),
        ("p", C.c_double), ("k_out", C.c_uint32), ("k_in_exc", C.c_uint32),
        ("k_in_inh", C.c_uint32), ("w_uniform", C.c_uint32),
        ("w_exc", C.c_float), ("w_inh", C.c_float), ("w_lo", C.c_float), ("w_hi", C.c_float),
        ("delay_min", C.c_uint32), ("delay_max", C.c_uint32),
        ("ext_lambda", C.c_double), ("ext_w", C.c_float), ("acc_mode", C.c_uint32),
        ("src_rate_hz", C.c_double), ("fixed_shift", C.c_int32), ("delivery", C.c_uint32),
        ("syn_format", C.c_uint32), ("step_mode", C.c_uint32), ("max_steps", C.c_uint64),
        ("raster_capacity", C.c_uint64),
    ]


class spk_stats_t(C.Structure):
    _fields_ = [
        ("n", C.c_uint64), ("nnz", C.c_uint64), ("steps", C.c_uint64),
        ("device_bytes", C.c_uint64),
        ("n_exc", C.c_uint32), ("ref_steps", C.c_uint32), ("ring_slots", C.c_uint32),
        ("delay_lists", C.c_uint32), ("max_row", C.c_uint32), ("pois_len", C.c_uint32),
        ("fixed_shift", C.c_int32), ("k", C.c_float), ("bytes_per_synapse", C.c_double),
        ("tile_width", C.c_uint32), ("tiles", C.c_uint32), ("delivery", C.c_uint32),
        ("page_cap", C.c_uint32), ("step_mode", C.c_uint32),
        ("batch_steps", C.c_uint32), ("setup_ms", C.c_double), ("gen_ms", C.c_double), ("range_ms", C.c_double),
    ]


_lib = None


def lib():
    """Load libspk.so (raises if it is missing: there is no other path)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"libspk.so not built at {_LIB_PATH}; run "
                               "`python -m paper_2102_04681_amd._build`")
        L = C.CDLL(_LIB_PATH)
        P, u64, u32, i32 = C.c_void_p, C.c_uint64, C.c_uint32, C.c_int
        sig = {
            "spk_preset": (i32, [i32, i32, C.c_double, u64, C.POINTER(spk_params)]),
            "spk_create": (i32, [C.POINTER(spk_params), P, C.POINTER(P)]),
            "spk_create_from_csr": (i32, [C.POINTER(spk_params), u32, P, P, P, P, P, C.POINTER(P)]),
            "spk_step": (i32, [P, u64]),
            "spk_sync": (i32, [P]),
            "spk_read_spike_counts": (i32, [P, u64, u64, P]),
            "spk_read_events": (i32, [P, u64, u64, P]),
            "spk_read_delivered": (i32, [P, u64, u64, P]),
            "spk_read_raster": (i32, [P, u64, u64, P, P, u64]),
            "spk_read_state": (i32, [P, P, P]),
            "spk_debug_deliver": (i32, [P, P, u64, u32, P, P]),
            "spk_export_rows": (i32, [P, P, u64, P, P, P, P, P, u64]),
            "spk_poisson_table": (i32, [P, P, u32, C.POINTER(u32)]),
            "spk_stats": (i32, [P, C.POINTER(spk_stats_t)]),
            "spk_set_profiling": (i32, [P, i32]),
            "spk_read_kernel_ms": (i32, [P, C.POINTER(C.c_double), C.POINTER(C.c_double),
                                         C.POINTER(C.c_double), C.POINTER(u64), C.POINTER(u64)]),
            "spk_hbm_copy": (i32, [P, u64, i32, C.POINTER(C.c_double)]),
            "spk_hbm_read": (i32, [P, u64, i32, C.POINTER(C.c_double)]),
            "spk_deliver_noalloc": (i32, [P, P, u64, u32, P]),
            "spk_destroy": (None, [P]),
            "spk_last_error": (C.c_char_p, []),
            "spk_abi_version": (u32, []),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        if L.spk_abi_version() != SPK_ABI_VERSION:
            raise RuntimeError("libspk ABI version mismatch")
        _lib = L
    return _lib


class SpkError(RuntimeError):
    def __init__(self, code: int, what: str):
        msg = lib().spk_last_error().decode(errors="replace")
        super().__init__(f"{what}: status {code}: {msg}")
        self.code = code


def _check(rc: int, what: str):
    if rc != SPK_OK:
        raise SpkError(rc, what)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _stream_handle(stream):
    """HIP stream handle for the C ABI; None = a library-owned stream.

    The legacy default stream (handle 0) cannot be named through the ABI
    (NULL there means "create a stream"), so passing it is an error: use a
    torch.cuda.Stream() and make it current instead."""
    if stream is None:
        return None
    h = stream if isinstance(stream, int) else int(stream.cuda_stream)
    if h == 0:
        raise ValueError("the default (null) stream cannot be shared with libspk; "
                         "pass a torch.cuda.Stream()")
    return h


def make_params(cfg: dict, max_steps: int | None = None, raster_capacity: int = 0) -> spk_params:
    p = spk_params()
    p.abi_version = SPK_ABI_VERSION
    for name, _ in spk_params._fields_:
        if name in cfg:
            setattr(p, name, cfg[name])
    p.max_steps = int(max_steps if max_steps is not None else cfg.get("max_steps", cfg.get("steps", 1)))
    p.raster_capacity = int(raster_capacity if raster_capacity else cfg.get("raster_capacity", 0))
    return p


def preset(index: int, driven: bool = False, rate_hz: float = 10.0, seed: int = 1) -> dict:
    """spk_preset as a dictionary of spk_params fields."""
    p = spk_params()
    _check(lib().spk_preset(index, 1 if driven else 0, rate_hz, seed, C.byref(p)), "spk_preset")
    return {name: getattr(p, name) for name, _ in spk_params._fields_}


class Net:
    """A network owned by libspk (thin handle; all work happens in HIP)."""

    def __init__(self, cfg: dict, stream=None, max_steps: int | None = None,
                 raster_capacity: int = 0, csr=None):
        self.cfg = dict(cfg)
        self._p = make_params(cfg, max_steps, raster_capacity)
        h = C.c_void_p()
        s = _stream_handle(stream)
        if csr is None:
            _check(lib().spk_create(C.byref(self._p), s, C.byref(h)), "spk_create")
            self.n = int(cfg["n"])
        else:
            row_ptr, col, w, delay = csr
            self._csr_keep = (np.ascontiguousarray(row_ptr, dtype=np.uint64),
                              np.ascontiguousarray(col, dtype=np.uint32),
                              np.ascontiguousarray(w, dtype=np.float32),
                              None if delay is None else np.ascontiguousarray(delay, dtype=np.uint8))
            rp, cc, ww, dd = self._csr_keep
            self.n = len(rp) - 1
            _check(lib().spk_create_from_csr(C.byref(self._p), self.n, _ptr(rp), _ptr(cc), _ptr(ww),
                                             _ptr(dd), s, C.byref(h)), "spk_create_from_csr")
        self._h = h
        self.fixed = int(cfg.get("acc_mode", 0)) == SPK_ACC_FIXED

    def close(self):
        if getattr(self, "_h", None):
            lib().spk_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def step(self, n_steps: int):
        _check(lib().spk_step(self._h, n_steps), "spk_step")

    def sync(self):
        _check(lib().spk_sync(self._h), "spk_sync")

    def stats(self) -> dict:
        s = spk_stats_t()
        _check(lib().spk_stats(self._h, C.byref(s)), "spk_stats")
        return {name: getattr(s, name) for name, _ in spk_stats_t._fields_}

    @property
    def t(self) -> int:
        return int(self.stats()["steps"])

    def spike_counts(self, t0: int = 0, n: int | None = None) -> np.ndarray:
        n = self.t - t0 if n is None else n
        out = np.zeros(n, dtype=np.uint32)
        _check(lib().spk_read_spike_counts(self._h, t0, n, _ptr(out)), "spk_read_spike_counts")
        return out

    def events(self, t0: int = 0, n: int | None = None) -> np.ndarray:
        n = self.t - t0 if n is None else n
        out = np.zeros(n, dtype=np.uint64)
        _check(lib().spk_read_events(self._h, t0, n, _ptr(out)), "spk_read_events")
        return out

    def delivered(self, t0: int = 0, n: int | None = None) -> np.ndarray:
        n = self.t - t0 if n is None else n
        out = np.zeros(n, dtype=np.uint64)
        _check(lib().spk_read_delivered(self._h, t0, n, _ptr(out)), "spk_read_delivered")
        return out

    def raster(self, t0: int = 0, n: int | None = None):
        n = self.t - t0 if n is None else n
        counts = self.spike_counts(t0, n)
        cap = int(counts.sum())
        offs = np.zeros(n + 1, dtype=np.uint64)
        ids = np.zeros(max(cap, 1), dtype=np.uint32)
        _check(lib().spk_read_raster(self._h, t0, n, _ptr(offs), _ptr(ids), cap), "spk_read_raster")
        return offs, ids[:int(offs[-1])]

    def state(self):
        v = np.zeros(self.n, dtype=np.float32)
        ref = np.zeros(self.n, dtype=np.uint8)
        _check(lib().spk_read_state(self._h, _ptr(v), _ptr(ref)), "spk_read_state")
        return v, ref

    def debug_deliver(self, spikes, delay: int = 0) -> np.ndarray:
        spikes = np.ascontiguousarray(spikes, dtype=np.uint32)
        if self.fixed:
            out = np.zeros(self.n, dtype=np.int32)
            _check(lib().spk_debug_deliver(self._h, _ptr(spikes), len(spikes), delay, None, _ptr(out)),
                   "spk_debug_deliver")
        else:
            out = np.zeros(self.n, dtype=np.float32)
            _check(lib().spk_debug_deliver(self._h, _ptr(spikes), len(spikes), delay, _ptr(out), None),
                   "spk_debug_deliver")
        return out

    def deliver_noalloc(self, d_spikes: int, n_spikes: int, d_out: int, delay: int = 0):
        """spk_deliver_noalloc on device pointers (ints); asynchronous."""
        _check(lib().spk_deliver_noalloc(self._h, C.c_void_p(d_spikes or None), n_spikes, delay,
                                         C.c_void_p(d_out or None)), "spk_deliver_noalloc")

    def export_rows(self, rows, cap: int | None = None):
        rows = np.ascontiguousarray(rows, dtype=np.uint32)
        st = self.stats()
        if cap is None:
            cap = max(1, int(st["nnz"]) if len(rows) > 64 else
                      len(rows) * max(1, int(st["max_row"])))
        offs = np.zeros(len(rows) + 1, dtype=np.uint64)
        col = np.zeros(cap, dtype=np.uint32)
        w = np.zeros(cap, dtype=np.float32)
        wq = np.zeros(cap, dtype=np.int32)
        d = np.zeros(cap, dtype=np.uint8)
        _check(lib().spk_export_rows(self._h, _ptr(rows), len(rows), _ptr(offs), _ptr(col), _ptr(w),
                                     _ptr(wq), _ptr(d), cap), "spk_export_rows")
        m = int(offs[-1])
        return offs, col[:m].copy(), (wq if self.fixed else w)[:m].copy(), d[:m].copy()

    def csr(self):
        """All rows (row_ptr, col, weight, delay) in canonical row order."""
        offs, col, w, d = self.export_rows(np.arange(self.n, dtype=np.uint32),
                                           cap=max(1, int(self.stats()["nnz"])))
        return offs, col, w, d

    def poisson_table(self) -> np.ndarray:
        thr = np.zeros(256, dtype=np.uint64)
        L = C.c_uint32()
        _check(lib().spk_poisson_table(self._h, _ptr(thr), 256, C.byref(L)), "spk_poisson_table")
        return thr[:L.value].copy()

    def set_profiling(self, on: bool):
        _check(lib().spk_set_profiling(self._h, 1 if on else 0), "spk_set_profiling")

    def kernel_ms(self) -> dict:
        """Summed kernel durations (ms) since set_profiling: push, tile and
        persistent launches, with the step and persistent-launch counts."""
        d, u, r = C.c_double(), C.c_double(), C.c_double()
        n, nr = C.c_uint64(), C.c_uint64()
        _check(lib().spk_read_kernel_ms(self._h, C.byref(d), C.byref(u), C.byref(r), C.byref(n),
                                        C.byref(nr)), "spk_read_kernel_ms")
        return {"push_ms": d.value, "tile_ms": u.value, "run_ms": r.value, "steps": n.value,
                "run_launches": nr.value}

    def hbm_read(self, nbytes: int, reps: int = 10) -> float:
        ms = C.c_double()
        _check(lib().spk_hbm_read(self._h, nbytes, reps, C.byref(ms)), "spk_hbm_read")
        return ms.value

    def hbm_copy(self, nbytes: int, reps: int = 10) -> float:
        ms = C.c_double()
        _check(lib().spk_hbm_copy(self._h, nbytes, reps, C.byref(ms)), "spk_hbm_copy")
        return ms.value
