"""Host-side checks of libspk that need no GPU: the library loads, exports
every symbol include/spk.h declares, presets match the workload
definitions, and parameter validation rejects bad input before any device
call."""
import ctypes as C
import os
import re
import subprocess

import numpy as np
import pytest

import inputs as I
import paper_2102_04681_amd as pkg
from paper_2102_04681_amd import spk

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "spk.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(spk_[a-z_0-9]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    L = spk.lib()
    names = _declared()
    assert len(names) >= 19
    for name in names:
        assert hasattr(L, name), name
    assert sorted(names) == sorted(spk.EXPORTED)
    assert L.spk_abi_version() == spk.SPK_ABI_VERSION


@pytest.mark.parametrize("struct", [spk.spk_params, spk.spk_stats_t])
def test_struct_layout_matches_header(struct, tmp_path):
    # compile a probe against include/spk.h and compare every field offset
    # and the size with the ctypes mirror used by the binding
    name = struct.__name__
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "spk.h"', "int main(void){",
             f'printf("%zu\\n", sizeof({name}));']
    for f, _ in struct._fields_:
        lines.append(f'printf("%zu\\n", offsetof({name}, {f}));')
    lines.append("return 0;}")
    src = tmp_path / "probe.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "probe"
    subprocess.check_call(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)])
    out = [int(x) for x in subprocess.check_output([str(exe)]).split()]
    assert out[0] == C.sizeof(struct)
    assert out[1:] == [getattr(struct, f).offset for f, _ in struct._fields_]


_FIELDS = ["n", "neuron_kind", "conn_kind", "frac_exc", "dt_ms", "tau_m_ms", "t_ref_ms", "v_rest",
           "v_th", "v_reset", "v0_lo", "v0_hi", "i_bias", "p", "k_out", "k_in_exc", "k_in_inh",
           "w_uniform", "w_exc", "w_inh", "w_lo", "w_hi", "delay_min", "delay_max", "ext_lambda",
           "ext_w", "src_rate_hz", "acc_mode", "fixed_shift"]


@pytest.mark.parametrize("index", range(5))
@pytest.mark.parametrize("driven", [False, True])
def test_presets_match_workload_definitions(index, driven):
    got = pkg.preset(index, driven=driven, rate_hz=10.0, seed=3)
    want = I.config(index, driven=driven, seed=3, rate_hz=10.0)
    for f in _FIELDS:
        assert np.float32(got[f]) == np.float32(want[f]) or got[f] == want[f], (f, got[f], want[f])
    assert got["seed"] == 3 and got["max_steps"] == want["steps"]


def _status(cfg, **over):
    p = spk.make_params(dict(cfg, **over), max_steps=10)
    h = C.c_void_p()
    return spk.lib().spk_create(C.byref(p), None, C.byref(h))


@pytest.mark.parametrize("over", [
    dict(n=0), dict(delay_min=0), dict(delay_min=5, delay_max=4), dict(delay_max=300),
    dict(delay_min=1, delay_max=70), dict(dt_ms=0.0), dict(tau_m_ms=-1.0), dict(p=1.5),
    dict(frac_exc=2.0), dict(neuron_kind=7), dict(conn_kind=9), dict(acc_mode=4),
    dict(t_ref_ms=100.0), dict(ext_lambda=500.0), dict(acc_mode=1, fixed_shift=40),
])
def test_invalid_parameters_rejected_on_host(over):
    assert _status(I.config(0), **over) == spk.SPK_EINVAL


def test_fixed_point_weight_range_rejected_on_host():
    assert _status(I.config(0), acc_mode=1, fixed_shift=30, w_inh=-4.5) == spk.SPK_EOVERFLOW


def test_abi_version_checked():
    p = spk.make_params(I.config(0), max_steps=10)
    p.abi_version = 99
    h = C.c_void_p()
    assert spk.lib().spk_create(C.byref(p), None, C.byref(h)) == spk.SPK_EINVAL
    assert b"abi" in spk.lib().spk_last_error()


def test_null_safety():
    L = spk.lib()
    L.spk_destroy(None)
    assert L.spk_step(None, 1) == spk.SPK_EINVAL
    assert L.spk_preset(7, 0, 0.0, 1, C.byref(spk.spk_params())) == spk.SPK_EINVAL


def test_kernel_reciprocal_divisions_are_exact():
    # The persistent kernel replaces two run-time divisions by multiplies
    # with precomputed reciprocals; both are exact over the operand ranges
    # the kernel uses (checked exhaustively here, in exact integers):
    #  - x / T8 as the high 32 bits of x * ceil(2^32 / T8), for x * T8 < 2^32
    #    (x: buckets < 1024, fill counters < 2048, resets < 4096; T8 <= 256);
    #  - q / spc as (q * ceil(2^16 / spc)) >> 16 for q < 256, spc <= 256.
    import numpy as np
    x = np.arange(4096, dtype=np.uint64)
    for t8 in range(2, 257):
        inv = ((1 << 32) + t8 - 1) // t8
        assert inv < (1 << 32)
        got = (x * np.uint64(inv)) >> np.uint64(32)
        assert np.array_equal(got, x // np.uint64(t8)), t8
    q = np.arange(256, dtype=np.uint64)
    for spc in range(1, 257):
        inv = (65536 + spc - 1) // spc
        got = (q * np.uint64(inv)) >> np.uint64(16)
        assert np.array_equal(got, q // np.uint64(spc)), spc
