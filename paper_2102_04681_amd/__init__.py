"""MI355X-native spike transmission + neuron update (arXiv 2102.04681).

The compute path is libspk.so: HIP kernels for gfx950 behind the C ABI in
include/spk.h.  This package is its Python binding (ctypes) and build
script; PyTorch is only used by callers for streams and device memory.
"""
from .spk import (Net, SpkError, lib, make_params, preset, SPK_ACC_F32, SPK_ACC_FIXED,  # noqa: F401
                  SPK_LIF, SPK_SOURCE, SPK_CONN_BERNOULLI, SPK_CONN_FIXED_OUT, SPK_CONN_FIXED_IN,
                  SPK_CONN_EXPLICIT, SPK_OK, SPK_EINVAL, SPK_ENOMEM, SPK_EHIP, SPK_EOVERFLOW,
                  SPK_ESTATE, SPK_STEP_AUTO, SPK_STEP_GRAPH, SPK_STEP_PERSISTENT, EXPORTED)

__all__ = ["Net", "SpkError", "lib", "make_params", "preset"]
