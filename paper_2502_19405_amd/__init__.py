"""Bitwise-reproducible fp32 operators (RepOps, Verde arXiv 2502.19405,
Section 3) for AMD MI355X / gfx950.

The operators live in librepops.so (HIP kernels behind the C ABI of
include/repops.h); ``paper_2502_19405_amd.repops`` is the Python binding.
The binding is imported on first use of one of its names so that the input
generators can be imported without torch.
"""
_BINDING_NAMES = ("matmul", "bmm", "bmm_raw", "softmax_rows", "layernorm_rows", "gelu", "exp",
                  "Order", "Launch", "RepopsError", "gemm_configs", "abi_version", "load")


def __getattr__(name):
    if name in _BINDING_NAMES:
        from . import repops
        return getattr(repops, name)
    raise AttributeError(name)
