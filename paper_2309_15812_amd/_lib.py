"""ctypes binding of the C ABI in include/o1d.h (argument marshalling only).

Every computation runs in the HIP library ``libo1d.so``; if it is missing or
fails to load, these functions raise instead of falling back to anything.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libo1d.so")

O1D_F32, O1D_BF16 = 0, 1
O1D_NCHW, O1D_NHWC = 0, 1
O1D_FLOOR, O1D_BILINEAR = 0, 1
STATUS = {0: "O1D_OK", 1: "O1D_ERR_INVALID", 2: "O1D_ERR_UNSUPPORTED", 3: "O1D_ERR_WORKSPACE", 4: "O1D_ERR_HIP"}
MAX_K = 127

# name -> (restype, argtypes), mirroring include/o1d.h
_vp, _i, _sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
SIGNATURES = {
    "o1d_fwd": (_i, [_vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp]),
    "o1d_bwd_input": (_i, [_vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp]),
    "o1d_bwd_weight": (_i, [_vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp, _sz, _vp]),
    "o1d_bwd": (_i, [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp, _sz, _vp]),
    "o1d_bwd_noalloc": (_i, [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp]),
    "o1d_bwd_weight_workspace_bytes": (_sz, [_i, _i, _i, _i, _i, _i]),
    "o1d_fwd_ex": (_i, [_vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _i, _i, _i, _vp]),
    "o1d_bwd_input_ex": (_i, [_vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _i, _i, _i, _vp]),
    "o1d_bwd_weight_ex": (_i, [_vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _i, _i, _i, _vp, _sz, _vp]),
    "o1d_bwd_weight_ex_workspace_bytes": (_sz, [_i, _i, _i, _i, _i, _i, _i, _i, _i]),
    "o1d_dsc_fwd": (_i, [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _i, _vp]),
    "o1d_dsc_bwd": (_i, [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _i, _vp, _sz, _vp]),
    "o1d_dsc_bwd_workspace_bytes": (_sz, [_i, _i, _i, _i, _i, _i, _i]),
    "o1d_kernel_name": (ctypes.c_char_p, [_i, _i, _i, _i, _i, _i, _i, _i, _i, _i, _i]),
    "o1d_kernel_variant": (ctypes.c_char_p, [_i]),
    "o1d_status_str": (ctypes.c_char_p, [_i]),
    "o1d_last_error": (ctypes.c_char_p, []),
    "o1d_version": (ctypes.c_char_p, []),
}

_lib = None


class O1DError(RuntimeError):
    def __init__(self, fn: str, status: int, detail: str):
        super().__init__(f"{fn} -> {STATUS.get(status, status)}: {detail}")
        self.status = status


def lib() -> ctypes.CDLL:
    """Load libo1d.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing; build it with `python -m paper_2309_15812_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(handle, name)
            f.restype = res
            f.argtypes = args
        _lib = handle
    return _lib


def check(fn: str, status: int) -> None:
    if status != 0:
        raise O1DError(fn, status, lib().o1d_last_error().decode())


def kernel_name(op: int, N: int, C: int, H: int, W: int, K: int, stride: int = 1, layout: int = O1D_NCHW,
                sampling: int = O1D_FLOOR, dtype: int = O1D_F32, aligned: bool = True) -> str:
    """The kernel(s) a call would launch (host-side planning only, no GPU needed).
    op: 0 forward, 1 input gradient, 2 weight gradient, 3 both gradients (o1d_bwd)."""
    return lib().o1d_kernel_name(op, N, C, H, W, K, stride, layout, sampling, dtype, int(aligned)).decode()


def kernel_variants() -> list[str]:
    """Every kernel instantiation compiled into the library."""
    out, i = [], 0
    while True:
        v = lib().o1d_kernel_variant(i)
        if v is None:
            return out
        out.append(v.decode())
        i += 1


def call(fn: str, *args) -> int:
    """Raw call of a C ABI entry point; returns the status code."""
    return getattr(lib(), fn)(*args)
