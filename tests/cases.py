"""Parity cases derived from the library's own kernel planning.

`variant_cases()` finds, for every kernel instantiation compiled into
libo1d.so (o1d_kernel_variant), a small problem that the library's planner
(o1d_kernel_name, the same host code the entry points run) routes to it.  The
GPU parity suite runs every one of these cases against the oracle; the host
suite checks that no compiled variant is left without a case.  Only host-side
planning is called here: no GPU is needed to build the list.
"""
from __future__ import annotations

import functools

from paper_2309_15812_amd import _lib

OPS = {0: "fwd", 1: "bwd_input", 2: "bwd_weight", 3: "bwd"}


def _candidates():
    """Problem sizes (N, C, H, W, K, layout, aligned), smallest first."""
    out = []
    # strip kernels: W a multiple of 4, aligned tensors, every tile stride
    for K in (7, 31, 33, 63):
        for M in range(4, 132, 4):
            for H, W in ((M, M), (max(1, M // 3), M), (max(1, M // 4), M), (M, max(4, (M // 3) // 4 * 4))):
                out.append((3, 4, H, W, K, _lib.O1D_NCHW, True))
    # plane kernels: small NCHW planes with at least eight images
    for K in (7, 31, 63, 127):
        for H, W in ((14, 14), (16, 16), (5, 9), (13, 20), (40, 12), (40, 8)):
            out.append((8, 4, H, W, K, _lib.O1D_NCHW, True))
            out.append((8, 4, H, W, K, _lib.O1D_NCHW, False))
    # general kernels: ragged or unaligned NCHW, NHWC, small and large planes
    for K in (7, 31, 63, 127):
        for H, W in ((14, 14), (5, 9), (30, 30), (40, 33), (130, 70)):
            out.append((3, 4, H, W, K, _lib.O1D_NCHW, False))
            out.append((3, 4, H, W, K, _lib.O1D_NHWC, True))
    out.sort(key=lambda c: (c[0] * c[1] * c[2] * c[3] * c[4], c))
    return out


@functools.lru_cache(maxsize=None)
def variant_cases() -> dict:
    """{variant name: (N, C, H, W, K, dtype, layout, aligned)} for every variant the planner reaches."""
    want = set(_lib.kernel_variants())
    found = {}
    for dt, dname in ((_lib.O1D_F32, "f32"), (_lib.O1D_BF16, "bf16")):
        for (N, C, H, W, K, layout, aligned) in _candidates():
            ops = (0, 1, 2, 3) if layout == _lib.O1D_NCHW else (0, 1, 2)
            for op in ops:
                if layout == _lib.O1D_NHWC and op == 3:
                    continue
                name = _lib.kernel_name(op, N, C, H, W, K, 1, layout, _lib.O1D_FLOOR, dt, aligned)
                for v in name.split("+"):
                    if v in want and v not in found:
                        found[v] = (N, C, H, W, K, dname, "nhwc" if layout == _lib.O1D_NHWC else "nchw", aligned)
            if len(found) == len(want):
                return found
    return found
