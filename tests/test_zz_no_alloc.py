"""The no-allocation entry point o1d_bwd_noalloc against o1d_bwd.

o1d_bwd_noalloc keeps the weight gradient's partial rows in the library's
fixed device scratch instead of a caller workspace.  Called through the C
ABI, twice in a row (the second call with a smaller problem, so stale
partial rows of the first call would show), its dx and dw must match
o1d_bwd's on the same inputs, and both must be
bitwise equal (the same kernels and fixed-order sums write them).
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_2309_15812_amd import _lib, ops, synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _noalloc(x, dy, w, th, dx, dw):
    L = _lib.lib()
    f = L.o1d_bwd_noalloc
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_void_p] * 6 + [ctypes.c_int] * 6 + [ctypes.c_void_p]
    N, C, H, W = x.shape
    dt = _lib.O1D_F32 if x.dtype == torch.float32 else _lib.O1D_BF16
    st = f(x.data_ptr(), dy.data_ptr(), w.data_ptr(), th.data_ptr(), dx.data_ptr(), dw.data_ptr(), N, C, H, W,
           w.shape[1], dt, torch.cuda.current_stream().cuda_stream)
    _lib.check("o1d_bwd_noalloc", st)


def _case(N, C, H, W, K, dtype, seed):
    wl = synth.Workload("noalloc", N, C, H, W, K, dtype, "uniform", "fwd+bwd", seed)
    d = synth.make_inputs(wl)
    dt = torch.float32 if dtype == "f32" else torch.bfloat16
    t = {k: torch.from_numpy(d[k]).to(DEV).to(dt) for k in ("x", "dy", "w")}
    return t["x"], t["dy"], t["w"], torch.from_numpy(d["theta"]).to(DEV)


@pytest.mark.parametrize("shapes", [
    ((8, 24, 56, 56, 31, "f32"), (3, 8, 28, 28, 31, "f32")),   # fused strip kernel both times
    ((6, 16, 14, 14, 31, "bf16"), (2, 5, 9, 13, 7, "bf16")),   # general kernels both times
    ((4, 12, 56, 56, 63, "f32"), (2, 4, 20, 24, 15, "f32")),   # strip gather + general weight gradient
])
def test_noalloc_matches_bwd_twice(shapes):
    for i, (N, C, H, W, K, dtype) in enumerate(shapes):
        print(f"[noalloc] call {i}: N={N} C={C} H={H} W={W} K={K} {dtype}", flush=True)
        x, dy, w, th = _case(N, C, H, W, K, dtype, 81 + i)
        rdx, rdw = ops.bwd(x, dy, w, th)
        dx = torch.full_like(x, float("nan"))
        dw = torch.full_like(w, float("nan"))
        _noalloc(x, dy, w, th, dx, dw)
        torch.cuda.synchronize()
        a, b = dw.float().cpu().numpy(), rdw.float().cpu().numpy()
        e = float(np.max(np.abs(a - b)) / np.max(np.abs(b)))
        print(f"[noalloc] call {i}: dw err {e:.2e} dx equal {torch.equal(dx, rdx)}", flush=True)
        assert e <= (1e-5 if dtype == "f32" else 2e-2)
        assert torch.equal(dx, rdx) and torch.equal(dw, rdw)


def test_noalloc_rejects_oversized_problem():
    # the partial rows of this problem exceed the fixed scratch: a clear error, nothing launched
    L = _lib.lib()
    f = L.o1d_bwd_noalloc
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_void_p] * 6 + [ctypes.c_int] * 6 + [ctypes.c_void_p]
    p = [ctypes.c_void_p(a) for a in (0x10000, 0x90000000, 0x100000000, 0x200000000, 0x300000000, 0x400000000)]
    st = f(*p, 64, 65535, 8, 8, 127, _lib.O1D_F32, None)
    assert st == 2  # O1D_ERR_UNSUPPORTED
    assert "scratch" in L.o1d_last_error().decode()
