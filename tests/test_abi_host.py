"""Host-only checks of the C ABI (no GPU needed).

The library must load, export every function include/o1d.h declares, and
reject invalid arguments with the documented status before touching the GPU.
"""
import ctypes
import os
import re

import pytest

from paper_2309_15812_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "o1d.h")

OK, INVALID, UNSUPPORTED, WORKSPACE = 0, 1, 2, 3
F32, BF16 = 0, 1
# a fake non-NULL device address; every call below fails validation before any use
P = ctypes.c_void_p(0x10000)
Q = ctypes.c_void_p(0x90000000)
R = ctypes.c_void_p(0x100000000)


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(o1d_[a-z_]+)\s*\(", text)))


def test_header_declares_the_abi():
    names = declared_functions()
    assert {"o1d_fwd", "o1d_bwd_input", "o1d_bwd_weight", "o1d_bwd", "o1d_bwd_weight_workspace_bytes",
            "o1d_status_str", "o1d_last_error", "o1d_version"} <= set(names)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(_lib.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert set(declared_functions()) == set(_lib.SIGNATURES)


def test_version_and_status_strings():
    L = _lib.lib()
    assert b"gfx950" in L.o1d_version()
    for st, nm in _lib.STATUS.items():
        assert L.o1d_status_str(st).decode().startswith(nm)


def fwd(*, x=P, w=Q, th=R, y=ctypes.c_void_p(0x200000000), N=2, C=3, H=5, W=6, K=7, dt=F32):
    return _lib.call("o1d_fwd", x, w, th, y, N, C, H, W, K, dt, None)


@pytest.mark.parametrize("kw,status", [
    (dict(K=4), INVALID), (dict(K=0), INVALID), (dict(K=-3), INVALID),
    (dict(N=-1), INVALID), (dict(H=-2), INVALID), (dict(dt=7), INVALID),
    (dict(x=None), INVALID), (dict(w=None), INVALID), (dict(th=None), INVALID), (dict(y=None), INVALID),
    (dict(y=P), INVALID),                         # output aliases input
    (dict(K=_lib.MAX_K + 2), UNSUPPORTED), (dict(C=70000), UNSUPPORTED), (dict(N=70000), UNSUPPORTED),
    (dict(H=1 << 16, W=1 << 16), UNSUPPORTED),
])
def test_forward_rejects(kw, status):
    assert fwd(**kw) == status
    assert _lib.lib().o1d_last_error().decode().startswith("o1d_fwd")
    assert _lib.call("o1d_bwd_input", kw.get("x", P), kw.get("w", Q), kw.get("th", R),
                     kw.get("y", ctypes.c_void_p(0x200000000)), kw.get("N", 2), kw.get("C", 3), kw.get("H", 5),
                     kw.get("W", 6), kw.get("K", 7), kw.get("dt", F32), None) == status


def test_empty_forward_is_a_noop():
    # nothing to compute: no pointer is touched and no device work is enqueued
    assert fwd(N=0, x=None, y=None) == OK
    assert fwd(C=0, x=None, w=None, th=None, y=None) == OK
    assert fwd(H=0, W=9) == OK


def test_workspace_size_and_rejection():
    L = _lib.lib()
    need = L.o1d_bwd_weight_workspace_bytes(64, 96, 56, 56, 31, F32)
    assert need > 0 and need % (96 * 31 * 4) == 0
    assert need == L.o1d_bwd_weight_workspace_bytes(64, 96, 56, 56, 31, F32)  # deterministic
    assert L.o1d_bwd_weight_workspace_bytes(64, 96, 56, 56, 30, F32) == 0     # invalid K -> 0
    st = _lib.call("o1d_bwd_weight", P, Q, R, ctypes.c_void_p(0x300000000), 64, 96, 56, 56, 31, F32,
                   ctypes.c_void_p(0x400000000), need - 4, None)
    assert st == WORKSPACE
    st = _lib.call("o1d_bwd_weight", P, Q, R, ctypes.c_void_p(0x300000000), 64, 96, 56, 56, 31, F32, None, need,
                   None)
    assert st == WORKSPACE
    st = _lib.call("o1d_bwd_weight", P, Q, R, ctypes.c_void_p(0x300000000), 2, 3, 5, 6, 8, F32, None, 0, None)
    assert st == INVALID
    st = _lib.call("o1d_bwd_weight", P, Q, R, None, 2, 3, 5, 6, 7, F32, None, 0, None)
    assert st == INVALID


DX, DW, WS, WT = (ctypes.c_void_p(a) for a in (0x200000000, 0x300000000, 0x400000000, 0x500000000))


def bwd(*, x=P, dy=Q, w=WT, th=R, dx=DX, dw=DW, N=64, C=96, H=56, W=56, K=31, dt=F32, ws=WS, nbytes=None):
    if nbytes is None:
        nbytes = _lib.lib().o1d_bwd_weight_workspace_bytes(N, C, H, W, K, dt)
    return _lib.call("o1d_bwd", x, dy, w, th, dx, dw, N, C, H, W, K, dt, ws, nbytes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(K=30), INVALID), (dict(N=-1), INVALID), (dict(dt=5), INVALID),
    (dict(x=None), INVALID), (dict(dy=None), INVALID), (dict(w=None), INVALID), (dict(th=None), INVALID),
    (dict(dx=None), INVALID), (dict(dw=None), INVALID),
    (dict(dx=P), INVALID),                                          # dx aliases x
    (dict(dx=ctypes.c_void_p(0x90000000 + 4096)), INVALID),         # dx overlaps dy
    (dict(dw=ctypes.c_void_p(0x200000000 + 64)), INVALID),          # dw inside dx
    (dict(dw=WT), INVALID),                                         # dw aliases w
    (dict(ws=ctypes.c_void_p(0x200000000)), INVALID),               # workspace aliases dx
    (dict(ws=None), WORKSPACE), (dict(nbytes=16), WORKSPACE),
    (dict(K=_lib.MAX_K + 2), UNSUPPORTED), (dict(C=70000), UNSUPPORTED),
])
def test_fused_backward_rejects(kw, status):
    assert bwd(**kw) == status
    assert _lib.lib().o1d_last_error().decode().startswith("o1d_bwd")


def test_fused_backward_without_channels_is_a_noop():
    assert bwd(C=0, x=None, dy=None, w=None, th=None, dx=None, dw=None, ws=None, nbytes=0) == OK


def test_python_wrapper_refuses_cpu_tensors():
    import torch

    from paper_2309_15812_amd import ops

    x = torch.zeros(1, 2, 4, 4)
    with pytest.raises(ValueError):
        ops.fwd(x, torch.zeros(2, 3), torch.zeros(2))


def fwd_ex(*, stride=1, layout=0, sampling=0, K=7, N=2, C=3, H=5, W=6, x=P, y=ctypes.c_void_p(0x200000000)):
    return _lib.call("o1d_fwd_ex", x, Q, R, y, N, C, H, W, K, stride, layout, sampling, F32, None)


@pytest.mark.parametrize("kw,status", [
    (dict(stride=0), INVALID), (dict(stride=-2), INVALID), (dict(layout=2), INVALID), (dict(sampling=3), INVALID),
    (dict(K=8), INVALID), (dict(x=None), INVALID), (dict(y=P), INVALID),
    (dict(stride=65), UNSUPPORTED), (dict(K=_lib.MAX_K + 2), UNSUPPORTED),
])
def test_ex_entry_points_reject(kw, status):
    assert fwd_ex(**kw) == status
    assert _lib.lib().o1d_last_error().decode().startswith("o1d_fwd_ex")
    a = dict(stride=1, layout=0, sampling=0, K=7)
    a.update({k: v for k, v in kw.items() if k in a})
    st = _lib.call("o1d_bwd_input_ex", kw.get("x", P), Q, R, kw.get("y", ctypes.c_void_p(0x200000000)), 2, 3, 5, 6,
                   a["K"], a["stride"], a["layout"], a["sampling"], F32, None)
    assert st == status


def test_ex_empty_and_workspace():
    assert fwd_ex(N=0, x=None, y=None) == OK
    L = _lib.lib()
    need = L.o1d_bwd_weight_ex_workspace_bytes(2, 3, 40, 40, 15, 2, 1, 1, F32)
    assert need > 0 and need % (3 * 15 * 4) == 0
    st = _lib.call("o1d_bwd_weight_ex", P, Q, R, ctypes.c_void_p(0x300000000), 2, 3, 40, 40, 15, 2, 1, 1, F32,
                   ctypes.c_void_p(0x400000000), need - 4, None)
    assert st == WORKSPACE
    assert L.o1d_bwd_weight_ex_workspace_bytes(2, 3, 40, 40, 15, 0, 1, 1, F32) == 0  # invalid stride -> 0
