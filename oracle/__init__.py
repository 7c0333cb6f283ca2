"""Reference oracle for oriented 1D depthwise convolution (CPU, float64).

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
benchmark's CPU-baseline leg may import this package.  The library's product
path never loads it; it shares no code with the HIP kernels.

The arithmetic lives in ``o1d_oracle.c`` (plain C loops, double precision,
scatter-form backward) and follows Definition 1 / Eq. (1)-(2) of Kirchmeyer &
Deng, "Convolutional Networks with Oriented 1D Kernels", with pad = K // 2
placed inside the floor as the appendix section "Padding" requires.  This
module only compiles it with gcc and marshals numpy arrays through ctypes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "o1d_oracle.c")
_LIB = os.path.join(_HERE, "libo1d_oracle.so")
_lib = None

_D = ctypes.POINTER(ctypes.c_double)
_I = ctypes.POINTER(ctypes.c_int)


def build(force: bool = True) -> str:
    """Compile the C oracle into ``oracle/libo1d_oracle.so`` with gcc."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-D_GNU_SOURCE",
               "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        lib.oracle_offsets_real.argtypes = [ctypes.c_double, ctypes.c_int, ctypes.c_int, _D, _D]
        lib.oracle_offsets_real.restype = None
        lib.oracle_offsets.argtypes = [ctypes.c_double, ctypes.c_int, ctypes.c_int, _I, _I]
        lib.oracle_offsets.restype = None
        for name in ("oracle_fwd", "oracle_bwd_input", "oracle_bwd_weight"):
            f = getattr(lib, name)
            f.argtypes = [_D, _D, _D, _D] + [ctypes.c_int] * 6
            f.restype = None
        for name in ("oracle_fwd_ex", "oracle_bwd_input_ex", "oracle_bwd_weight_ex"):
            f = getattr(lib, name)
            f.argtypes = [_D, _D, _D, _D] + [ctypes.c_int] * 8
            f.restype = None
        lib.oracle_tap_samples.argtypes = [ctypes.c_double, ctypes.c_int, ctypes.c_int, _I, _I, _D]
        lib.oracle_tap_samples.restype = None
        _lib = lib
    return _lib


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a: np.ndarray, t=_D):
    return a.ctypes.data_as(t)


def default_threads() -> int:
    return max(1, len(os.sched_getaffinity(0)))


def offsets_real(theta_deg: float, K: int, pad: int | None = None):
    """Unrounded filter offsets (dh, dw) = R_theta (0, k - pad)^T for k < K."""
    lib = _load()
    pad = K // 2 if pad is None else pad
    vh = np.zeros(K, np.float64)
    vw = np.zeros(K, np.float64)
    lib.oracle_offsets_real(float(theta_deg), K, pad, _ptr(vh), _ptr(vw))
    return vh, vw


def offsets(theta_deg: float, K: int, pad: int | None = None):
    """Integer filter offsets floor(R_theta (0, k - pad)^T) (Eq. 2)."""
    lib = _load()
    pad = K // 2 if pad is None else pad
    dh = np.zeros(K, np.int32)
    dw = np.zeros(K, np.int32)
    lib.oracle_offsets(float(theta_deg), K, pad, _ptr(dh, _I), _ptr(dw, _I))
    return dh, dw


def _check(x, K, C):
    if x.ndim != 4:
        raise ValueError("expected an NCHW array")
    if K < 1 or K % 2 == 0:
        raise ValueError("K must be odd and positive")


MODES = {"floor": 0, "bilinear": 1}


def out_size(n: int, stride: int) -> int:
    """Output length along one axis for a centred odd kernel: floor((n - 1) / stride) + 1."""
    return (n - 1) // stride + 1


def _plain(stride: int, mode: str) -> bool:
    if stride < 1:
        raise ValueError("stride must be >= 1")
    if mode not in MODES:
        raise ValueError(f"unknown mode {mode!r}")
    return stride == 1 and mode == "floor"


def tap_samples(theta_deg: float, K: int, mode: str = "floor"):
    """Per tap, four (row offset, column offset, coefficient) samples: rounding down uses one with
    coefficient 1, bilinear interpolation the four surrounding pixels."""
    sh = np.zeros(4 * K, np.int32)
    sw = np.zeros(4 * K, np.int32)
    sc = np.zeros(4 * K, np.float64)
    _load().oracle_tap_samples(float(theta_deg), K, MODES[mode], _ptr(sh, _I), _ptr(sw, _I), _ptr(sc))
    return sh.reshape(K, 4), sw.reshape(K, 4), sc.reshape(K, 4)


def fwd(x, w, theta_deg, threads: int | None = None, stride: int = 1, mode: str = "floor") -> np.ndarray:
    """y = oriented depthwise 1D convolution of x (N,C,H,W) with w (C,K); y is (N,C,P,Q)."""
    x = _f64(x); w = _f64(w); th = _f64(theta_deg)
    N, C, H, W = x.shape
    K = w.shape[1]
    _check(x, K, C)
    lib, t = _load(), threads or default_threads()
    if _plain(stride, mode):
        y = np.empty_like(x)
        lib.oracle_fwd(_ptr(x), _ptr(w), _ptr(th), _ptr(y), N, C, H, W, K, t)
        return y
    y = np.empty((N, C, out_size(H, stride), out_size(W, stride)), np.float64)
    lib.oracle_fwd_ex(_ptr(x), _ptr(w), _ptr(th), _ptr(y), N, C, H, W, K, stride, MODES[mode], t)
    return y


def bwd_input(dy, w, theta_deg, threads: int | None = None, stride: int = 1, mode: str = "floor",
              in_hw: tuple[int, int] | None = None) -> np.ndarray:
    """dL/dx (N,C,H,W) given dL/dy (N,C,P,Q) (scatter form of the adjoint of Eq. 1).  With stride > 1 the
    input size (H, W) is not implied by (P, Q) and must be given as in_hw."""
    dy = _f64(dy); w = _f64(w); th = _f64(theta_deg)
    N, C, P, Q = dy.shape
    K = w.shape[1]
    _check(dy, K, C)
    lib, t = _load(), threads or default_threads()
    if _plain(stride, mode) and in_hw in (None, (P, Q)):
        dx = np.empty_like(dy)
        lib.oracle_bwd_input(_ptr(dy), _ptr(w), _ptr(th), _ptr(dx), N, C, P, Q, K, t)
        return dx
    H, W = (P, Q) if in_hw is None else in_hw
    if (out_size(H, stride), out_size(W, stride)) != (P, Q):
        raise ValueError(f"dy {P}x{Q} is not the stride-{stride} output of a {H}x{W} input")
    dx = np.empty((N, C, H, W), np.float64)
    lib.oracle_bwd_input_ex(_ptr(dy), _ptr(w), _ptr(th), _ptr(dx), N, C, H, W, K, stride, MODES[mode], t)
    return dx


def bwd_weight(x, dy, theta_deg, K: int, threads: int | None = None, stride: int = 1,
               mode: str = "floor") -> np.ndarray:
    """dL/dw (C,K) given the input x (N,C,H,W) and dL/dy (N,C,P,Q) (scatter form of the adjoint of Eq. 1)."""
    x = _f64(x); dy = _f64(dy); th = _f64(theta_deg)
    N, C, H, W = x.shape
    _check(x, K, C)
    if dy.shape != (N, C, out_size(H, stride), out_size(W, stride)):
        raise ValueError(f"dy {dy.shape} does not match x {x.shape} at stride {stride}")
    lib, t = _load(), threads or default_threads()
    dw = np.empty((C, K), np.float64)
    if _plain(stride, mode):
        lib.oracle_bwd_weight(_ptr(x), _ptr(dy), _ptr(th), _ptr(dw), N, C, H, W, K, t)
    else:
        lib.oracle_bwd_weight_ex(_ptr(x), _ptr(dy), _ptr(th), _ptr(dw), N, C, H, W, K, stride, MODES[mode], t)
    return dw


# ---------------------------------------------------------------- depthwise separable block

def dsc_fwd(x, w_dw, theta_deg, w_pw, threads: int | None = None) -> tuple[np.ndarray, np.ndarray]:
    """Oriented 1D depthwise separable convolution (Sec. 3.2, "Computational cost analysis", and Table 1's
    "Oriented 1D DSC" row): the oriented depthwise convolution z = fwd(x, w_dw, theta) followed by the
    pointwise (1 x 1) convolution y[n,o] = sum_c w_pw[o,c] z[n,c] that mixes C channels into C' = w_pw.shape[0].
    Returns (z, y)."""
    w_pw = _f64(w_pw)
    z = fwd(x, w_dw, theta_deg, threads)
    if w_pw.ndim != 2 or w_pw.shape[1] != z.shape[1]:
        raise ValueError(f"w_pw {w_pw.shape} must be (C', C) with C = {z.shape[1]}")
    y = np.tensordot(w_pw, z, axes=([1], [1])).transpose(1, 0, 2, 3)  # (C', N, H, W) -> (N, C', H, W)
    return z, np.ascontiguousarray(y)


def dsc_bwd(x, dy, w_dw, theta_deg, w_pw, threads: int | None = None):
    """Gradients of the block: with z the depthwise output, dz[n,c] = sum_o w_pw[o,c] dy[n,o],
    dw_pw[o,c] = sum_{n,h,w} dy[n,o,h,w] z[n,c,h,w], and (dx, dw_dw) the depthwise convolution's gradients
    for dz.  Returns (dx, dw_dw, dw_pw)."""
    w_pw = _f64(w_pw); dy = _f64(dy)
    K = np.asarray(w_dw).shape[1]
    z = fwd(x, w_dw, theta_deg, threads)
    dz = np.ascontiguousarray(np.tensordot(w_pw, dy, axes=([0], [1])).transpose(1, 0, 2, 3))
    dw_pw = np.tensordot(dy, z, axes=([0, 2, 3], [0, 2, 3]))
    dx = bwd_input(dz, w_dw, theta_deg, threads)
    dw_dw = bwd_weight(x, dz, theta_deg, K, threads)
    return dx, dw_dw, dw_pw
