"""torch-facing wrappers of the C ABI: tensors in, tensors out.

PyTorch supplies device memory and the current stream; the three entry points
below only check shapes, allocate outputs and hand raw pointers to
libo1d.so.  theta is a float32 tensor of per-channel angles in degrees.
"""
from __future__ import annotations

import torch

from . import _lib

_DT = {torch.float32: _lib.O1D_F32, torch.bfloat16: _lib.O1D_BF16}


def _stream(t: torch.Tensor) -> int:
    return torch.cuda.current_stream(t.device).cuda_stream


def _dt(t: torch.Tensor) -> int:
    if t.dtype not in _DT:
        raise TypeError(f"unsupported dtype {t.dtype}; use float32 or bfloat16")
    return _DT[t.dtype]


def _check_common(x: torch.Tensor, w: torch.Tensor, theta: torch.Tensor):
    if x.dim() != 4 or w.dim() != 2:
        raise ValueError("expected x as (N, C, H, W) and w as (C, K)")
    N, C, H, W = x.shape
    if w.shape[0] != C or theta.shape != (C,):
        raise ValueError(f"w {tuple(w.shape)} / theta {tuple(theta.shape)} do not match C={C}")
    if w.dtype != x.dtype:
        raise TypeError("x and w must share a dtype")
    if theta.dtype != torch.float32:
        raise TypeError("theta must be float32 degrees")
    for t in (x, w, theta):
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError("tensors must be contiguous and on the GPU")
    return N, C, H, W, int(w.shape[1])


def _out(out: torch.Tensor | None, like: torch.Tensor, shape=None) -> torch.Tensor:
    """A caller-given output must match what the kernels write (they take no strides or sizes of it)."""
    shape = tuple(like.shape) if shape is None else tuple(shape)
    if out is None:
        return torch.empty(shape, dtype=like.dtype, device=like.device)
    if tuple(out.shape) != shape or out.dtype != like.dtype or out.device != like.device or not out.is_contiguous():
        raise ValueError(f"output {tuple(out.shape)} {out.dtype} {out.device} must be a contiguous {shape} "
                         f"{like.dtype} tensor on {like.device}")
    return out


def fwd(x: torch.Tensor, w: torch.Tensor, theta: torch.Tensor, out: torch.Tensor | None = None) -> torch.Tensor:
    """y = oriented depthwise 1D convolution of x (Definition 1, Eq. 1-2)."""
    N, C, H, W, K = _check_common(x, w, theta)
    y = _out(out, x)
    _lib.check("o1d_fwd", _lib.call("o1d_fwd", x.data_ptr(), w.data_ptr(), theta.data_ptr(), y.data_ptr(),
                                    N, C, H, W, K, _dt(x), _stream(x)))
    return y


def bwd_input(dy: torch.Tensor, w: torch.Tensor, theta: torch.Tensor, out: torch.Tensor | None = None) -> torch.Tensor:
    """dx given dy (adjoint of Eq. 1 in x)."""
    N, C, H, W, K = _check_common(dy, w, theta)
    dx = _out(out, dy)
    _lib.check("o1d_bwd_input", _lib.call("o1d_bwd_input", dy.data_ptr(), w.data_ptr(), theta.data_ptr(),
                                          dx.data_ptr(), N, C, H, W, K, _dt(dy), _stream(dy)))
    return dx


def workspace_bytes(N: int, C: int, H: int, W: int, K: int, dtype: torch.dtype) -> int:
    return int(_lib.lib().o1d_bwd_weight_workspace_bytes(N, C, H, W, K, _DT[dtype]))


def _workspace(workspace: torch.Tensor | None, like: torch.Tensor, need: int) -> tuple[torch.Tensor, int]:
    """A caller-given workspace must be device memory the kernels may write: a contiguous tensor on like's GPU
    holding at least `need` bytes."""
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=like.device)
    if not workspace.is_cuda or workspace.device != like.device or not workspace.is_contiguous():
        raise ValueError(f"workspace must be a contiguous tensor on {like.device}, got {workspace.device} "
                         f"(contiguous={workspace.is_contiguous()})")
    nbytes = workspace.numel() * workspace.element_size()
    if nbytes < need:
        raise ValueError(f"workspace holds {nbytes} bytes, {need} needed")
    return workspace, nbytes


def bwd_weight(x: torch.Tensor, dy: torch.Tensor, theta: torch.Tensor, K: int, out: torch.Tensor | None = None,
               workspace: torch.Tensor | None = None) -> torch.Tensor:
    """dw (C, K) given x and dy (adjoint of Eq. 1 in w)."""
    if dy.shape != x.shape or dy.dtype != x.dtype:
        raise ValueError("x and dy must have the same shape and dtype")
    N, C, H, W = x.shape
    dw = _out(out, x, (C, K))
    _check_common(x, dw, theta)
    if not dy.is_cuda or not dy.is_contiguous():
        raise ValueError("tensors must be contiguous and on the GPU")
    workspace, nbytes = _workspace(workspace, x, workspace_bytes(N, C, H, W, K, x.dtype))
    _lib.check("o1d_bwd_weight", _lib.call("o1d_bwd_weight", x.data_ptr(), dy.data_ptr(), theta.data_ptr(),
                                           dw.data_ptr(), N, C, H, W, K, _dt(x), workspace.data_ptr(), nbytes,
                                           _stream(x)))
    return dw


def bwd(x: torch.Tensor, dy: torch.Tensor, w: torch.Tensor, theta: torch.Tensor,
        out: tuple[torch.Tensor, torch.Tensor] | None = None,
        workspace: torch.Tensor | None = None) -> tuple[torch.Tensor, torch.Tensor]:
    """(dx, dw) given x and dy: both adjoints of Eq. 1 in one call."""
    if dy.shape != x.shape or dy.dtype != x.dtype:
        raise ValueError("x and dy must have the same shape and dtype")
    N, C, H, W, K = _check_common(x, w, theta)
    if not dy.is_cuda or not dy.is_contiguous():
        raise ValueError("tensors must be contiguous and on the GPU")
    dx, dw = (_out(None, x), _out(None, w)) if out is None else (_out(out[0], x), _out(out[1], w))
    workspace, nbytes = _workspace(workspace, x, workspace_bytes(N, C, H, W, K, x.dtype))
    _lib.check("o1d_bwd", _lib.call("o1d_bwd", x.data_ptr(), dy.data_ptr(), w.data_ptr(), theta.data_ptr(),
                                    dx.data_ptr(), dw.data_ptr(), N, C, H, W, K, _dt(x), workspace.data_ptr(),
                                    nbytes, _stream(x)))
    return dx, dw


# ---------------------------------------------------------------- stride, layout, sampling

_LAYOUT = {"nchw": _lib.O1D_NCHW, "nhwc": _lib.O1D_NHWC}
_SAMPLING = {"floor": _lib.O1D_FLOOR, "bilinear": _lib.O1D_BILINEAR}


def out_size(n: int, stride: int) -> int:
    """Output length along one axis: floor((n - 1) / stride) + 1."""
    return (n - 1) // stride + 1


def _ex_args(x: torch.Tensor, w: torch.Tensor, theta: torch.Tensor, layout: str, sampling: str):
    if layout not in _LAYOUT or sampling not in _SAMPLING:
        raise ValueError(f"layout must be one of {list(_LAYOUT)}, sampling one of {list(_SAMPLING)}")
    if x.dim() != 4 or w.dim() != 2:
        raise ValueError("expected a 4-d x and w as (C, K)")
    if layout == "nchw":
        N, C, H, W = x.shape
    else:
        N, H, W, C = x.shape
    if w.shape[0] != C or theta.shape != (C,):
        raise ValueError(f"w {tuple(w.shape)} / theta {tuple(theta.shape)} do not match C={C}")
    if w.dtype != x.dtype:
        raise TypeError("x and w must share a dtype")
    if theta.dtype != torch.float32:
        raise TypeError("theta must be float32 degrees")
    for t in (x, w, theta):
        if not t.is_cuda or not t.is_contiguous() or t.device != x.device:
            raise ValueError("tensors must be contiguous and on one GPU")
    return N, C, H, W, int(w.shape[1])


def _shape(layout: str, N: int, C: int, H: int, W: int) -> tuple:
    return (N, C, H, W) if layout == "nchw" else (N, H, W, C)


def fwd_ex(x: torch.Tensor, w: torch.Tensor, theta: torch.Tensor, stride: int = 1, layout: str = "nchw",
           sampling: str = "floor", out: torch.Tensor | None = None) -> torch.Tensor:
    """Forward pass with stride, NCHW / NHWC layout and rounded-down or bilinear sampling."""
    N, C, H, W, K = _ex_args(x, w, theta, layout, sampling)
    y = _out(out, x, _shape(layout, N, C, out_size(H, stride), out_size(W, stride)))
    _lib.check("o1d_fwd_ex", _lib.call("o1d_fwd_ex", x.data_ptr(), w.data_ptr(), theta.data_ptr(), y.data_ptr(),
                                       N, C, H, W, K, stride, _LAYOUT[layout], _SAMPLING[sampling], _dt(x),
                                       _stream(x)))
    return y


def bwd_input_ex(dy: torch.Tensor, w: torch.Tensor, theta: torch.Tensor, in_hw: tuple[int, int], stride: int = 1,
                 layout: str = "nchw", sampling: str = "floor", out: torch.Tensor | None = None) -> torch.Tensor:
    """dx (input plane in_hw = (H, W)) given dy of the stride-`stride` output plane."""
    N, C, P, Q, K = _ex_args(dy, w, theta, layout, sampling)
    H, W = in_hw
    if (out_size(H, stride), out_size(W, stride)) != (P, Q):
        raise ValueError(f"dy plane {P}x{Q} is not the stride-{stride} output of {H}x{W}")
    dx = _out(out, dy, _shape(layout, N, C, H, W))
    _lib.check("o1d_bwd_input_ex", _lib.call("o1d_bwd_input_ex", dy.data_ptr(), w.data_ptr(), theta.data_ptr(),
                                             dx.data_ptr(), N, C, H, W, K, stride, _LAYOUT[layout],
                                             _SAMPLING[sampling], _dt(dy), _stream(dy)))
    return dx


def workspace_bytes_ex(N: int, C: int, H: int, W: int, K: int, dtype: torch.dtype, stride: int = 1,
                       layout: str = "nchw", sampling: str = "floor") -> int:
    return int(_lib.lib().o1d_bwd_weight_ex_workspace_bytes(N, C, H, W, K, stride, _LAYOUT[layout],
                                                            _SAMPLING[sampling], _DT[dtype]))


def bwd_weight_ex(x: torch.Tensor, dy: torch.Tensor, theta: torch.Tensor, K: int, stride: int = 1,
                  layout: str = "nchw", sampling: str = "floor", out: torch.Tensor | None = None,
                  workspace: torch.Tensor | None = None) -> torch.Tensor:
    """dw (C, K) given x and dy of the stride-`stride` output plane."""
    if layout not in _LAYOUT or sampling not in _SAMPLING:
        raise ValueError(f"layout must be one of {list(_LAYOUT)}, sampling one of {list(_SAMPLING)}")
    N, H, W, C = (x.shape[0], x.shape[1], x.shape[2], x.shape[3]) if layout == "nhwc" else \
        (x.shape[0], x.shape[2], x.shape[3], x.shape[1])
    if tuple(dy.shape) != _shape(layout, N, C, out_size(H, stride), out_size(W, stride)) or dy.dtype != x.dtype:
        raise ValueError(f"dy {tuple(dy.shape)} does not match x {tuple(x.shape)} at stride {stride}")
    dw = _out(out, x, (C, K))
    _ex_args(x, dw, theta, layout, sampling)
    if not dy.is_cuda or not dy.is_contiguous() or dy.device != x.device:
        raise ValueError("tensors must be contiguous and on one GPU")
    workspace, nbytes = _workspace(workspace, x, workspace_bytes_ex(N, C, H, W, K, x.dtype, stride, layout, sampling))
    _lib.check("o1d_bwd_weight_ex", _lib.call("o1d_bwd_weight_ex", x.data_ptr(), dy.data_ptr(), theta.data_ptr(),
                                              dw.data_ptr(), N, C, H, W, K, stride, _LAYOUT[layout],
                                              _SAMPLING[sampling], _dt(x), workspace.data_ptr(), nbytes,
                                              _stream(x)))
    return dw


class OrientedConv1dFunction(torch.autograd.Function):
    """Autograd glue: forward -> o1d_fwd, backward -> o1d_bwd (or one of its halves); theta gets no gradient."""

    @staticmethod
    def forward(ctx, x, w, theta):
        # the kernels take dense tensors: save the dense copies that the forward used
        x, w, theta = x.contiguous(), w.contiguous(), theta.contiguous()
        ctx.save_for_backward(x, w, theta)
        return fwd(x, w, theta)

    @staticmethod
    def backward(ctx, gy):
        x, w, theta = ctx.saved_tensors
        gy = gy.contiguous()
        if ctx.needs_input_grad[0] and ctx.needs_input_grad[1]:
            gx, gw = bwd(x, gy, w, theta)
            return gx, gw, None
        gx = bwd_input(gy, w, theta) if ctx.needs_input_grad[0] else None
        gw = bwd_weight(x, gy, theta, w.shape[1]) if ctx.needs_input_grad[1] else None
        return gx, gw, None


# ---------------------------------------------------------------- depthwise separable block

def _check_pw(w_pw: torch.Tensor, like: torch.Tensor, C: int) -> int:
    if w_pw.dim() != 2 or w_pw.shape[1] != C or w_pw.dtype != like.dtype:
        raise ValueError(f"w_pw must be (C', {C}) of dtype {like.dtype}, got {tuple(w_pw.shape)} {w_pw.dtype}")
    if not w_pw.is_cuda or not w_pw.is_contiguous():
        raise ValueError("tensors must be contiguous and on the GPU")
    return int(w_pw.shape[0])


def dsc_fwd(x: torch.Tensor, w_dw: torch.Tensor, theta: torch.Tensor, w_pw: torch.Tensor,
            out: tuple[torch.Tensor, torch.Tensor] | None = None) -> tuple[torch.Tensor, torch.Tensor]:
    """(z, y): z the oriented depthwise convolution of x, y = w_pw mixing z's channels (Sec. 3.2, Table 1)."""
    N, C, H, W, K = _check_common(x, w_dw, theta)
    Co = _check_pw(w_pw, x, C)
    z, y = (_out(None, x), _out(None, x, (N, Co, H, W))) if out is None else \
        (_out(out[0], x), _out(out[1], x, (N, Co, H, W)))
    _lib.check("o1d_dsc_fwd", _lib.call("o1d_dsc_fwd", x.data_ptr(), w_dw.data_ptr(), theta.data_ptr(),
                                        w_pw.data_ptr(), z.data_ptr(), y.data_ptr(), N, C, Co, H, W, K, _dt(x),
                                        _stream(x)))
    return z, y


def dsc_workspace_bytes(N: int, C: int, Co: int, H: int, W: int, K: int, dtype: torch.dtype) -> int:
    return int(_lib.lib().o1d_dsc_bwd_workspace_bytes(N, C, Co, H, W, K, _DT[dtype]))


def dsc_bwd(x: torch.Tensor, z: torch.Tensor, dy: torch.Tensor, w_dw: torch.Tensor, theta: torch.Tensor,
            w_pw: torch.Tensor, out: tuple[torch.Tensor, torch.Tensor, torch.Tensor] | None = None,
            workspace: torch.Tensor | None = None) -> tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """(dx, dw_dw, dw_pw) of the block given x, the forward's z and dy."""
    N, C, H, W, K = _check_common(x, w_dw, theta)
    Co = _check_pw(w_pw, x, C)
    if z.shape != x.shape or z.dtype != x.dtype or dy.shape != (N, Co, H, W) or dy.dtype != x.dtype:
        raise ValueError("z must match x, dy must be (N, C', H, W) of x's dtype")
    for t in (z, dy):
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError("tensors must be contiguous and on the GPU")
    if out is None:
        dx, dwd, dwp = _out(None, x), _out(None, w_dw), _out(None, w_pw)
    else:
        dx, dwd, dwp = _out(out[0], x), _out(out[1], w_dw), _out(out[2], w_pw)
    workspace, nbytes = _workspace(workspace, x, dsc_workspace_bytes(N, C, Co, H, W, K, x.dtype))
    _lib.check("o1d_dsc_bwd", _lib.call("o1d_dsc_bwd", x.data_ptr(), z.data_ptr(), dy.data_ptr(), w_dw.data_ptr(),
                                        theta.data_ptr(), w_pw.data_ptr(), dx.data_ptr(), dwd.data_ptr(),
                                        dwp.data_ptr(), N, C, Co, H, W, K, _dt(x), workspace.data_ptr(), nbytes,
                                        _stream(x)))
    return dx, dwd, dwp
