"""MI355X (gfx950) implementation of depthwise convolution with oriented 1D kernels.

Kirchmeyer & Deng, "Convolutional Networks with Oriented 1D Kernels" (ICCV 2023),
Definition 1: every channel c convolves its H x W plane with a length-K 1D
kernel laid along angle theta_c, sampling pixels at the floored rotated offsets
of Eq. (2), with zero padding.  Forward pass, input gradient and weight gradient
run in hand-written HIP kernels behind the C ABI of include/o1d.h.

    from paper_2309_15812_amd import ops
    y = ops.fwd(x, w, theta)            # x: (N,C,H,W) float32/bfloat16 on the GPU
    dx = ops.bwd_input(dy, w, theta)
    dw = ops.bwd_weight(x, dy, theta, K)
"""

__all__ = ["ops", "synth", "build"]
