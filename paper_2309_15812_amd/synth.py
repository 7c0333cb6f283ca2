"""Seeded synthetic inputs for the oriented 1D depthwise convolution.

This module only draws random numbers; it contains none of the operation's
arithmetic.  Both the oracle and the GPU path consume what it returns, so
it is the single source of inputs for tests, the smoke check and the
benchmark.

The paper benchmarks the operation on ConvNeXt feature maps (N = 64 and
per-stage channel counts at 56x56 / 28x28 / 14x14 resolution, Table 1 and the
"speed" tables of the appendix); seeded Gaussian tensors of those shapes stand
in for the ImageNet activations it used.  Angles follow the paper's practice
of D equally spaced directions i * 180 / D degrees (Section 3.1), or are drawn
uniformly in [0, 180) for the "any angle" cases.

Distributions: x, dy ~ N(0, 1); w ~ N(0, 1/K); theta in float32 degrees.
bfloat16 tensors are the round-to-nearest-even images of those float32 draws.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

BASE_SEED = 20230915


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    N: int
    C: int
    H: int
    W: int
    K: int
    dtype: str = "f32"        # "f32" or "bf16"
    theta: str = "discrete8"  # "ramp", "discrete8", "uniform", "zero", "ninety", "groups:D"
    ops: str = "fwd+bwd"      # "fwd" or "fwd+bwd"
    seed_index: int = 0

    @property
    def elems(self) -> int:
        return self.N * self.C * self.H * self.W

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five configurations the operation is measured and checked on.
WORKLOADS = {
    # Forward only, small: theta_c = 22.5 * c degrees, c < 8.
    "c1": Workload("c1", 1, 8, 32, 32, 7, "f32", "ramp", "fwd", 0),
    # ConvNeXt-T stage-1 shape, forward.
    "c2": Workload("c2", 64, 96, 56, 56, 31, "f32", "discrete8", "fwd", 1),
    # Stage-2 shape, forward + both gradients.
    "c3": Workload("c3", 64, 192, 28, 28, 31, "f32", "discrete8", "fwd+bwd", 2),
    # Stage-3 shape, bfloat16 storage, continuous angles.
    "c4": Workload("c4", 64, 384, 14, 14, 31, "bf16", "uniform", "fwd+bwd", 3),
    # Angle-cost sweep shape (K and theta mode vary).
    "c5": Workload("c5", 32, 256, 56, 56, 31, "f32", "uniform", "fwd+bwd", 4),
    # The headline measurement: stage-1 shape, forward + both gradients.
    "metric": Workload("metric", 64, 96, 56, 56, 31, "f32", "discrete8", "fwd+bwd", 1),
    # The depthwise separable block of Table 1 (C' = C = 512), four angle groups.
    "dsc": Workload("dsc", 64, 512, 56, 56, 31, "f32", "groups:4", "fwd+bwd", 5),
}


def draw_theta(mode: str, C: int, rng: np.random.Generator) -> np.ndarray:
    """Per-channel angles in float32 degrees."""
    if mode == "ramp":
        th = 22.5 * np.arange(C)
    elif mode == "discrete8":
        th = 22.5 * rng.integers(0, 8, size=C)
    elif mode == "uniform":
        th = rng.uniform(0.0, 180.0, size=C)
    elif mode == "zero":
        th = np.zeros(C)
    elif mode == "ninety":
        th = np.full(C, 90.0)
    elif mode.startswith("groups:"):
        # Section 3.1: D equal channel groups, group i at i * 180 / D degrees.
        D = int(mode.split(":")[1])
        th = (np.arange(C) * D // C) * (180.0 / D)
    else:
        raise ValueError(f"unknown theta mode {mode!r}")
    return th.astype(np.float32)


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even, via torch on the CPU."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> exact float32 values."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def make_inputs(wl: Workload, seed: Optional[int] = None, planes: Optional[int] = None) -> dict:
    """Draw x, dy, w, theta for a workload.

    Returns float32 numpy arrays 'x', 'dy' (N,C,H,W), 'w' (C,K), 'theta' (C,);
    for bf16 workloads 'x', 'dy', 'w' already hold the bfloat16-rounded values
    (as float32) and '*_bits' hold the uint16 patterns.  `planes` limits N
    (a leading slice of the batch) for bounded CPU work.
    """
    rng = np.random.default_rng(BASE_SEED + wl.seed_index if seed is None else seed)
    N = wl.N if planes is None else min(wl.N, planes)
    theta = draw_theta(wl.theta, wl.C, rng)
    w = (rng.standard_normal((wl.C, wl.K)) / np.sqrt(wl.K)).astype(np.float32)
    x = rng.standard_normal((N, wl.C, wl.H, wl.W), dtype=np.float32)
    dy = rng.standard_normal((N, wl.C, wl.H, wl.W), dtype=np.float32)
    out = {"x": x, "dy": dy, "w": w, "theta": theta}
    if wl.dtype == "bf16":
        for k in ("x", "dy", "w"):
            bits = to_bf16_bits(out[k])
            out[k + "_bits"] = bits
            out[k] = bf16_bits_to_f32(bits)
    return out


def make_pointwise(wl: Workload, cout: int, seed: Optional[int] = None, planes: Optional[int] = None) -> dict:
    """Draw the depthwise separable block's extra tensors: pointwise weights 'w_pw' (cout, C) ~ N(0, 1/C) and
    the block's upstream gradient 'dy_pw' (N, cout, H, W) ~ N(0, 1), float32 (bfloat16-rounded values and
    '*_bits' for bf16 workloads, as make_inputs)."""
    rng = np.random.default_rng(BASE_SEED + 1000 + wl.seed_index if seed is None else seed)
    N = wl.N if planes is None else min(wl.N, planes)
    out = {"w_pw": (rng.standard_normal((cout, wl.C)) / np.sqrt(wl.C)).astype(np.float32),
           "dy_pw": rng.standard_normal((N, cout, wl.H, wl.W), dtype=np.float32)}
    if wl.dtype == "bf16":
        for k in ("w_pw", "dy_pw"):
            bits = to_bf16_bits(out[k])
            out[k + "_bits"] = bits
            out[k] = bf16_bits_to_f32(bits)
    return out
