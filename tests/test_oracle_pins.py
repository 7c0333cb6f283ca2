"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

None of these tests re-types the oracle's formula.  Each compares the oracle
with something independent of it:
  * exact real-arithmetic offsets (60-digit decimal trig) for Eq. (2);
  * the worked example of the appendix section "Rotation vs Shearing";
  * torch's float64 conv2d (a library correlation) at 0 and 90 degrees and,
    through the rasterised K x K mask, at every angle;
  * central finite differences and adjoint identities for the gradients;
  * impulse responses, K = 1 and one-hot weights.
A plausible slip in the oracle (sign of sin, pad outside the floor, swapped
h/w, transposed weight layout, a dropped boundary check, a missing
duplicate-tap sum, a wrong adjoint index) fails at least one of them.
"""
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from exact_offsets import exact_offsets, min_distance_to_integer, sin_cos_deg

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
RNG = np.random.default_rng(1234)

ANGLES = sorted({7.5 * i for i in range(48)} | {-45.0, -90.0, 359.0, 360.0, 405.0, -157.5, 1e-3, 89.999, 12.34})


def rand(*shape):
    return RNG.standard_normal(shape)


# ---------------------------------------------------------------- offsets (Eq. 2)

@pytest.mark.parametrize("K", [1, 3, 7, 15, 31, 63])
def test_offsets_equal_exact_floor(K):
    for th in ANGLES:
        dh, dw = oracle.offsets(th, K)
        edh, edw = exact_offsets(th, K)
        assert list(dh) == edh, (th, K)
        assert list(dw) == edw, (th, K)


def test_snap_reading_only_differs_next_to_exact_integer_angles():
    # Pure real arithmetic and the 1e-9 reading agree except where a product is
    # within 1e-9 of an integer without being one (e.g. 0.001 degrees).
    for th in ANGLES:
        for K in (7, 31, 63):
            same = exact_offsets(th, K, snap=True) == exact_offsets(th, K, snap=False)
            assert same or min_distance_to_integer(th, K) <= 1e-9, (th, K)
    assert exact_offsets(1e-3, 3, snap=False)[1] == [-1, 0, 0]
    assert list(oracle.offsets(1e-3, 3)[1]) == exact_offsets(1e-3, 3)[1] == [-1, 0, 1]


def test_offsets_random_float32_angles():
    th32 = np.random.default_rng(7).uniform(-360, 360, 300).astype(np.float32)
    for th in th32:
        for K in (7, 31):
            dh, dw = oracle.offsets(float(th), K)
            edh, edw = exact_offsets(float(th), K)
            assert list(dh) == edh and list(dw) == edw, (float(th), K)


def test_offsets_rational_sine_angles():
    # 30 and 150 degrees: sin = 1/2 exactly, so j = -2 must give dh = floor(1) = 1.
    for th in (30.0, 150.0):
        dh, dw = oracle.offsets(th, 7)
        assert dh[1] == 1  # k = 1 -> j = -2
        assert dh[5] == -1  # k = 5 -> j = +2
    # 90 degrees: cos is exactly 0, so every dw is 0 (no half-column shift).
    dh, dw = oracle.offsets(90.0, 31)
    assert list(dw) == [0] * 31
    assert list(dh) == [15 - k for k in range(31)]


def test_offsets_bounded_and_centred():
    for th in ANGLES:
        for K in (3, 7, 31, 63):
            dh, dw = oracle.offsets(th, K)
            pad = K // 2
            assert np.all(np.abs(dh) <= pad) and np.all(np.abs(dw) <= pad)
            assert dh[pad] == 0 and dw[pad] == 0  # the convolution origin (appendix, "Convolution origin")


def test_paper_worked_example_minus45():
    spec = {}
    with open(os.path.join(GOLDEN, "paper_example_minus45_pad0.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                key, val = line.split()
                spec[key] = val
    theta, pad = float(spec["theta_deg"]), int(spec["pad"])
    assert spec["dh_per_k"] == "sqrt2/2" and spec["dw_per_k"] == "sqrt2/2"
    K = 9
    vh, vw = oracle.offsets_real(theta, K, pad)
    for k in range(K):
        assert vh[k] == pytest.approx(k * math.sqrt(2) / 2, abs=1e-13)
        assert vw[k] == pytest.approx(k * math.sqrt(2) / 2, abs=1e-13)
    dh, dw = oracle.offsets(theta, K, pad)
    # floor(k / sqrt(2)) by integer arithmetic: the largest m with 2 m^2 <= k^2.
    expect = [math.isqrt(k * k // 2) for k in range(K)]
    assert list(dh) == expect and list(dw) == expect


def test_paper_general_offset_form():
    # Same passage: the rotation gives offsets (-k sin theta, k cos theta) (pad = 0).
    for th in (10.0, 33.0, 120.0, 250.0):
        s, c = (float(v) for v in sin_cos_deg(th))
        vh, vw = oracle.offsets_real(th, 7, 0)
        for k in range(7):
            assert vh[k] == pytest.approx(-k * s, abs=1e-13)
            assert vw[k] == pytest.approx(k * c, abs=1e-13)


def test_redundancy_duplicates_exist():
    # The same passage notes redundant offsets under round-down; at 45 degrees K = 31
    # has 31 taps but fewer distinct cells.
    dh, dw = oracle.offsets(45.0, 31)
    assert len(set(zip(dh, dw))) < 31


# ------------------------------------------------------------- forward (Eq. 1)

def _torch_corr(x, kern, padding):
    xt = torch.from_numpy(x)
    kt = torch.from_numpy(kern)
    return F.conv2d(xt, kt, padding=padding, groups=x.shape[1]).numpy()


@pytest.mark.parametrize("H,W,K", [(9, 13, 5), (12, 7, 7), (5, 5, 9), (16, 16, 15), (3, 40, 31)])
def test_theta0_is_horizontal_correlation(H, W, K):
    N, C = 2, 3
    x, w = rand(N, C, H, W), rand(C, K)
    y = oracle.fwd(x, w, np.zeros(C))
    ref = _torch_corr(x, w.reshape(C, 1, 1, K), (0, K // 2))
    np.testing.assert_allclose(y, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("H,W,K", [(9, 13, 5), (12, 7, 7), (5, 5, 9), (40, 3, 31)])
def test_theta90_is_vertical_convolution(H, W, K):
    # theta = 90: dh = pad - k, dw = 0, i.e. a vertical correlation with the reversed kernel.
    N, C = 2, 3
    x, w = rand(N, C, H, W), rand(C, K)
    y = oracle.fwd(x, w, np.full(C, 90.0))
    ref = _torch_corr(x, w[:, ::-1].copy().reshape(C, 1, K, 1), (K // 2, 0))
    np.testing.assert_allclose(y, ref, rtol=0, atol=1e-12)


def _mask(theta_deg, w_row, K):
    pad = K // 2
    dh, dw = exact_offsets(theta_deg, K)
    m = np.zeros((K, K))
    for k in range(K):
        m[pad + dh[k], pad + dw[k]] += w_row[k]  # duplicates add
    return m


@pytest.mark.parametrize("K", [3, 7, 15, 31])
def test_any_angle_is_rasterised_2d_correlation(K):
    N, H, W = 2, 19, 23
    thetas = np.array([0, 22.5, 45, 67.5, 90, 112.5, 135, 157.5, 30, 150, 200, -33.3, 301.7])
    C = len(thetas)
    x, w = rand(N, C, H, W), rand(C, K)
    y = oracle.fwd(x, w, thetas)
    kern = np.stack([_mask(float(thetas[c]), w[c], K) for c in range(C)])[:, None]
    ref = _torch_corr(x, kern, K // 2)
    np.testing.assert_allclose(y, ref, rtol=0, atol=1e-11)


def test_k1_is_scaling():
    x, w = rand(2, 4, 6, 7), rand(4, 1)
    y = oracle.fwd(x, w, np.array([0.0, 33.0, 90.0, 271.0]))
    np.testing.assert_allclose(y, x * w[None, :, :, None], rtol=0, atol=0)


def test_one_hot_weight_is_shift_with_zero_fill():
    N, C, H, W, K = 1, 4, 11, 12, 9
    thetas = np.array([22.5, 67.5, 135.0, 300.0])
    x = rand(N, C, H, W)
    for k in range(K):
        w = np.zeros((C, K)); w[:, k] = 1.0
        y = oracle.fwd(x, w, thetas)
        for c in range(C):
            dh, dw = exact_offsets(float(thetas[c]), K)
            ref = np.zeros((H, W))
            for p in range(H):
                for q in range(W):
                    h, ww = p + dh[k], q + dw[k]
                    if 0 <= h < H and 0 <= ww < W:
                        ref[p, q] = x[0, c, h, ww]
            np.testing.assert_array_equal(y[0, c], ref)


def test_impulse_response():
    H, W, K = 21, 21, 11
    thetas = np.array([0.0, 22.5, 45.0, 112.5, 157.5, 77.7])
    C = len(thetas)
    w = rand(C, K)
    x = np.zeros((1, C, H, W)); h0, w0 = 10, 9
    x[0, :, h0, w0] = 1.0
    y = oracle.fwd(x, w, thetas)
    for c in range(C):
        dh, dw = exact_offsets(float(thetas[c]), K)
        ref = np.zeros((H, W))
        for k in range(K):  # y[p,q] picks x at (p+dh, q+dw): nonzero where p = h0 - dh
            ref[h0 - dh[k], w0 - dw[k]] += w[c, k]
        np.testing.assert_allclose(y[0, c], ref, rtol=0, atol=1e-15)


def test_linearity():
    x1, x2, w = rand(2, 3, 8, 9), rand(2, 3, 8, 9), rand(3, 7)
    th = np.array([10.0, 95.0, 170.0])
    a, b = 0.75, -1.5
    np.testing.assert_allclose(oracle.fwd(a * x1 + b * x2, w, th),
                               a * oracle.fwd(x1, w, th) + b * oracle.fwd(x2, w, th), atol=1e-12)


# --------------------------------------------------------------- gradients

@pytest.mark.parametrize("K", [3, 5, 7])
def test_gradients_match_finite_differences(K):
    N, C, H, W = 2, 3, 5, 6
    th = np.array([22.5, 101.0, 315.0])
    x, w, dy = rand(N, C, H, W), rand(C, K), rand(N, C, H, W)
    loss = lambda xx, ww: float(np.sum(oracle.fwd(xx, ww, th, threads=1) * dy))
    gx = oracle.bwd_input(dy, w, th, threads=1)
    gw = oracle.bwd_weight(x, dy, th, K, threads=1)
    # the loss is linear in x and in w, so a unit central difference is exact up to rounding
    fx = np.zeros_like(x)
    for idx in np.ndindex(x.shape):
        e = np.zeros_like(x); e[idx] = 1.0
        fx[idx] = (loss(x + e, w) - loss(x - e, w)) / 2
    fw = np.zeros_like(w)
    for idx in np.ndindex(w.shape):
        e = np.zeros_like(w); e[idx] = 1.0
        fw[idx] = (loss(x, w + e) - loss(x, w - e)) / 2
    np.testing.assert_allclose(gx, fx, rtol=0, atol=1e-10)
    np.testing.assert_allclose(gw, fw, rtol=0, atol=1e-10)


@pytest.mark.parametrize("K", [7, 31])
def test_adjoint_identities(K):
    N, C, H, W = 3, 8, 20, 24
    th = np.random.default_rng(3).uniform(0, 360, C)
    x, w, dy = rand(N, C, H, W), rand(C, K), rand(N, C, H, W)
    y = oracle.fwd(x, w, th)
    lhs = float(np.sum(y * dy))
    rhs_x = float(np.sum(x * oracle.bwd_input(dy, w, th)))
    rhs_w = float(np.sum(w * oracle.bwd_weight(x, dy, th, K)))
    assert rhs_x == pytest.approx(lhs, rel=1e-12, abs=1e-9)
    assert rhs_w == pytest.approx(lhs, rel=1e-12, abs=1e-9)


def test_bwd_input_is_transposed_mask_correlation():
    # dx = correlation of dy with the point-reflected rasterised mask (conv_transpose of the mask).
    N, H, W, K = 2, 13, 17, 9
    th = np.array([0.0, 45.0, 112.5, 200.0])
    C = len(th)
    dy, w = rand(N, C, H, W), rand(C, K)
    dx = oracle.bwd_input(dy, w, th)
    kern = np.stack([_mask(float(th[c]), w[c], K) for c in range(C)])[:, None]
    ref = F.conv_transpose2d(torch.from_numpy(dy), torch.from_numpy(kern), padding=K // 2, groups=C).numpy()
    np.testing.assert_allclose(dx, ref, rtol=0, atol=1e-11)


def test_bwd_weight_via_torch_autograd_of_mask_conv():
    N, H, W, K = 2, 11, 14, 7
    th = np.array([22.5, 90.0, 157.5])
    C = len(th)
    x, dy, w = rand(N, C, H, W), rand(N, C, H, W), rand(C, K)
    gw = oracle.bwd_weight(x, dy, th, K)
    # build the mask as a differentiable function of w and let autograd do the adjoint
    wt = torch.from_numpy(w).requires_grad_(True)
    rows = []
    pad = K // 2
    for c in range(C):
        dh, dw = exact_offsets(float(th[c]), K)
        m = torch.zeros(K, K, dtype=torch.float64)
        for k in range(K):
            onehot = torch.zeros(K, K, dtype=torch.float64)
            onehot[pad + dh[k], pad + dw[k]] = 1.0
            m = m + onehot * wt[c, k]
        rows.append(m)
    kern = torch.stack(rows)[:, None]
    y = F.conv2d(torch.from_numpy(x), kern, padding=pad, groups=C)
    (y * torch.from_numpy(dy)).sum().backward()
    np.testing.assert_allclose(gw, wt.grad.numpy(), rtol=0, atol=1e-10)


def test_discrete_angles_are_well_conditioned():
    # The eight angles i * 22.5 degrees keep every non-integer product at least 0.01
    # away from an integer for K <= 63, so any two correct double-precision
    # evaluations of Eq. (2) agree on the floors.
    for i in range(8):
        assert min_distance_to_integer(22.5 * i, 63) > 0.01
