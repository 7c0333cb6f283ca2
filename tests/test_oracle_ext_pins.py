"""Pins of the oracle's stride and bilinear-interpolation extensions.

Stride is the `str` of Definition 1, Eq. (2); the bilinear variant is the
alternative to rounding down that the section "Discretization and
Interpolation" weighs.  Each test compares the oracle with something
independent of its code:
  * stride: the stride-1 output subsampled at (str p, str q) (Eq. 2 with
    str = 1 versus str > 1), torch's float64 strided conv2d at 0 degrees and
    through the rasterised K x K mask at every angle, torch autograd of that
    convolution for both gradients;
  * bilinear: scipy's bilinear sampler (ndimage.map_coordinates, order 1,
    zero outside the plane) at the exact real offsets, the rounded-down
    result where the offsets are integers, the partition of unity on a
    constant image, finite differences, adjoint identities and one-hot
    weights for the gradients.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F
from scipy import ndimage

import oracle
from exact_offsets import exact_offsets, sin_cos_deg

RNG = np.random.default_rng(4321)
THETAS = np.array([0, 22.5, 45, 67.5, 90, 112.5, 135, 157.5, 30, 150, 200, -33.3, 301.7, 11.0])


def rand(*shape):
    return RNG.standard_normal(shape)


def _mask(theta_deg, w_row, K):
    pad = K // 2
    dh, dw = exact_offsets(theta_deg, K)
    m = np.zeros((K, K))
    for k in range(K):
        m[pad + dh[k], pad + dw[k]] += w_row[k]
    return m


# ------------------------------------------------------------------ stride

def test_output_size_reading():
    # P = floor((H - 1) / str) + 1: the size torch gives a centred odd kernel with padding K // 2
    for H in (1, 2, 7, 8, 56, 57):
        for s in (1, 2, 3, 4):
            for K in (1, 3, 7, 31):
                ref = F.conv2d(torch.zeros(1, 1, H, 3, dtype=torch.float64), torch.zeros(1, 1, K, 1,
                               dtype=torch.float64), stride=(s, 1), padding=(K // 2, 0)).shape[2]
                assert oracle.out_size(H, s) == ref


@pytest.mark.parametrize("mode", ["floor", "bilinear"])
@pytest.mark.parametrize("s", [2, 3, 4])
def test_stride_is_subsampled_stride1(mode, s):
    C = len(THETAS)
    for H, W, K in ((17, 23, 7), (16, 16, 15), (9, 30, 31)):
        x, w = rand(2, C, H, W), rand(C, K)
        y1 = oracle.fwd(x, w, THETAS, mode=mode)
        ys = oracle.fwd(x, w, THETAS, stride=s, mode=mode)
        np.testing.assert_array_equal(ys, y1[:, :, ::s, ::s])


@pytest.mark.parametrize("s", [2, 3])
def test_stride_theta0_is_strided_horizontal_correlation(s):
    N, C, H, W, K = 2, 3, 11, 14, 7
    x, w = rand(N, C, H, W), rand(C, K)
    y = oracle.fwd(x, w, np.zeros(C), stride=s)
    ref = F.conv2d(torch.from_numpy(x), torch.from_numpy(w.reshape(C, 1, 1, K)), stride=s, padding=(0, K // 2),
                   groups=C).numpy()
    np.testing.assert_allclose(y, ref, rtol=0, atol=1e-12)


def _mask_conv(x, w, thetas, K, s):
    """torch conv2d with the rasterised mask, differentiable in x and in w."""
    C = len(thetas)
    sel = np.zeros((C, K, K * K))
    for c in range(C):
        dh, dw = exact_offsets(float(thetas[c]), K)
        for k in range(K):
            sel[c, k, (K // 2 + dh[k]) * K + K // 2 + dw[k]] = 1.0
    xt = torch.tensor(x, requires_grad=True)
    wt = torch.tensor(w, requires_grad=True)
    kern = torch.einsum("ck,ckm->cm", wt, torch.from_numpy(sel)).reshape(C, 1, K, K)
    return xt, wt, F.conv2d(xt, kern, stride=s, padding=K // 2, groups=C)


@pytest.mark.parametrize("s", [1, 2, 3])
@pytest.mark.parametrize("K", [5, 15])
def test_stride_any_angle_and_gradients_via_torch(s, K):
    C = len(THETAS)
    N, H, W = 2, 19, 22
    x, w = rand(N, C, H, W), rand(C, K)
    xt, wt, yt = _mask_conv(x, w, THETAS, K, s)
    y = oracle.fwd(x, w, THETAS, stride=s)
    np.testing.assert_allclose(y, yt.detach().numpy(), rtol=0, atol=1e-11)
    dy = rand(*y.shape)
    yt.backward(torch.from_numpy(dy))
    dx = oracle.bwd_input(dy, w, THETAS, stride=s, in_hw=(H, W))
    dw = oracle.bwd_weight(x, dy, THETAS, K, stride=s)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=0, atol=1e-10)
    np.testing.assert_allclose(dw, wt.grad.numpy(), rtol=0, atol=1e-9)


# ---------------------------------------------------------------- bilinear

def _exact_real_offsets(theta, K):
    s, c = sin_cos_deg(theta)
    pad = K // 2
    return ([float(-(k - pad) * s) for k in range(K)], [float((k - pad) * c) for k in range(K)])


def _scipy_bilinear(x, w, thetas, K, s=1):
    N, C, H, W = x.shape
    P, Q = (H - 1) // s + 1, (W - 1) // s + 1
    pp, qq = np.meshgrid(np.arange(P) * s, np.arange(Q) * s, indexing="ij")
    y = np.zeros((N, C, P, Q))
    for c in range(C):
        rh, rw = _exact_real_offsets(float(thetas[c]), K)
        for k in range(K):
            coords = np.stack([(pp + rh[k]).ravel(), (qq + rw[k]).ravel()])
            for n in range(N):
                y[n, c] += w[c, k] * ndimage.map_coordinates(x[n, c], coords, order=1, mode="grid-constant",
                                                              cval=0.0).reshape(P, Q)
    return y


@pytest.mark.parametrize("s", [1, 2])
@pytest.mark.parametrize("K", [3, 7, 31])
def test_bilinear_matches_scipy_sampler(K, s):
    C = len(THETAS)
    x, w = rand(2, C, 13, 17), rand(C, K)
    y = oracle.fwd(x, w, THETAS, stride=s, mode="bilinear")
    np.testing.assert_allclose(y, _scipy_bilinear(x, w, THETAS, K, s), rtol=0, atol=1e-10)


def test_bilinear_equals_round_down_at_axis_angles():
    th = np.array([0.0, 90.0, 180.0, 270.0, -90.0, 360.0])
    C = len(th)
    for K in (3, 7, 31):
        x, w = rand(2, C, 12, 15), rand(C, K)
        np.testing.assert_allclose(oracle.fwd(x, w, th, mode="bilinear"), oracle.fwd(x, w, th), rtol=0, atol=1e-12)


def test_bilinear_partition_of_unity():
    # on a constant image every sample that stays inside the plane is exactly 1
    K = 7
    C = len(THETAS)
    w = rand(C, K)
    y = oracle.fwd(np.ones((1, C, 24, 24)), w, THETAS, mode="bilinear")
    inner = y[:, :, K:-K, K:-K]
    np.testing.assert_allclose(inner, np.broadcast_to(w.sum(1)[None, :, None, None], inner.shape), rtol=0, atol=1e-12)


def test_bilinear_coefficients():
    for th in THETAS:
        sh, sw, sc = oracle.tap_samples(float(th), 9, "bilinear")
        rh, rw = _exact_real_offsets(float(th), 9)
        np.testing.assert_allclose(sc.sum(1), 1.0, atol=1e-15)
        # the interpolated position is the coefficient-weighted mean of the corners
        np.testing.assert_allclose((sc * sh).sum(1), rh, atol=1e-12)
        np.testing.assert_allclose((sc * sw).sum(1), rw, atol=1e-12)
        assert (sc >= 0).all()


@pytest.mark.parametrize("s", [1, 2])
def test_bilinear_gradients_finite_differences(s):
    C, K, H, W = 3, 5, 6, 7
    th = np.array([22.5, 61.0, 143.0])
    x, w = rand(1, C, H, W), rand(C, K)
    y = oracle.fwd(x, w, th, stride=s, mode="bilinear")
    dy = rand(*y.shape)
    dx = oracle.bwd_input(dy, w, th, stride=s, mode="bilinear", in_hw=(H, W))
    dw = oracle.bwd_weight(x, dy, th, K, stride=s, mode="bilinear")
    L = lambda xx, ww: float(np.sum(oracle.fwd(xx, ww, th, stride=s, mode="bilinear") * dy))
    for _ in range(12):
        i = tuple(RNG.integers(0, n) for n in x.shape)
        e = np.zeros_like(x); e[i] = 1.0
        assert abs((L(x + e, w) - L(x - e, w)) / 2 - dx[i]) < 1e-10
    for c in range(C):
        for k in range(K):
            e = np.zeros_like(w); e[c, k] = 1.0
            assert abs((L(x, w + e) - L(x, w - e)) / 2 - dw[c, k]) < 1e-10


@pytest.mark.parametrize("mode", ["floor", "bilinear"])
@pytest.mark.parametrize("s", [1, 2, 3])
def test_adjoint_identities_ext(mode, s):
    C, K, H, W = len(THETAS), 15, 20, 21
    x, w = rand(2, C, H, W), rand(C, K)
    y = oracle.fwd(x, w, THETAS, stride=s, mode=mode)
    dy = rand(*y.shape)
    lhs = float(np.sum(y * dy))
    dx = oracle.bwd_input(dy, w, THETAS, stride=s, mode=mode, in_hw=(H, W))
    dw = oracle.bwd_weight(x, dy, THETAS, K, stride=s, mode=mode)
    assert abs(lhs - float(np.sum(x * dx))) <= 1e-9 * max(1.0, abs(lhs))
    assert abs(lhs - float(np.sum(w * dw))) <= 1e-9 * max(1.0, abs(lhs))


def test_bilinear_weight_gradient_is_one_hot_forward():
    # dw[c,k] = <dy, fwd(x; e_k)> (the forward is linear in w and pinned by scipy above)
    C, K = len(THETAS), 7
    x, dy = rand(2, C, 10, 12), rand(2, C, 10, 12)
    dw = oracle.bwd_weight(x, dy, THETAS, K, mode="bilinear")
    for k in range(K):
        e = np.zeros((C, K)); e[:, k] = 1.0
        ref = np.sum(oracle.fwd(x, e, THETAS, mode="bilinear") * dy, axis=(0, 2, 3))
        np.testing.assert_allclose(dw[:, k], ref, rtol=0, atol=1e-10)
