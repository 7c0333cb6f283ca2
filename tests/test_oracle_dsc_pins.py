"""Pins of the oracle's depthwise separable block (Sec. 3.2, Table 1 "Oriented 1D DSC"): the pointwise
stage against a closed form written out by hand, the identity pointwise stage, and every gradient
against central finite differences of a scalar loss.  Pointwise weights are non-square and not
symmetric, so a transposed operand fails."""
import math

import numpy as np
import pytest

import oracle


def _inputs(N, C, Co, H, W, K, seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((N, C, H, W))
    w_dw = rng.standard_normal((C, K)) / math.sqrt(K)
    th = rng.uniform(0, 180, C).astype(np.float32)
    w_pw = rng.standard_normal((Co, C)) / math.sqrt(C)
    return x, w_dw, th, w_pw


def test_k1_closed_form():
    # K = 1: the depthwise stage scales each channel by its single tap at any angle, so
    # y[n,o,h,w] = sum_c w_pw[o,c] w_dw[c,0] x[n,c,h,w]
    x, w_dw, th, w_pw = _inputs(2, 3, 5, 4, 6, 1, 1)
    _, y = oracle.dsc_fwd(x, w_dw, th, w_pw)
    ref = np.zeros((2, 5, 4, 6))
    for n in range(2):
        for o in range(5):
            for h in range(4):
                for w in range(6):
                    ref[n, o, h, w] = sum(w_pw[o, c] * w_dw[c, 0] * x[n, c, h, w] for c in range(3))
    assert np.allclose(y, ref, rtol=1e-13, atol=1e-13)


def test_identity_pointwise_is_depthwise():
    x, w_dw, th, _ = _inputs(2, 4, 4, 9, 7, 5, 2)
    z, y = oracle.dsc_fwd(x, w_dw, th, np.eye(4))
    assert np.array_equal(y, z)
    assert np.array_equal(z, oracle.fwd(x, w_dw, th))


def test_channel_mix_is_linear_in_w_pw():
    x, w_dw, th, w_pw = _inputs(1, 3, 2, 5, 5, 3, 3)
    _, y1 = oracle.dsc_fwd(x, w_dw, th, w_pw)
    _, y2 = oracle.dsc_fwd(x, w_dw, th, 2.5 * w_pw)
    _, ys = oracle.dsc_fwd(x, w_dw, th, w_pw + np.ones_like(w_pw))
    _, y1s = oracle.dsc_fwd(x, w_dw, th, np.ones_like(w_pw))
    assert np.allclose(y2, 2.5 * y1, rtol=1e-13, atol=1e-13)
    assert np.allclose(ys, y1 + y1s, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("which", ["x", "w_dw", "w_pw"])
def test_gradients_match_finite_differences(which):
    N, C, Co, H, W, K = 2, 3, 4, 5, 6, 5
    x, w_dw, th, w_pw = _inputs(N, C, Co, H, W, K, 4)
    g = np.random.default_rng(5).standard_normal((N, Co, H, W))  # dL/dy for L = <g, y>
    dx, dw_dw, dw_pw = oracle.dsc_bwd(x, g, w_dw, th, w_pw)
    params = {"x": x, "w_dw": w_dw, "w_pw": w_pw}
    grad = {"x": dx, "w_dw": dw_dw, "w_pw": dw_pw}[which]
    p = params[which]
    rng = np.random.default_rng(6)
    for idx in [tuple(rng.integers(0, s) for s in p.shape) for _ in range(6)]:
        h = 1e-6
        def loss(delta):
            q = {k: v.copy() for k, v in params.items()}
            q[which][idx] += delta
            return float(np.sum(g * oracle.dsc_fwd(q["x"], q["w_dw"], th, q["w_pw"])[1]))
        fd = (loss(h) - loss(-h)) / (2 * h)
        assert abs(fd - grad[idx]) <= 1e-6 * max(1.0, abs(fd)), (which, idx, fd, grad[idx])
