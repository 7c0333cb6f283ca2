"""GPU parity, part 2: every compiled kernel variant, stride, NHWC, bilinear
sampling, large planes, bfloat16 rounding and the device-side offsets.

Same bar as test_parity_gpu.py (per tensor max|g - r| / max|r| <= 1e-5 for
float32, 2e-2 for bfloat16 storage, against the float64 oracle on the inputs
the GPU saw), plus an element-wise bound for bfloat16 stores that only
round-to-nearest-even meets.  NHWC cases feed the oracle (which takes NCHW)
the permuted tensors.
"""
import numpy as np
import pytest
import torch

import oracle
from cases import variant_cases
from paper_2309_15812_amd import _lib, ops, synth

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}
DEV = "cuda:0"


def err(g, r):
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    den = np.max(np.abs(r)) if r.size else 0.0
    return float(np.max(np.abs(g - r)) / den) if den > 0 else float(np.max(np.abs(g - r), initial=0.0))


def tdt(name):
    return torch.float32 if name == "f32" else torch.bfloat16


def dev(a, dtype, offset_elems=0):
    """A device tensor holding a; offset_elems > 0 places it that many elements into a larger buffer
    (a base pointer that is not vector aligned)."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dtype)
    if offset_elems == 0:
        return t.to(DEV)
    buf = torch.zeros(t.numel() + offset_elems, dtype=dtype, device=DEV)
    buf[offset_elems:] = t.reshape(-1).to(DEV)
    return buf[offset_elems:].view(t.shape)


def host(t):
    return t.float().cpu().numpy()


def to_layout(a, layout):
    return np.ascontiguousarray(a.transpose(0, 2, 3, 1)) if layout == "nhwc" else a


def from_layout(a, layout):
    return np.ascontiguousarray(a.transpose(0, 3, 1, 2)) if layout == "nhwc" else a


def run_ex(N, C, H, W, K, dtype="f32", theta="uniform", stride=1, layout="nchw", sampling="floor", seed=31,
           offset=0, label=""):
    """fwd_ex, bwd_input_ex and bwd_weight_ex against the oracle at this stride / layout / sampling."""
    print(f"[parity-ex] {label} N={N} C={C} H={H} W={W} K={K} {dtype} theta={theta} stride={stride} "
          f"{layout} {sampling} offset={offset}", flush=True)
    wl = synth.Workload("ex", N, C, H, W, K, dtype, theta, "fwd+bwd", seed)
    d = synth.make_inputs(wl)
    P, Q = oracle.out_size(H, stride), oracle.out_size(W, stride)
    dy = d["dy"][:, :, :P, :Q].copy()  # the upstream gradient has the output plane's shape
    dt = tdt(dtype)
    x = dev(to_layout(d["x"], layout), dt, offset)
    g = dev(to_layout(dy, layout), dt, offset)
    w = dev(d["w"], dt)
    th = torch.from_numpy(d["theta"]).to(DEV)
    y = ops.fwd_ex(x, w, th, stride, layout, sampling)
    dx = ops.bwd_input_ex(g, w, th, (H, W), stride, layout, sampling)
    dw = ops.bwd_weight_ex(x, g, th, K, stride, layout, sampling)
    torch.cuda.synchronize()
    res = {
        "fwd": err(from_layout(host(y), layout), oracle.fwd(d["x"], d["w"], d["theta"], stride=stride, mode=sampling)),
        "bwd_input": err(from_layout(host(dx), layout),
                         oracle.bwd_input(dy, d["w"], d["theta"], stride=stride, mode=sampling, in_hw=(H, W))),
        "bwd_weight": err(host(dw), oracle.bwd_weight(d["x"], dy, d["theta"], K, stride=stride, mode=sampling)),
    }
    print(f"[parity-ex] {label}: " + " ".join(f"{k}={v:.2e}" for k, v in res.items()), flush=True)
    for k, v in res.items():
        assert v <= TOL[dtype], f"{label} {k}: err {v:.3e} > {TOL[dtype]}"
    return res


def run_plain(N, C, H, W, K, dtype, theta="uniform", seed=41, offset=0, label=""):
    """o1d_fwd, o1d_bwd_input, o1d_bwd_weight and o1d_bwd against the oracle (NCHW, stride 1)."""
    print(f"[parity] {label} N={N} C={C} H={H} W={W} K={K} {dtype} theta={theta} offset={offset}", flush=True)
    wl = synth.Workload("plain", N, C, H, W, K, dtype, theta, "fwd+bwd", seed)
    d = synth.make_inputs(wl)
    dt = tdt(dtype)
    x, dy = dev(d["x"], dt, offset), dev(d["dy"], dt, offset)
    w = dev(d["w"], dt)
    th = torch.from_numpy(d["theta"]).to(DEV)
    y = ops.fwd(x, w, th)
    dx = ops.bwd_input(dy, w, th)
    dw = ops.bwd_weight(x, dy, th, K)
    fdx, fdw = ops.bwd(x, dy, w, th)
    torch.cuda.synchronize()
    rdx = oracle.bwd_input(d["dy"], d["w"], d["theta"])
    rdw = oracle.bwd_weight(d["x"], d["dy"], d["theta"], K)
    res = {"fwd": err(host(y), oracle.fwd(d["x"], d["w"], d["theta"])), "bwd_input": err(host(dx), rdx),
           "bwd_weight": err(host(dw), rdw), "bwd.dx": err(host(fdx), rdx), "bwd.dw": err(host(fdw), rdw)}
    print(f"[parity] {label}: " + " ".join(f"{k}={v:.2e}" for k, v in res.items()), flush=True)
    for k, v in res.items():
        assert v <= TOL[dtype], f"{label} {k}: err {v:.3e} > {TOL[dtype]}"


# ------------------------------------------------------------ every compiled variant

VARIANTS = variant_cases()


@pytest.mark.parametrize("variant", sorted(VARIANTS))
def test_every_compiled_variant(variant):
    N, C, H, W, K, dtype, layout, aligned = VARIANTS[variant]
    off = 0 if aligned else 1
    if layout == "nchw":
        run_plain(N, C, H, W, K, dtype, offset=off, label=variant)
    else:
        run_ex(N, C, H, W, K, dtype, layout=layout, offset=off, label=variant)


# ------------------------------------------------------------ stride, layout, sampling

EX = [
    # (N, C, H, W, K, dtype, theta, stride, layout, sampling)
    (2, 5, 23, 29, 7, "f32", "uniform", 2, "nchw", "floor"),
    (2, 4, 30, 30, 31, "f32", "discrete8", 2, "nchw", "floor"),
    (1, 3, 41, 37, 15, "f32", "uniform", 3, "nchw", "floor"),
    (2, 3, 17, 20, 9, "bf16", "uniform", 4, "nchw", "floor"),
    (3, 6, 14, 14, 31, "f32", "uniform", 1, "nhwc", "floor"),
    (2, 12, 28, 28, 31, "f32", "discrete8", 1, "nhwc", "floor"),
    (2, 20, 14, 14, 31, "bf16", "uniform", 1, "nhwc", "floor"),
    (2, 9, 19, 22, 7, "f32", "uniform", 2, "nhwc", "floor"),
    (2, 5, 23, 29, 7, "f32", "uniform", 1, "nchw", "bilinear"),
    (2, 4, 28, 28, 31, "f32", "discrete8", 1, "nchw", "bilinear"),
    (1, 3, 33, 31, 15, "f32", "uniform", 2, "nchw", "bilinear"),
    (2, 6, 14, 14, 31, "bf16", "uniform", 1, "nchw", "bilinear"),
    (2, 10, 16, 18, 11, "f32", "uniform", 1, "nhwc", "bilinear"),
    (1, 3, 12, 12, 63, "f32", "uniform", 1, "nchw", "bilinear"),
    (1, 2, 20, 24, 127, "f32", "uniform", 1, "nchw", "floor"),
    (1, 2, 9, 9, 127, "f32", "uniform", 2, "nchw", "bilinear"),
]


# small planes with at least eight images (the plane kernels): strides,
# bilinear sampling, image counts that leave a ragged last group of images,
# planes whose size allows vector accesses of four, two or one element
PLANE_EX = [
    (16, 6, 14, 14, 31, "f32", "uniform", 1, "nchw", "floor"),
    (9, 5, 14, 14, 31, "bf16", "uniform", 1, "nchw", "floor"),
    (70, 2, 14, 14, 31, "bf16", "discrete8", 1, "nchw", "floor"),
    (12, 4, 23, 29, 7, "f32", "uniform", 2, "nchw", "floor"),
    (10, 3, 17, 20, 9, "bf16", "uniform", 3, "nchw", "bilinear"),
    (16, 4, 14, 14, 31, "f32", "discrete8", 2, "nchw", "bilinear"),
    (20, 3, 13, 11, 15, "f32", "uniform", 4, "nchw", "floor"),
    (8, 2, 6, 20, 63, "bf16", "uniform", 1, "nchw", "bilinear"),
    (40, 3, 7, 7, 31, "f32", "uniform", 1, "nchw", "bilinear"),
    (33, 3, 10, 6, 15, "f32", "uniform", 1, "nchw", "floor"),
]

# general kernels whose workgroups hold more (channel, tap) pairs than
# threads (NHWC channel blocks with long kernels): every tap's cells built
EX_MANY_TAPS = [
    (2, 16, 14, 14, 63, "bf16", "uniform", 1, "nhwc", "floor"),
    (2, 8, 9, 9, 127, "f32", "uniform", 1, "nhwc", "floor"),
    (2, 12, 11, 13, 33, "bf16", "uniform", 2, "nhwc", "bilinear"),
]


# the plane shapes of the bench line's general-kernel configurations (NHWC
# at 56 x 56, stride 2 at 224 x 224, bilinear at 56 x 56), with few images
# and channels: the band plans depend on the plane, K and the channel block
EX_BENCH_SHAPES = [
    (2, 8, 56, 56, 31, "f32", "discrete8", 1, "nhwc", "floor"),
    (1, 4, 224, 224, 31, "f32", "discrete8", 2, "nchw", "floor"),
    (2, 3, 56, 56, 31, "f32", "discrete8", 1, "nchw", "bilinear"),
]


@pytest.mark.parametrize("case", EX + PLANE_EX + EX_MANY_TAPS + EX_BENCH_SHAPES, ids=lambda c: "-".join(map(str, c)))
def test_stride_layout_sampling(case):
    N, C, H, W, K, dtype, theta, s, layout, sampling = case
    run_ex(N, C, H, W, K, dtype, theta, s, layout, sampling, label=str(case))


def test_ex_matches_plain_at_stride1_nchw_floor():
    # with stride 1, NCHW and rounding down, the _ex calls are the plain ones (same kernels, bitwise)
    wl = synth.Workload("same", 3, 5, 28, 28, 31, "f32", "discrete8", "fwd+bwd", 51)
    d = synth.make_inputs(wl)
    x, dy, w = dev(d["x"], torch.float32), dev(d["dy"], torch.float32), dev(d["w"], torch.float32)
    th = torch.from_numpy(d["theta"]).to(DEV)
    a = [ops.fwd(x, w, th), ops.bwd_input(dy, w, th), ops.bwd_weight(x, dy, th, 31)]
    b = [ops.fwd_ex(x, w, th), ops.bwd_input_ex(dy, w, th, (28, 28)), ops.bwd_weight_ex(x, dy, th, 31)]
    torch.cuda.synchronize()
    for u, v in zip(a, b):
        assert torch.equal(u, v)


def _random_ex(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        H, W = int(rng.integers(1, 50)), int(rng.integers(1, 50))
        K = int(rng.choice([1, 3, 7, 15, 31, 33, 63]))
        out.append((int(rng.integers(1, 4)), int(rng.integers(1, 13)), H, W, K,
                    "f32" if rng.random() < 0.6 else "bf16", str(rng.choice(["uniform", "discrete8"])),
                    int(rng.choice([1, 1, 2, 3])), str(rng.choice(["nchw", "nhwc"])),
                    str(rng.choice(["floor", "bilinear"]))))
    return out


@pytest.mark.parametrize("case", _random_ex(16, 20261203), ids=lambda c: "-".join(map(str, c)))
def test_random_ex(case):
    N, C, H, W, K, dtype, theta, s, layout, sampling = case
    run_ex(N, C, H, W, K, dtype, theta, s, layout, sampling, label=f"random {case}")


# ------------------------------------------------------------ large planes, alignment

@pytest.mark.parametrize("case", [(1, 2, 224, 224, 31, "f32"), (1, 2, 224, 224, 31, "bf16"),
                                  (1, 1, 512, 512, 31, "f32"), (1, 2, 512, 130, 63, "f32")],
                         ids=lambda c: "x".join(map(str, c[:5])) + "-" + c[5])
def test_large_planes(case):
    N, C, H, W, K, dtype = case
    run_plain(N, C, H, W, K, dtype, label=f"large {case}")


def test_large_plane_stride2_nhwc():
    run_ex(1, 3, 224, 224, 31, "f32", "uniform", 2, "nhwc", "floor", label="224^2 stride 2 nhwc")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_misaligned_base_pointers_both_dtypes(dtype):
    # one element past an aligned base: the planner must route to kernels that take any alignment
    run_plain(2, 6, 19, 24, 9, dtype, offset=1, label=f"misaligned {dtype}")
    run_plain(2, 4, 28, 28, 31, dtype, offset=1, label=f"misaligned strip shape {dtype}")


# ------------------------------------------------------------ bfloat16 rounding

def _ulp_bf16(v):
    _, e = np.frexp(np.abs(v))  # |v| = m 2^e, m in [0.5, 1)
    return np.ldexp(1.0, e - 8)  # 8 significant bits


@pytest.mark.parametrize("shape", [(4, 16, 14, 14, 31), (2, 8, 28, 28, 31), (2, 8, 20, 24, 7)])
def test_bf16_stores_round_to_nearest_even(shape):
    # |g - r| <= half an ulp of bfloat16 plus the float32 accumulation error, element by element:
    # a truncating store (errors up to a whole ulp) fails this for about half of the elements
    N, C, H, W, K = shape
    wl = synth.Workload("rne", N, C, H, W, K, "bf16", "uniform", "fwd+bwd", 61)
    d = synth.make_inputs(wl)
    x, dy, w = dev(d["x"], torch.bfloat16), dev(d["dy"], torch.bfloat16), dev(d["w"], torch.bfloat16)
    th = torch.from_numpy(d["theta"]).to(DEV)
    y, dx = ops.fwd(x, w, th), ops.bwd_input(dy, w, th)
    fdx, _ = ops.bwd(x, dy, w, th)
    torch.cuda.synchronize()
    for name, g, r, a in (
            ("fwd", host(y), oracle.fwd(d["x"], d["w"], d["theta"]),
             oracle.fwd(np.abs(d["x"]), np.abs(d["w"]), d["theta"])),
            ("bwd_input", host(dx), oracle.bwd_input(d["dy"], d["w"], d["theta"]),
             oracle.bwd_input(np.abs(d["dy"]), np.abs(d["w"]), d["theta"])),
            ("bwd.dx", host(fdx), oracle.bwd_input(d["dy"], d["w"], d["theta"]),
             oracle.bwd_input(np.abs(d["dy"]), np.abs(d["w"]), d["theta"]))):
        bound = 0.5 * np.maximum(_ulp_bf16(r), _ulp_bf16(g)) + K * 2.0 ** -23 * a
        over = np.abs(g - r) > bound
        print(f"[rne] {shape} {name}: {int(over.sum())} of {over.size} elements over the bound", flush=True)
        assert not over.any()


# ------------------------------------------------------------ device-side offsets

def _decode_offsets(y, K, c0):
    """From y of an impulse at (c0, c0) with w_k = 2^k: the offset (dh_k, dw_k) of every tap."""
    C = y.shape[1]
    dh = np.full((C, K), 99, np.int64)
    dw = np.full((C, K), 99, np.int64)
    for c in range(C):
        ps, qs = np.nonzero(y[0, c])
        for p, q in zip(ps, qs):
            v = int(round(float(y[0, c, p, q])))
            for k in range(K):
                if (v >> k) & 1:
                    assert dh[c, k] == 99, (c, k)
                    dh[c, k], dw[c, k] = c0 - p, c0 - q
    return dh, dw


@pytest.mark.parametrize("K,M", [(31, 32), (31, 31), (63, 64), (15, 20)])
def test_device_offsets_equal_oracle(K, M):
    # every tap's offset as the GPU computes it, read back through the forward pass, for 10^4 random
    # float32 angles (plus the exact-integer ones), against the oracle's offsets
    rng = np.random.default_rng(71 + K + M)
    th = np.concatenate([rng.uniform(-360, 360, 10000), np.arange(0, 360, 7.5), [30, 150, -90, 1e-3]])
    th = th.astype(np.float32)
    C, c0 = len(th), K // 2
    x = np.zeros((1, C, M, M), np.float32)
    x[0, :, c0, c0] = 1.0
    w = np.tile(np.ldexp(1.0, np.arange(K)), (C, 1)).astype(np.float32)
    print(f"[offsets] K={K} M={M} kernel={_lib.kernel_name(0, 1, C, M, M, K)}", flush=True)
    xt, wt, tt = dev(x, torch.float32), dev(w, torch.float32), torch.from_numpy(th).to(DEV)
    y = host(ops.fwd(xt, wt, tt))
    dx = host(ops.bwd_input(xt, wt, tt))  # mirrored taps: the impulse lands at (c0 + dh, c0 + dw)
    dh, dw = _decode_offsets(y, K, c0)
    mh, mw = _decode_offsets(dx, K, c0)
    bad = 0
    for c in range(C):
        rh, rw = oracle.offsets(float(th[c]), K)
        if not (np.array_equal(dh[c], rh) and np.array_equal(dw[c], rw) and np.array_equal(mh[c], -rh)
                and np.array_equal(mw[c], -rw)):
            bad += 1
            print(f"[offsets] theta={th[c]!r}: gpu {list(zip(dh[c], dw[c]))} oracle {list(zip(rh, rw))}", flush=True)
    assert bad == 0


def test_device_bilinear_coefficients_equal_oracle():
    # one channel per (angle, tap) with a one-hot weight: the forward of an impulse is the tap's
    # bilinear footprint (coefficients at the corners), read back and compared with the oracle's
    K, M, c0 = 7, 12, 6
    th = np.random.default_rng(5).uniform(0, 360, 300).astype(np.float32)
    C = len(th) * K
    x = np.zeros((1, C, M, M), np.float32)
    x[0, :, c0, c0] = 1.0
    w = np.zeros((C, K), np.float32)
    w[np.arange(C), np.arange(C) % K] = 1.0
    tt = np.repeat(th, K)
    y = host(ops.fwd_ex(dev(x, torch.float32), dev(w, torch.float32), torch.from_numpy(tt).to(DEV),
                        sampling="bilinear"))
    for c in range(C):
        k = c % K
        sh, sw, sc = oracle.tap_samples(float(tt[c]), K, "bilinear")
        ref = np.zeros((M, M))
        for s in range(4):
            if sc[k, s] != 0:
                ref[c0 - sh[k, s], c0 - sw[k, s]] += sc[k, s]
        assert np.max(np.abs(y[0, c] - ref)) <= 1e-6, (float(tt[c]), k)


# ------------------------------------------------------------ wrapper checks

def test_wrapper_rejects_bad_workspace():
    x = torch.randn(2, 3, 8, 8, device=DEV)
    w = torch.randn(3, 5, device=DEV)
    th = torch.zeros(3, device=DEV)
    need = ops.workspace_bytes(2, 3, 8, 8, 5, torch.float32)
    for bad in (torch.empty(need, dtype=torch.uint8),  # host memory
                torch.empty(max(need - 1, 0), dtype=torch.uint8, device=DEV),  # too small
                torch.empty(2 * need, dtype=torch.uint8, device=DEV)[::2]):  # not contiguous
        with pytest.raises(ValueError):
            ops.bwd_weight(x, x, th, 5, workspace=bad)
        with pytest.raises(ValueError):
            ops.bwd(x, x, w, th, workspace=bad)


def test_autograd_with_channels_last_input():
    wl = synth.Workload("cl", 2, 5, 17, 20, 11, "f32", "uniform", "fwd+bwd", 17)
    d = synth.make_inputs(wl)
    x = dev(d["x"], torch.float32).to(memory_format=torch.channels_last).requires_grad_(True)
    w = dev(d["w"], torch.float32).requires_grad_(True)
    th = torch.from_numpy(d["theta"]).to(DEV)
    y = ops.OrientedConv1dFunction.apply(x, w, th)
    y.backward(dev(d["dy"], torch.float32))
    torch.cuda.synchronize()
    assert err(host(y.detach()), oracle.fwd(d["x"], d["w"], d["theta"])) <= 1e-5
    assert err(host(x.grad), oracle.bwd_input(d["dy"], d["w"], d["theta"])) <= 1e-5
    assert err(host(w.grad), oracle.bwd_weight(d["x"], d["dy"], d["theta"], wl.K)) <= 1e-5
