"""GPU parity: the HIP kernels against the float64 CPU oracle, element by element.

Bar (per output tensor): err = max_i |g_i - r_i| / max_i |r_i|, with r the oracle
in float64 on exactly the inputs the GPU saw, is at most 1e-5 for float32 and
2e-2 for bfloat16 storage (float32 accumulation).  The offsets are integer
decisions; both sides take them in double precision under the same reading of
Eq. (2), so they agree exactly and the float tolerance only covers the float32
(or bfloat16) rounding of the sums.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2309_15812_amd import ops, synth

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}
DEV = "cuda:0"


def err(g, r):
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    den = np.max(np.abs(r)) if r.size else 0.0
    return float(np.max(np.abs(g - r)) / den) if den > 0 else float(np.max(np.abs(g - r), initial=0.0))


def dev_tensor(a, dtype):
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(DEV).to(dtype)


def host(t):
    return t.float().cpu().numpy()


def torch_dtype(name):
    return torch.float32 if name == "f32" else torch.bfloat16


def run_case(wl, ops_to_check=("fwd", "bwd_input", "bwd_weight", "bwd"), inputs=None, label=""):
    print(f"[parity] {label or wl.name}: N={wl.N} C={wl.C} H={wl.H} W={wl.W} K={wl.K} {wl.dtype} "
          f"theta={wl.theta} ops={ops_to_check}", flush=True)
    d = synth.make_inputs(wl) if inputs is None else inputs
    dt = torch_dtype(wl.dtype)
    x, dy, w = dev_tensor(d["x"], dt), dev_tensor(d["dy"], dt), dev_tensor(d["w"], dt)
    th = torch.from_numpy(d["theta"]).to(DEV)
    tol = TOL[wl.dtype]
    res = {}
    if "fwd" in ops_to_check:
        y = ops.fwd(x, w, th)
        torch.cuda.synchronize()
        res["fwd"] = err(host(y), oracle.fwd(d["x"], d["w"], d["theta"]))
    ref = {}

    def ref_dx():
        if "dx" not in ref:
            ref["dx"] = oracle.bwd_input(d["dy"], d["w"], d["theta"])
        return ref["dx"]

    def ref_dw():
        if "dw" not in ref:
            ref["dw"] = oracle.bwd_weight(d["x"], d["dy"], d["theta"], wl.K)
        return ref["dw"]

    if "bwd_input" in ops_to_check:
        dx = ops.bwd_input(dy, w, th)
        torch.cuda.synchronize()
        res["bwd_input"] = err(host(dx), ref_dx())
    if "bwd_weight" in ops_to_check:
        dw = ops.bwd_weight(x, dy, th, wl.K)
        torch.cuda.synchronize()
        res["bwd_weight"] = err(host(dw), ref_dw())
    if "bwd" in ops_to_check:  # both gradients from one call
        fdx, fdw = ops.bwd(x, dy, w, th)
        torch.cuda.synchronize()
        res["bwd.dx"] = err(host(fdx), ref_dx())
        res["bwd.dw"] = err(host(fdw), ref_dw())
    print(f"[parity] {label or wl.name}: " + " ".join(f"{k}={v:.2e}" for k, v in res.items()), flush=True)
    for k, v in res.items():
        assert v <= tol, f"{label or wl.name} {k}: err {v:.3e} > {tol}"
    return res


# ------------------------------------------------------------ the five configurations

def test_c1_small_forward():
    run_case(synth.WORKLOADS["c1"], ("fwd",))


def test_c1_all_ops():
    run_case(synth.WORKLOADS["c1"])


def test_c2_stage1_forward():
    run_case(synth.WORKLOADS["c2"], ("fwd",))


def test_metric_stage1_fwd_bwd():
    run_case(synth.WORKLOADS["metric"])


def test_c3_stage2_fwd_bwd():
    run_case(synth.WORKLOADS["c3"])


def test_c4_stage3_bf16_continuous():
    run_case(synth.WORKLOADS["c4"])


@pytest.mark.parametrize("K", [7, 15, 31, 63])
@pytest.mark.parametrize("mode", ["zero", "ninety", "uniform"])
def test_c5_angle_sweep(K, mode):
    run_case(synth.WORKLOADS["c5"].replace(K=K, theta=mode), label=f"c5 K={K} {mode}")


# ------------------------------------------------------------ edges

EDGE = [
    # (N, C, H, W, K, theta mode)
    (2, 5, 13, 57, 7, "uniform"),      # ragged, H != W
    (3, 4, 1, 1, 31, "uniform"),       # 1x1 plane, K > H
    (2, 8, 7, 7, 31, "discrete8"),     # K much larger than the plane
    (1, 3, 3, 200, 15, "uniform"),     # very wide
    (1, 3, 200, 3, 15, "uniform"),     # very tall
    (2, 6, 130, 70, 31, "uniform"),    # several tiles per plane, ragged tiles
    (2, 4, 45, 45, 1, "uniform"),      # K = 1
    (2, 4, 45, 45, 3, "discrete8"),
    (1, 3, 40, 33, 63, "uniform"),
    (1, 2, 20, 24, 127, "uniform"),    # the largest supported K
    (1, 9, 57, 57, 31, "groups:8"),    # the paper's D equal groups
]


@pytest.mark.parametrize("case", EDGE, ids=lambda c: "x".join(map(str, c[:5])) + "-" + c[5])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_edges(case, dtype):
    N, C, H, W, K, mode = case
    wl = synth.Workload("edge", N, C, H, W, K, dtype, mode, "fwd+bwd", 11)
    run_case(wl, label=f"edge {case} {dtype}")


# Shapes the strip kernels take (W % 4 == 0, aligned tensors): non-square
# planes in both staging frames, bands that do not fill the last strip,
# groups of several planes with a partial last group, walks of up to 64
# cells, the split diagonal lane layout (bands in fours of more than 8
# column groups), and the line-kernel fallback next to them.
EDGE_STRIP = [
    # (N, C, H, W, K, theta mode)
    (3, 5, 20, 44, 31, "uniform"),     # H != W, ragged bands, several planes per group
    (5, 3, 44, 20, 15, "discrete8"),   # tall plane, N not a multiple of the group
    (2, 4, 56, 56, 1, "uniform"),      # one cell
    (2, 4, 56, 56, 3, "discrete8"),
    (2, 3, 36, 48, 45, "uniform"),     # walks of up to 64 cells (weight gradient: line kernel)
    (7, 2, 12, 16, 31, "uniform"),     # K larger than the plane, many planes per group
    (3, 2, 96, 8, 7, "uniform"),       # tall and narrow
    (2, 3, 8, 100, 7, "uniform"),      # short and wide
    (1, 2, 64, 64, 31, "uniform"),     # more tasks than a workgroup: line kernels
    (9, 4, 28, 28, 31, "groups:8"),    # the paper's D equal groups
    (4, 3, 24, 32, 31, "uniform"),     # split diagonal layout: 4 bands of 10 column groups
    (2, 3, 79, 28, 15, "uniform"),     # split diagonal layout: 12 bands of 9 column groups
]


@pytest.mark.parametrize("case", EDGE_STRIP, ids=lambda c: "x".join(map(str, c[:5])) + "-" + c[5])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_strip_edges(case, dtype):
    N, C, H, W, K, mode = case
    wl = synth.Workload("strip-edge", N, C, H, W, K, dtype, mode, "fwd+bwd", 13)
    run_case(wl, label=f"strip edge {case} {dtype}")


def test_angles_outside_zero_180():
    wl = synth.Workload("angles", 2, 12, 23, 29, 15, "f32", "uniform", "fwd+bwd", 12)
    d = synth.make_inputs(wl)
    d["theta"] = np.array([-45, -90, -157.5, 180, 202.5, 270, 359, 360, 405, 720.5, -1000.25, 30],
                          dtype=np.float32)
    run_case(wl, inputs=d, label="angles outside [0,180)")


def test_exact_integer_angles():
    # 0, 30, 90, 150, 180 ... degrees, where double-precision products sit a rounding error
    # away from integers; both sides must take the exact-arithmetic offsets.
    wl = synth.Workload("int-angles", 2, 10, 31, 31, 31, "f32", "uniform", "fwd+bwd", 13)
    d = synth.make_inputs(wl)
    d["theta"] = np.array([0, 30, 60, 90, 120, 150, 180, 210, 270, 330], dtype=np.float32)
    run_case(wl, inputs=d, label="exact-integer angles")


def test_misaligned_base_pointers():
    wl = synth.Workload("misaligned", 2, 6, 19, 21, 9, "f32", "uniform", "fwd+bwd", 14)
    d = synth.make_inputs(wl)
    n = d["x"].size
    xb = torch.zeros(n + 1, device=DEV); xb[1:] = torch.from_numpy(d["x"].ravel()).to(DEV)
    x = xb[1:].view(d["x"].shape)
    yb = torch.full((n + 1,), float("nan"), device=DEV)
    y = yb[1:].view(d["x"].shape)
    w = dev_tensor(d["w"], torch.float32)
    th = torch.from_numpy(d["theta"]).to(DEV)
    ops.fwd(x, w, th, out=y)
    torch.cuda.synchronize()
    assert err(host(y), oracle.fwd(d["x"], d["w"], d["theta"])) <= 1e-5
    assert torch.isnan(yb[0])  # the element before the output was not touched
    # the fused backward with misaligned tensors takes the separate kernels
    dyb = torch.zeros(n + 1, device=DEV); dyb[1:] = torch.from_numpy(d["dy"].ravel()).to(DEV)
    dy = dyb[1:].view(d["x"].shape)
    dxb = torch.full((n + 1,), float("nan"), device=DEV)
    dx, dw = ops.bwd(x, dy, w, th, out=(dxb[1:].view(d["x"].shape), torch.empty_like(w)))
    torch.cuda.synchronize()
    assert err(host(dx), oracle.bwd_input(d["dy"], d["w"], d["theta"])) <= 1e-5
    assert err(host(dw), oracle.bwd_weight(d["x"], d["dy"], d["theta"], wl.K)) <= 1e-5
    assert torch.isnan(dxb[0])


def test_outputs_fully_written_and_guard_regions_intact():
    wl = synth.Workload("guard", 3, 7, 37, 41, 31, "f32", "uniform", "fwd+bwd", 15)
    d = synth.make_inputs(wl)
    x, dy = dev_tensor(d["x"], torch.float32), dev_tensor(d["dy"], torch.float32)
    w = dev_tensor(d["w"], torch.float32)
    th = torch.from_numpy(d["theta"]).to(DEV)
    n, g = d["x"].size, 4096
    for fn, a in ((ops.fwd, x), (ops.bwd_input, dy)):
        buf = torch.full((n + 2 * g,), float("nan"), device=DEV)
        fn(a, w, th, out=buf[g:g + n].view(d["x"].shape))
        torch.cuda.synchronize()
        assert not torch.isnan(buf[g:g + n]).any()
        assert torch.isnan(buf[:g]).all() and torch.isnan(buf[g + n:]).all()
    ck = wl.C * wl.K
    buf = torch.full((ck + 2 * g,), float("nan"), device=DEV)
    ops.bwd_weight(x, dy, th, wl.K, out=buf[g:g + ck].view(wl.C, wl.K))
    torch.cuda.synchronize()
    assert not torch.isnan(buf[g:g + ck]).any()
    assert torch.isnan(buf[:g]).all() and torch.isnan(buf[g + ck:]).all()
    # the fused backward, on a shape its one-pass kernel takes (W % 4 == 0)
    wl = synth.Workload("guard", 3, 7, 36, 40, 31, "f32", "uniform", "fwd+bwd", 15)
    d = synth.make_inputs(wl)
    x, dy = dev_tensor(d["x"], torch.float32), dev_tensor(d["dy"], torch.float32)
    w = dev_tensor(d["w"], torch.float32)
    th = torch.from_numpy(d["theta"]).to(DEV)
    n, ck = d["x"].size, wl.C * wl.K
    bx = torch.full((n + 2 * g,), float("nan"), device=DEV)
    bw = torch.full((ck + 2 * g,), float("nan"), device=DEV)
    ops.bwd(x, dy, w, th, out=(bx[g:g + n].view(d["x"].shape), bw[g:g + ck].view(wl.C, wl.K)))
    torch.cuda.synchronize()
    for b, m in ((bx, n), (bw, ck)):
        assert not torch.isnan(b[g:g + m]).any()
        assert torch.isnan(b[:g]).all() and torch.isnan(b[g + m:]).all()


def test_bitwise_reproducible():
    # no atomics anywhere: every op is bitwise equal run to run
    wl = synth.WORKLOADS["c3"].replace(N=8)
    d = synth.make_inputs(wl)
    x, dy = dev_tensor(d["x"], torch.float32), dev_tensor(d["dy"], torch.float32)
    w = dev_tensor(d["w"], torch.float32)
    th = torch.from_numpy(d["theta"]).to(DEV)
    a = [ops.fwd(x, w, th), ops.bwd_input(dy, w, th), ops.bwd_weight(x, dy, th, wl.K), *ops.bwd(x, dy, w, th)]
    b = [ops.fwd(x, w, th), ops.bwd_input(dy, w, th), ops.bwd_weight(x, dy, th, wl.K), *ops.bwd(x, dy, w, th)]
    torch.cuda.synchronize()
    for u, v in zip(a, b):
        assert torch.equal(u, v)


def test_nonfinite_angle_poisons_only_its_channel():
    wl = synth.Workload("nan-angle", 2, 4, 16, 16, 7, "f32", "uniform", "fwd+bwd", 16)
    d = synth.make_inputs(wl)
    d["theta"][2] = np.nan
    x, dy = dev_tensor(d["x"], torch.float32), dev_tensor(d["dy"], torch.float32)
    w = dev_tensor(d["w"], torch.float32)
    th = torch.from_numpy(d["theta"]).to(DEV)
    y, dx, dw = ops.fwd(x, w, th), ops.bwd_input(dy, w, th), ops.bwd_weight(x, dy, th, wl.K)
    fdx, fdw = ops.bwd(x, dy, w, th)
    torch.cuda.synchronize()
    for t in (y, dx, fdx):
        assert torch.isnan(t[:, 2]).all() and not torch.isnan(t[:, [0, 1, 3]]).any()
    for t in (dw, fdw):
        assert torch.isnan(t[2]).all() and not torch.isnan(t[[0, 1, 3]]).any()
    keep = [0, 1, 3]
    ref = oracle.fwd(d["x"][:, keep], d["w"][keep], d["theta"][keep])
    assert err(host(y)[:, keep], ref) <= 1e-5


def test_empty_inputs():
    w = torch.randn(3, 7, device=DEV)
    th = torch.zeros(3, device=DEV)
    x = torch.empty(0, 3, 8, 8, device=DEV)
    assert ops.fwd(x, w, th).shape == x.shape
    x = torch.empty(2, 3, 0, 8, device=DEV)
    dw = torch.full((3, 7), float("nan"), device=DEV)
    ops.bwd_weight(x, x, th, 7, out=dw)
    torch.cuda.synchronize()
    assert torch.equal(dw, torch.zeros_like(dw))  # empty sum
    dw.fill_(float("nan"))
    ops.bwd(x, x, w, th, out=(torch.empty_like(x), dw))
    torch.cuda.synchronize()
    assert torch.equal(dw, torch.zeros_like(dw))


def test_autograd_function_matches_oracle():
    wl = synth.Workload("autograd", 2, 5, 17, 19, 11, "f32", "uniform", "fwd+bwd", 17)
    d = synth.make_inputs(wl)
    x = dev_tensor(d["x"], torch.float32).requires_grad_(True)
    w = dev_tensor(d["w"], torch.float32).requires_grad_(True)
    th = torch.from_numpy(d["theta"]).to(DEV)
    y = ops.OrientedConv1dFunction.apply(x, w, th)
    y.backward(dev_tensor(d["dy"], torch.float32))
    torch.cuda.synchronize()
    assert err(host(y.detach()), oracle.fwd(d["x"], d["w"], d["theta"])) <= 1e-5
    assert err(host(x.grad), oracle.bwd_input(d["dy"], d["w"], d["theta"])) <= 1e-5
    assert err(host(w.grad), oracle.bwd_weight(d["x"], d["dy"], d["theta"], wl.K)) <= 1e-5


def test_fused_backward_matches_separate_calls():
    # the one-pass kernel walks the input gradient's program (same cells,
    # weights and per-output order as the separate call), so dx agrees
    # bitwise; dw sums the same products in another order
    for dtype in ("f32", "bf16"):
        wl = synth.WORKLOADS["metric"].replace(N=6, dtype=dtype)
        d = synth.make_inputs(wl)
        dt = torch_dtype(dtype)
        x, dy, w = dev_tensor(d["x"], dt), dev_tensor(d["dy"], dt), dev_tensor(d["w"], dt)
        th = torch.from_numpy(d["theta"]).to(DEV)
        dx, dw = ops.bwd_input(dy, w, th), ops.bwd_weight(x, dy, th, wl.K)
        fdx, fdw = ops.bwd(x, dy, w, th)
        torch.cuda.synchronize()
        print(f"[fused] {dtype}: dx equal={torch.equal(dx, fdx)} dw err={err(host(fdw), host(dw)):.2e}", flush=True)
        assert torch.equal(dx, fdx)
        assert err(host(fdw), host(dw)) <= TOL[dtype]


def _random_cases(n, seed):
    rng = np.random.default_rng(seed)
    cases = []
    for _ in range(n):
        H = int(rng.integers(1, 61))
        W = int(rng.choice([4, 8, 12, 16, 20, 28, 32, 40, 44, 52, 56, 60])) if rng.random() < 0.7 else \
            int(rng.integers(1, 61))
        K = int(rng.choice([1, 3, 5, 7, 9, 15, 21, 31, 33, 63]))
        N, C = int(rng.integers(1, 10)), int(rng.integers(1, 7))
        mode = str(rng.choice(["uniform", "discrete8", "ramp"]))
        dtype = "f32" if rng.random() < 0.6 else "bf16"
        cases.append((N, C, H, W, K, mode, dtype))
    return cases


# Seeded random shapes: small and ragged planes, both staging frames, dense
# and blocked lane layouts, partial plane groups, walks of up to 63 cells,
# and the fused backward on and off its one-pass kernel.
@pytest.mark.parametrize("case", _random_cases(24, 20261202), ids=lambda c: "x".join(map(str, c[:5])) + "-" + c[5] + "-" + c[6])
def test_random_shapes(case):
    N, C, H, W, K, mode, dtype = case
    wl = synth.Workload("random", N, C, H, W, K, dtype, mode, "fwd+bwd", 21)
    run_case(wl, label=f"random {case}")


def test_wrapper_rejects_mismatched_outputs():
    # the kernels take no strides or sizes of their outputs: the wrapper checks them first
    x = torch.randn(2, 3, 8, 8, device=DEV)
    w = torch.randn(3, 5, device=DEV)
    th = torch.zeros(3, device=DEV)
    for bad in (torch.empty(2, 3, 8, 7, device=DEV), torch.empty(2, 3, 8, 8, device=DEV, dtype=torch.bfloat16),
                torch.empty(2, 3, 8, 16, device=DEV)[..., ::2]):
        with pytest.raises(ValueError):
            ops.fwd(x, w, th, out=bad)
        with pytest.raises(ValueError):
            ops.bwd_input(x, w, th, out=bad)
        with pytest.raises(ValueError):
            ops.bwd(x, x, w, th, out=(bad, torch.empty_like(w)))
    with pytest.raises(ValueError):
        ops.bwd_weight(x, x, th, 5, out=torch.empty(3, 4, device=DEV))
    with pytest.raises(ValueError):
        ops.bwd(x, x, w, th, out=(torch.empty_like(x), torch.empty(3, 4, device=DEV)))
