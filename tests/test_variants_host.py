"""Host-side planning: which kernel every call takes, and that every compiled
kernel variant is reached by a GPU parity case.

The planner is the library's own host code (o1d_kernel_name runs the same
routing as the entry points), so these tests need no GPU.
"""
import pytest

from cases import variant_cases
from paper_2309_15812_amd import _lib


def test_every_compiled_variant_has_a_parity_case():
    variants = _lib.kernel_variants()
    assert len(variants) == len(set(variants)) > 0
    missing = sorted(set(variants) - set(variant_cases()))
    assert not missing, f"compiled variants without a GPU parity case: {missing}"


def test_planned_names_are_compiled_variants():
    known = set(_lib.kernel_variants())
    for case in variant_cases().values():
        N, C, H, W, K, dt, layout, aligned = case
        d = _lib.O1D_F32 if dt == "f32" else _lib.O1D_BF16
        lay = _lib.O1D_NHWC if layout == "nhwc" else _lib.O1D_NCHW
        for op in (0, 1, 2):
            for v in _lib.kernel_name(op, N, C, H, W, K, 1, lay, _lib.O1D_FLOOR, d, aligned).split("+"):
                assert v in known, v


@pytest.mark.parametrize("args,expect", [
    # the headline shape: strip kernels, fused backward
    ((0, 64, 96, 56, 56, 31), "strip_gather/f32/S77/KB32"),
    ((3, 64, 96, 56, 56, 31), "strip_bwd/f32/S77/KB32"),
    ((3, 64, 192, 28, 28, 31), "strip_bwd/f32/S51/KB32"),
    # K = 63: strip gather; both gradients in the general one-pass kernel (the
    # strip one stops at 31 cells)
    ((0, 32, 256, 56, 56, 63), "strip_gather/f32/S103/KB64"),
    ((3, 32, 256, 56, 56, 63), "gen_bwd/f32/nchw/RP4/KB64"),
    # 14 x 14 planes (W not a multiple of 4) with many images: plane kernels
    # (lanes over images), two rows per lane
    ((0, 64, 384, 14, 14, 31), "plane_gather/f32/RP2"),
    ((3, 64, 384, 14, 14, 31), "plane_bwd/f32/RP2/KB32"),
    ((0, 64, 384, 14, 14, 31, 1, 0, 0, 1), "plane_gather/bf16/RP2"),
    # fewer than eight images: general kernels
    ((0, 4, 384, 14, 14, 31), "gen_gather/f32/nchw/RP4"),
    # planes too large for the strip tiles
    ((0, 1, 2, 224, 224, 31), "gen_gather/f32/nchw/RP8"),
])
def test_routing(args, expect):
    assert _lib.kernel_name(*args) == expect


def test_routing_of_options():
    assert _lib.kernel_name(0, 2, 4, 56, 56, 31, 2).startswith("gen_gather/")
    assert _lib.kernel_name(0, 2, 4, 56, 56, 31, 1, _lib.O1D_NHWC).startswith("gen_gather/f32/nhwc")
    assert _lib.kernel_name(2, 2, 4, 56, 56, 31, 1, _lib.O1D_NCHW, _lib.O1D_BILINEAR).startswith("gen_wgrad/")
    assert _lib.kernel_name(0, 2, 4, 56, 56, 31, aligned=False).startswith("gen_gather/")
    assert _lib.kernel_name(0, 2, 4, 56, 56, 31, dtype=_lib.O1D_BF16) == "strip_gather/bf16/S77/KB32"
    # invalid or empty sizes name no kernel
    assert _lib.kernel_name(0, 2, 4, 56, 56, 30) == ""
    assert _lib.kernel_name(0, 0, 4, 56, 56, 31) == ""
    assert _lib.kernel_name(3, 2, 4, 56, 56, 31, 2) == ""  # o1d_bwd has no stride
    # unaligned tensors: the general one-pass backward
    assert _lib.kernel_name(3, 2, 4, 56, 56, 31, aligned=False) == "gen_bwd/f32/nchw/RP8/KB32"


def test_workspace_sizes_cover_every_route():
    # the workspace covers both the aligned and the unaligned route, and the _ex sizes the general kernels
    lib = _lib.lib()
    for (N, C, H, W, K) in ((64, 96, 56, 56, 31), (3, 4, 14, 14, 31), (2, 3, 224, 224, 63)):
        plain = lib.o1d_bwd_weight_workspace_bytes(N, C, H, W, K, 0)
        ex = lib.o1d_bwd_weight_ex_workspace_bytes(N, C, H, W, K, 1, 0, 0, 0)
        assert plain == ex > 0 and plain % (C * K * 4) == 0
        for s in (2, 3):
            for lay in (0, 1):
                for smp in (0, 1):
                    b = lib.o1d_bwd_weight_ex_workspace_bytes(N, C, H, W, K, s, lay, smp, 0)
                    assert b > 0 and b % (C * K * 4) == 0
