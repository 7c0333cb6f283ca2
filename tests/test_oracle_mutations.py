"""The pins catch plausible mistakes in the oracle.

Each case plants one slip in a scratch copy of the C oracle (on the CPU, in a
temporary directory) and runs the pin suite against that copy: it must fail.
The slips are the ones a reader of Definition 1 / Eq. (1)-(2) could make: the
sign of the sine inside the floor, sine for cosine, no snap of exact integers,
the pad moved out of the centring shift, a transposed weight layout, a
flipped kernel in the input gradient, a transposed image index in the weight
gradient, radians taken for degrees.  The extensions (stride, bilinear
interpolation) get slips of their own, checked against their own pin suite:
the stride ignored, the output size, a swapped bilinear coefficient or
corner, no fraction, and a wrong coefficient in either adjoint.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTATIONS = {
    "sin-sign": ("dh_real[k] = -j * s;", "dh_real[k] = j * s;"),
    "sin-for-cos": ("dw_real[k] = j * c;", "dw_real[k] = j * s;"),
    "no-snap": ("if (fabs(v - r) <= ORACLE_SNAP_EPS) return r;", ""),
    "pad-outside": ("const double j = (double)(k - pad);", "const double j = (double)k;"),
    "weight-layout": ("acc += xp[(size_t)h * W + w] * wt[(size_t)c * K + k];",
                      "acc += xp[(size_t)h * W + w] * wt[(size_t)k * C + c];"),
    "bwd-input-flipped": ("xp[(size_t)h * W + w] += g * wt[(size_t)c * K + k];",
                          "xp[(size_t)h * W + w] += g * wt[(size_t)c * K + (K - 1 - k)];"),
    "bwd-weight-transposed": ("g[k] += gy * xp[(size_t)h * W + w];", "g[k] += gy * xp[(size_t)w * W + h];"),
    "radians": ("const double t = theta_deg * (M_PI / 180.0);", "const double t = theta_deg;"),
}


# (old, new, pin suite); every occurrence of `old` is replaced
EXT_MUTATIONS = {
    "stride-ignored": ("const int h = str * p + sh[4 * k + s];", "const int h = p + sh[4 * k + s];"),
    "out-size": ("int oracle_out_size(int n, int str) { return (n - 1) / str + 1; }",
                 "int oracle_out_size(int n, int str) { return n / str + (n % str > 1); }"),
    "bilinear-coef-swap": ("sc[4 * k + 1] = (1.0 - fh) * fw;", "sc[4 * k + 1] = (1.0 - fw) * fh;"),
    "bilinear-corner": ("sw[4 * k + s] = (int)w0 + (s & 1);", "sw[4 * k + s] = (int)w0 + (s >> 1);"),
    "bilinear-no-fraction": ("const double fh = (fabs(rh[k] - h0) <= ORACLE_SNAP_EPS) ? 0.0 : rh[k] - h0;",
                             "const double fh = 0.0;"),
    "bwd-input-ex-coef": ("xp[(size_t)h * W + w] += g * sc[4 * k + s] * wt[(size_t)c * K + k];",
                          "xp[(size_t)h * W + w] += g * sc[4 * k + (3 - s)] * wt[(size_t)c * K + k];"),
    "bwd-weight-ex-coef": ("g[k] += gy * sc[4 * k + s] * xp[(size_t)h * W + w];",
                           "g[k] += gy * sc[4 * k + (s ^ 1)] * xp[(size_t)h * W + w];"),
}
CASES = {**{n: (*v, "test_oracle_pins.py", False) for n, v in MUTATIONS.items()},
         **{n: (*v, "test_oracle_ext_pins.py", True) for n, v in EXT_MUTATIONS.items()}}


@pytest.mark.parametrize("name", sorted(CASES))
def test_pins_catch_planted_oracle_mistake(name, tmp_path):
    old, new, suite, every = CASES[name]
    shutil.copytree(os.path.join(ROOT, "oracle"), tmp_path / "oracle",
                    ignore=shutil.ignore_patterns("*.so", "__pycache__"))
    (tmp_path / "tests").mkdir()
    for f in ("conftest.py", "exact_offsets.py", suite):
        shutil.copy(os.path.join(ROOT, "tests", f), tmp_path / "tests" / f)
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), tmp_path / "tests" / "golden")
    src = tmp_path / "oracle" / "o1d_oracle.c"
    text = src.read_text()
    assert text.count(old) >= 1 and (every or text.count(old) == 1), f"mutation {name} does not apply"
    src.write_text(text.replace(old, new))
    r = subprocess.run([sys.executable, "-m", "pytest", f"tests/{suite}", "-x", "-q",
                        "-p", "no:cacheprovider", "-m", "not gpu"],
                       cwd=tmp_path, capture_output=True, text=True, timeout=600)
    # exit status 1 = tests ran and at least one failed (2+ would be a collection or usage error)
    assert r.returncode == 1, f"mutation {name} was not caught (rc={r.returncode}):\n{r.stdout[-2000:]}"
