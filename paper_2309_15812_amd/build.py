"""Builds the HIP library ``libo1d.so`` in-tree for gfx950 with hipcc.

Usage: ``python -m paper_2309_15812_amd.build`` (or ``build()`` from Python).
Cross-compiles without a GPU.  Every ``csrc/*.hip`` translation unit is
compiled to an object in parallel (the strip kernels are split per family,
storage type and cell bound for this), then the objects are linked into the
library.
"""
from __future__ import annotations

import concurrent.futures
import glob
import hashlib
import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libo1d.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    # Keep the compiler from forming packed FP32 instructions.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
]


def sources() -> list[str]:
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


# The strip kernels are sized to stay in registers (their walks keep a
# window and per-output accumulators of up to 60 values per lane); a spill to
# scratch memory would cost far more than it saves, so their translation
# units are compiled with resource remarks and rejected if any kernel in them
# uses scratch memory.  The general kernels are checked the same way.
CHECKED = ("o1d_strip_", "o1d_gen_", "o1d_plane_", "o1d_pw_")
REMARK = "-Rpass-analysis=kernel-resource-usage"


def _check_no_scratch(src: str, stderr: str) -> None:
    name, bad = None, []
    for line in stderr.splitlines():
        if "Function Name:" in line:
            name = line.split("Function Name:")[1].split()[0]
        elif "ScratchSize [bytes/lane]:" in line and name is not None:
            if int(line.split("ScratchSize [bytes/lane]:")[1].split()[0]) != 0:
                bad.append(name)
    if bad:
        raise RuntimeError(f"{os.path.basename(src)}: kernels use scratch memory (register spills): {bad}")


def _run(cmd: list[str], verbose: bool) -> None:
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed with exit code {res.returncode}: {' '.join(cmd[-3:])}")
    if REMARK in cmd:
        _check_no_scratch(cmd[-1], res.stderr)


def _key(src: str, flags: list[str]) -> str:
    """Hash of a translation unit, every header it may include and the flags."""
    h = hashlib.sha256(" ".join(flags).encode())
    for f in [src, *sorted(glob.glob(os.path.join(CSRC, "*.h"))), os.path.join(INCLUDE, "o1d.h")]:
        with open(f, "rb") as fh:
            h.update(os.path.basename(f).encode() + b"\0" + fh.read())
    return h.hexdigest()[:20]


def build(verbose: bool = False, jobs: int | None = None, incremental: bool = False) -> str:
    """Compiles every translation unit and links libo1d.so.  With incremental=True, objects whose source,
    headers and flags are unchanged are reused from _build/ (a development aid; the default always
    recompiles everything)."""
    srcs = sources()
    jobs = jobs or min(len(srcs), max(1, min(os.cpu_count() or 1, 16)))
    tmpdir = tempfile.mkdtemp(prefix="o1d_build_")
    cache = os.path.join(PKG, "_build")
    try:
        objs, cmds = [], []
        for src in srcs:
            extra = [REMARK] if os.path.basename(src).startswith(CHECKED) else []
            flags = [*FLAGS, *extra]
            obj = os.path.join(tmpdir, os.path.basename(src) + ".o")
            cached = os.path.join(cache, os.path.basename(src) + "." + _key(src, flags) + ".o")
            if incremental and os.path.exists(cached):
                shutil.copy(cached, obj)
            else:
                cmds.append(([HIPCC, *flags, "-I", INCLUDE, "-I", CSRC, "-c", "-o", obj, src], obj, cached))
            objs.append(obj)
        with concurrent.futures.ThreadPoolExecutor(max_workers=jobs) as ex:
            for fut in [ex.submit(_run, c, verbose) for c, _, _ in cmds]:
                fut.result()
        if incremental:
            os.makedirs(cache, exist_ok=True)
            for _, obj, cached in cmds:
                shutil.copy(obj, cached)
        tmp = LIB + ".tmp"
        _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs], verbose)
        os.replace(tmp, LIB)
    finally:
        shutil.rmtree(tmpdir, ignore_errors=True)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True, incremental="--incremental" in sys.argv))
