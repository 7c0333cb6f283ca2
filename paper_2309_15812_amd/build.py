"""Builds the HIP library ``libo1d.so`` in-tree for gfx950 with hipcc.

Usage: ``python -m paper_2309_15812_amd.build`` (or ``build()`` from Python).
Cross-compiles without a GPU.  Every ``csrc/*.hip`` translation unit is
compiled to an object in parallel (the line kernels are split per storage
type and kind for this), then the objects are linked into the library.
"""
from __future__ import annotations

import concurrent.futures
import glob
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


# The line kernels keep LDS reads in flight across inline-assembly blocks in
# registers the compiler believes are written; a register spill between two
# such blocks would store a value before it arrives.  Their translation units
# are therefore compiled with resource remarks and rejected if any kernel in
# them uses scratch memory.
CHECKED = ("o1d_line_", "o1d_strip_")
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


def build(verbose: bool = False, jobs: int | None = None) -> str:
    srcs = sources()
    jobs = jobs or min(len(srcs), max(1, min(os.cpu_count() or 1, 16)))
    tmpdir = tempfile.mkdtemp(prefix="o1d_build_")
    try:
        objs = [os.path.join(tmpdir, os.path.basename(s) + ".o") for s in srcs]
        cmds = [[HIPCC, *FLAGS, *([REMARK] if os.path.basename(s).startswith(CHECKED) else []),
                 "-I", INCLUDE, "-I", CSRC, "-c", "-o", o, s] for s, o in zip(srcs, objs)]
        with concurrent.futures.ThreadPoolExecutor(max_workers=jobs) as ex:
            for fut in [ex.submit(_run, c, verbose) for c in cmds]:
                fut.result()
        tmp = LIB + ".tmp"
        _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs], verbose)
        os.replace(tmp, LIB)
    finally:
        shutil.rmtree(tmpdir, ignore_errors=True)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
