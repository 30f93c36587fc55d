"""Builds libra_mi355x.so (HIP kernels + C ABI) for gfx950 with hipcc.

    python -m paper_2505_17623_amd.build

The library is built in-tree next to this file, so it travels with the
source tree.  Every HIP source is compiled with packed-FP32 instructions
disabled.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libra_mi355x.so")
SOURCES = ["witness.hip", "gemm.hip", "sumcheck.hip", "planes.hip", "xrounds.hip", "fp2.hip", "link.hip", "fs.hip", "commit.hip", "abi.hip", "noalloc.hip", "verify.cpp"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"


FLAGS = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
OBJDIR = os.path.join(ROOT, "_build")


def command(out: str = LIB):
    """One hipcc command that builds the whole library (for reference)."""
    return [HIPCC, *FLAGS, "-shared", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
            *[os.path.join(CSRC, s) for s in SOURCES], "-o", out]


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    errs = "\n".join(l for l in (res.stdout + res.stderr).splitlines()
                     if "packed-fp32-ops" not in l and l.strip())
    return res.returncode, errs


def build(verbose: bool = False) -> str:
    """Compile every source to an object in parallel (each is self-contained
    device code), then link the shared library."""
    from concurrent.futures import ThreadPoolExecutor
    os.makedirs(OBJDIR, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    objs, cmds = [], []
    for s in SOURCES:
        o = os.path.join(OBJDIR, os.path.splitext(s)[0] + ".o")
        objs.append(o)
        cmds.append([HIPCC, *FLAGS, *inc, "-c", os.path.join(CSRC, s), "-o", o])
    jobs = max(1, min(len(cmds), int(os.environ.get("MAX_JOBS", os.cpu_count() or 1))))
    with ThreadPoolExecutor(jobs) as ex:
        results = list(ex.map(_run, cmds))
    for cmd, (rc, errs) in zip(cmds, results):
        if verbose:
            print(" ".join(cmd), flush=True)
        if rc != 0:
            raise RuntimeError(f"hipcc failed ({rc}) on {cmd[-3]}:\n{errs}")
        if verbose and errs:
            print(errs, flush=True)
    tmp = LIB + ".tmp"
    rc, errs = _run([HIPCC, *FLAGS, "-shared", *objs, "-o", tmp])
    if rc != 0:
        raise RuntimeError(f"hipcc link failed ({rc}):\n{errs}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose="-q" not in sys.argv)
    print("built", LIB)
