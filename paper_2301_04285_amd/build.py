"""Builds the C-ABI shared library ``libtaps.so`` for gfx950 with hipcc.

Run as ``python -m paper_2301_04285_amd.build``; the library lands next to
this file so that it travels with the source tree.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libtaps.so")
SOURCES = ["taps_api.hip", "taps_kernels.hip"]
# VALU issue-rate calibration for the benchmark's roofline (not the cost-table path)
CALIB_LIB = os.path.join(HERE, "libtaps_calibrate.so")
CALIB_SOURCES = ["taps_calibrate.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libtaps.so)")


def command(out: str = LIB, sources=None) -> list:
    return [
        hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
        # the fp64 cost expression must not be contracted into FMAs
        "-ffp-contract=off",
        # keep the compiler from forming packed fp32 instructions
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        # the GPU scheduler that maximises instruction-level parallelism within a
        # wavefront: the edge kernels are bound by VALU issue with dependency
        # stalls between (about 0.7 % faster on the 96-layer GPT than the default)
        "-mllvm", "-amdgpu-sched-strategy=max-ilp",
        "-I", INCLUDE, "-I", CSRC,
        *[os.path.join(CSRC, s) for s in (sources or SOURCES)],
        "-o", out,
    ]


def _build_one(lib: str, sources, verbose: bool) -> None:
    tmp = lib + ".tmp"
    cmd = command(tmp, sources)
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"building {os.path.basename(lib)} failed")
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    """Builds libtaps.so and the calibration library; returns libtaps.so's path."""
    _build_one(LIB, SOURCES, verbose)
    _build_one(CALIB_LIB, CALIB_SOURCES, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
