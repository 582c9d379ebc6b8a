"""Build libeb.so (the HIP kernels and the C ABI) for gfx950 with hipcc.

    python -m paper_2609_30656_amd.build
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
SOURCES = [os.path.join(CSRC, f) for f in ("eb_forward.hip", "eb_fm.hip", "eb_seq.hip", "eb_backward.hip") if os.path.exists(os.path.join(CSRC, f))]
# the random-row gather rate measurement (a program of its own, not part of libeb.so)
GATHER_SRC = os.path.join(CSRC, "gather_ceiling.hip")
GATHER_BIN = os.path.join(PKG, "gather_ceiling")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libeb.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    # keep hipcc from forming packed fp32 instructions on its own
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
    "-Wno-unused-result",
]


def build(verbose: bool = False, extra_flags=()) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    tmp = LIB + ".tmp"
    cmd = [hipcc, *HIPCC_FLAGS, *extra_flags, "-I", INCLUDE, "-I", CSRC, *SOURCES, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def build_gather_ceiling(verbose: bool = False) -> str:
    """Compile the gather_ceiling measurement program next to libeb.so."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    flags = [f for f in HIPCC_FLAGS if f not in ("-shared", "-fPIC")]
    tmp = GATHER_BIN + ".tmp"
    cmd = [hipcc, *flags, GATHER_SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, GATHER_BIN)
    return GATHER_BIN


if __name__ == "__main__":
    print(build(verbose=True))
    print(build_gather_ceiling(verbose=True))
    sys.exit(0)
