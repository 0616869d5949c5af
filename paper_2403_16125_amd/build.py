"""Build the HIP library libarena.so in-tree for gfx950 (hipcc)."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OUT = os.path.join(PKG, "_build", "libarena.so")
SOURCES = [os.path.join(CSRC, "arena_host.cpp"), os.path.join(CSRC, "arena_kernels.hip"),
           os.path.join(CSRC, "arena_sched.hip"), os.path.join(CSRC, "arena_proxy.hip")]

VALU_RATE_SRC = os.path.join(CSRC, "valu_rate.hip")
VALU_RATE_OUT = os.path.join(PKG, "_build", "libvalu_rate.so")   # fp64-vs-fp32 issue-rate microbenchmark

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off",                      # keep the operation order of the formulas
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def build(verbose: bool = False) -> str:
    os.makedirs(os.path.dirname(OUT), exist_ok=True)
    tmp = OUT + ".tmp"
    cmd = [HIPCC] + FLAGS + ["-o", tmp] + SOURCES
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, OUT)
    tmp = VALU_RATE_OUT + ".tmp"
    cmd = [HIPCC] + FLAGS + ["-o", tmp, VALU_RATE_SRC]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, VALU_RATE_OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose=True))
    sys.exit(0)
