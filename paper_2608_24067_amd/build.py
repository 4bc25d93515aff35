"""Builds libsom.so (the HIP kernels and the C ABI of include/som.h) for gfx950 with hipcc."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libsom.so")
SOURCES = [os.path.join(CSRC, "som_sweep.hip"), os.path.join(CSRC, "som_kernels.hip"), os.path.join(CSRC, "som_update.hip"),
           os.path.join(CSRC, "som_api.cpp"), os.path.join(CSRC, "som_noalloc.hip")]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

# Packed fp32 instructions are kept out of every device code object; fp contraction
# is off so that every rounding is the one the source writes.
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
    f"-I{os.path.join(ROOT, 'include')}",
]


# The benchmark's read-stream probe (its bandwidth denominator), a library of its own.
PROBE_LIB = os.path.join(HERE, "libsomprobe.so")
PROBE_SOURCES = [os.path.join(CSRC, "probe.hip")]


def _compile(sources, out, verbose):
    tmp = out + ".tmp"
    cmd = [HIPCC, *FLAGS, *sources, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)


def build(verbose: bool = False) -> str:
    _compile(SOURCES, LIB, verbose)
    _compile(PROBE_SOURCES, PROBE_LIB, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
