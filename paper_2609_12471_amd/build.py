"""Build libkva.so (the HIP kernels and the C ABI) in-tree for gfx950.

    python -m paper_2609_12471_amd.build          # or build() from Python

Packed fp32 instructions are disabled for the device code
(-target-feature -packed-fp32-ops); floating-point contraction is off.
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libkva.so")
SOURCES = [os.path.join(CSRC, "kva_kernels.hip"), os.path.join(CSRC, "kva_prefix.hip"),
           os.path.join(CSRC, "kva_append.hip"), os.path.join(CSRC, "kva_prefill.hip"),
           os.path.join(CSRC, "kva_stream.hip"), os.path.join(CSRC, "kva_api.hip")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # no implicit contraction: the running maximum must be the rounded score
    # itself, so the maximum's own weight is exp2(0) = 1 exactly; wanted FMAs
    # are written explicitly
    "-ffp-contract=off",
    "-Wall", "-Wno-unused-function",
    "-I", INCLUDE, "-I", CSRC,
]


def build(verbose: bool = False, extra=()) -> str:
    """Compile every HIP source into paper_2609_12471_amd/libkva.so."""
    tmp = LIB + ".tmp"
    cmd = [HIPCC, *FLAGS, *extra, "-o", tmp, *SOURCES]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed building libkva.so")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
