"""Build step for libfleetsieve: compiles the gfx950 kernels and the C-ABI
host runtime into ``paper_2608_19659_amd/libfleetsieve.so`` with hipcc.

Flags that matter for the numerics: no fused multiply-add contraction and no
fast-math, so every binary32 multiply and every quotient rounds exactly as
the C ABI documents.  Packed FP32 instructions are disabled."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libfleetsieve.so")
SOURCES = [os.path.join(CSRC, "fs_kernels.hip"), os.path.join(CSRC, "fs_api.cpp")]

HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    "-I", INCLUDE, "-I", CSRC,
]


def hipcc() -> str:
    return os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def build_library(extra_flags=(), out: str = LIB, verbose: bool = False) -> str:
    """Compile libfleetsieve.so (always recompiles)."""
    tmp = out + ".tmp"
    cmd = [hipcc(), *HIP_FLAGS, *extra_flags, *SOURCES, "-o", tmp]
    if verbose:
        print(" ".join(cmd), file=sys.stderr)
    subprocess.run(cmd, check=True, cwd=HERE)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build_library(verbose=True))
