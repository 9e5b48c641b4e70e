"""Build the HIP library libleapquant.so in-tree for gfx950.

hipcc cross-compiles without a GPU.  Flags: -O3, IEEE fp32 division and square
root (hipcc's default), denormals kept, packed-fp32 instructions disabled.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libleapquant.so")
# measurement helpers for bench.py (not part of the method's C ABI)
BENCH_LIB = os.path.join(PKG, "libleapquant_bench.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def sources():
    return sorted(glob.glob(os.path.join(PKG, "csrc", "*.hip")))


# A build-time alternative of the library, for measuring one design choice
# against its alternative (never loaded unless named in LEAPQUANT_LIB):
# the decode's integer code product on the vector ALU instead of the matrix cores.
VALU_CP_LIB = os.path.join(PKG, "libleapquant_valucp.so")


def _compile(srcs, out, verbose, defines=()):
    tmp = out + ".tmp"
    cmd = [HIPCC, *FLAGS, *defines, "-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "csrc"),
           *srcs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), file=sys.stderr)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)


def build(verbose: bool = False) -> str:
    _compile(sources(), LIB, verbose)
    _compile(sorted(glob.glob(os.path.join(PKG, "bench_csrc", "*.hip"))), BENCH_LIB, verbose)
    return LIB


def build_valu_code_product(verbose: bool = False) -> str:
    _compile(sources(), VALU_CP_LIB, verbose, defines=("-DLQ_CODE_PRODUCT_VALU",))
    return VALU_CP_LIB


if __name__ == "__main__":
    if "--valu-code-product" in sys.argv:
        print(build_valu_code_product(verbose=True))
    else:
        print(build(verbose=True))
