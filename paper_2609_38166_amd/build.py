"""Build the HIP library libleapquant.so in-tree for gfx950.

hipcc cross-compiles without a GPU.  Flags: -O3, IEEE fp32 division and square
root (hipcc's default), denormals kept, packed-fp32 instructions disabled.
Each source is compiled to an object of its own (with the scheduler options of
SCHED below) and the objects are linked into the library.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libleapquant.so")
# measurement helpers for bench.py (not part of the method's C ABI)
BENCH_LIB = os.path.join(PKG, "libleapquant_bench.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]

# Machine scheduler options per source file (the LLVM AMDGPU backend's), each
# measured against the default on the KDA workload (8192 tiles, W = 64, r = 8):
#  - decode: the max-ILP strategy, 1.7% less time per launch over the window
#    positions (2.2% on the GQA GDN layer), no spill;
#  - tile kernel (quantize, commit): the AMDGPU register-pressure trackers,
#    6% less time per commit (quantize within 2%).
SCHED = {
    "lq_decode.hip": ["-mllvm", "-amdgpu-sched-strategy=max-ilp"],
    "lq_tile.hip": ["-mllvm", "-amdgpu-use-amdgpu-trackers"],
}


def sources():
    return sorted(glob.glob(os.path.join(PKG, "csrc", "*.hip")))


# A build-time alternative of the library, for measuring one design choice
# against its alternative (never loaded unless named in LEAPQUANT_LIB):
# the decode's integer code product on the vector ALU instead of the matrix cores.
VALU_CP_LIB = os.path.join(PKG, "libleapquant_valucp.so")


def _compile(srcs, out, verbose, defines=()):
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "csrc")]
    with tempfile.TemporaryDirectory() as td:
        def obj(src):
            o = os.path.join(td, os.path.basename(src) + ".o")
            cmd = [HIPCC, *FLAGS, *SCHED.get(os.path.basename(src), []), *defines, *inc, "-c", src, "-o", o]
            if verbose:
                print(" ".join(cmd), file=sys.stderr)
            subprocess.run(cmd, check=True)
            return o
        with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
            objs = list(ex.map(obj, srcs))
        tmp = out + ".tmp"
        cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
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
