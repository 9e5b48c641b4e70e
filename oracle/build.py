"""Build the CPU oracle shared library (test infrastructure only).

The oracle is plain C compiled with gcc, strict IEEE arithmetic (no fast-math,
no FMA contraction), OpenMP across independent tiles.  `lq_oracle.c` is
compiled twice: once with double arithmetic (the oracle, symbols ``lqo64_*``)
and once with float arithmetic (an fp32 twin for self-checks, ``lqo32_*``).
"""
from __future__ import annotations

import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liblqoracle.so")

CFLAGS = ["-O2", "-std=c11", "-fPIC", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
          "-Wall", "-Wextra", "-Wno-unused-parameter"]


def build(verbose: bool = False) -> str:
    """Compile the oracle into oracle/liblqoracle.so and return its path."""
    with tempfile.TemporaryDirectory() as tmp:
        objs = []
        units = [
            ("lq_formats.c", [], "fmt.o"),
            ("lq_oracle.c", ["-DOQ_REAL=double", "-DOQ(n)=lqo64_##n"], "o64.o"),
            ("lq_oracle.c", ["-DOQ_REAL=float", "-DOQ(n)=lqo32_##n"], "o32.o"),
        ]
        for src, defs, obj in units:
            out = os.path.join(tmp, obj)
            cmd = ["gcc", *CFLAGS, *defs, "-c", os.path.join(HERE, src), "-o", out]
            if verbose:
                print(" ".join(cmd), file=sys.stderr)
            subprocess.run(cmd, check=True)
            objs.append(out)
        tmp_lib = LIB + ".tmp"
        subprocess.run(["gcc", "-shared", "-fopenmp", "-o", tmp_lib, *objs, "-lm"], check=True)
        os.replace(tmp_lib, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
