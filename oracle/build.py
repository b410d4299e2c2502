"""Builds the CPU oracle (test infrastructure only) into oracle/liboracle.so.

The oracle is plain C compiled without floating-point contraction or fast-math
so that every fused multiply-add in it is an explicit fmaf() call.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")
FLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
         "-Wall", "-Wextra", "-Wno-unused-parameter"]


def build(verbose: bool = False) -> str:
    src = os.path.join(HERE, "qd_oracle.c")
    tmp = LIB + ".tmp"
    cmd = ["gcc", *FLAGS, src, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
