"""Builds the CPU oracle (test infrastructure only) into oracle/liboracle.so.

The oracle is plain C compiled without floating-point contraction or fast-math
so that every fused multiply-add in it is an explicit fmaf() call.  OpenMP
runs its per-offspring loops on several threads; build(openmp=False, path=...)
makes the single-threaded build of the same source (the pragmas are ignored).
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")
FLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
         "-Wall", "-Wextra", "-Wno-unused-parameter"]


def build(verbose: bool = False, openmp: bool = True, path: str = LIB) -> str:
    src = os.path.join(HERE, "qd_oracle.c")
    tmp = path + ".tmp"
    cmd = ["gcc", *FLAGS, *(["-fopenmp"] if openmp else []), src, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, path)
    return path


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
