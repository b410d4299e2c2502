"""VALU issue-rate probe (gfx950): builds and runs bench_issue.hip.

  python bench_issue.py --build     compile ./bench_issue for gfx950 (no GPU needed)
  python bench_issue.py             run it (GPU) and print its table

The figures back the instruction-issue reading of the roofline of the
generation kernel and of the policy rollout: which VALU forms issue two per
slot, what a 64-bit multiply-add and a DPP-broadcast fma cost, and how the
rate of one wave's chains depends on the waves per SIMD.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "bench_issue.hip")
BIN = os.path.join(HERE, "bench_issue")


def build(verbose: bool = False) -> str:
    from paper_2202_01258_amd import build as libbuild
    cmd = [libbuild.hipcc(), f"--offload-arch={libbuild.ARCH}", "-O3", "-std=c++17",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", SRC, "-o", BIN + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(BIN + ".tmp", BIN)
    return BIN


def main() -> int:
    if "--build" in sys.argv[1:]:
        build(verbose=True)
        return 0
    if not os.path.exists(BIN):
        print("bench_issue is not built: run python bench_issue.py --build first", file=sys.stderr)
        return 2
    return subprocess.run([BIN]).returncode


if __name__ == "__main__":
    sys.exit(main())
