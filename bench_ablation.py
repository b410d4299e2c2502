"""Fixed-budget batch-size ablation on Rastrigin and Sphere.

The experiment of the paper's Section 5.2 on this path: for each task and
batch size N_B, run MAP-Elites for a fixed number of evaluations H (20 million
for Rastrigin and Sphere), I = ceil(H / N_B) iterations with the first one
counted, over several seeds; then compare the final QD-scores of every pair of
batch sizes with the Wilcoxon rank-sum test and a Bonferroni correction for
the number of pairs.  The paper reports no significant difference (all
corrected p > 0.05).

QD-score (Eq. 1) needs non-negative objectives; Rastrigin and Sphere are
non-positive, so every filled cell's objective is shifted by the negated
minimum of the objective over the descriptor box [-5.12, 5.12]^n:
n (5.12^2 + 20) for Rastrigin and n 5.12^2 for Sphere.

  python bench_ablation.py [--tasks rastrigin sphere] [--batches 256 1024 ...]
                           [--seeds 10] [--evals 20000000] [--init LO HI]

--init replaces the first batch's uniform range (the configurations draw it
from [-0.1, 0.1), where the descriptor (theta_0, theta_1) starts inside a 2x2
block of cells; [-5.12, 5.12) starts it anywhere in the box).

Prints one JSON line per run, then one per task with the test results.
"""
from __future__ import annotations

import argparse
import itertools
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

TASKS = {"rastrigin": "rastrigin_grid_b128", "sphere": "sphere_grid_b16384"}


def log(msg: str):
    print(msg, file=sys.stderr, flush=True)


def offset_for(task: str, n: int) -> float:
    box = 5.12
    return n * (box * box + 20.0) if task == "rastrigin" else n * box * box


def run(w: dict, evals: int, offset: float) -> dict:
    import torch
    from paper_2202_01258_amd import qd

    iters = math.ceil(evals / w["batch"])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    a = qd.Archive(w, device="cuda:0")
    for g in range(1, iters):
        a.generation(g)
    st = a.stats(offset=offset)
    runtime = time.perf_counter() - t0
    del a
    return {"iterations": iters, "runtime_s": runtime, "qd_score": st["qd_score"],
            "coverage": st["num_occupied"], "best": st["best"]}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--tasks", nargs="+", default=["rastrigin", "sphere"])
    ap.add_argument("--batches", nargs="+", type=int, default=[256, 1024, 4096, 16384, 65536])
    ap.add_argument("--seeds", type=int, default=10)
    ap.add_argument("--evals", type=int, default=20_000_000)
    ap.add_argument("--init", nargs=2, type=float, metavar=("LO", "HI"))
    args = ap.parse_args()

    import torch
    from scipy import stats
    from paper_2202_01258_amd import workloads as W

    if not torch.cuda.is_available():
        print("bench_ablation.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    for task in args.tasks:
        base = TASKS[task]
        final = {}
        for nb in args.batches:
            final[nb] = []
            for seed in range(args.seeds):
                w = W.workload(base, batch=nb, seed=seed)
                if args.init:
                    w.update(init_lo=args.init[0], init_hi=args.init[1])
                off = offset_for(task, w["n"])
                r = run(w, args.evals, off)
                r.update(task=task, batch=nb, seed=seed, evals=args.evals, qd_offset=off,
                         init=[w["init_lo"], w["init_hi"]])
                print(json.dumps(r), flush=True)
                final[nb].append(r["qd_score"])
            log(f"ablation: {task} N_B={nb}: median QD-score "
                f"{sorted(final[nb])[len(final[nb]) // 2]:.6g} over {args.seeds} seeds")
        pairs = list(itertools.combinations(args.batches, 2))
        tests = []
        for b1, b2 in pairs:
            p = float(stats.ranksums(final[b1], final[b2]).pvalue)
            tests.append({"batches": [b1, b2], "p": p, "p_bonferroni": min(1.0, p * len(pairs))})
        worst = min(t["p_bonferroni"] for t in tests)
        print(json.dumps({"task": task, "evals": args.evals, "seeds": args.seeds,
                          "init": list(args.init) if args.init else None,
                          "medians": {str(b): sorted(v)[len(v) // 2] for b, v in final.items()},
                          "pairs": tests, "min_p_bonferroni": worst,
                          "significant_difference": worst <= 0.05}), flush=True)
        log(f"ablation: {task}: smallest Bonferroni-corrected rank-sum p = {worst:.3g}")


if __name__ == "__main__":
    main()
