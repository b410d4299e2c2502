"""Batch-size throughput sweep and runtime to a fixed evaluation budget.

The experiment of the paper's Section 5.3 (Figure 4, Table 1) on this path:
for N_B = 64, 128, ..., 131072 (doubling),

  * eval/s over N generations, the paper's definition mean_n(N_B / t_n), with
    t_n from HIP events around each generation, and, beside it, N_B N / T
    from the wall time of N back-to-back generations with nothing else on the
    stream;
  * runtime to H evaluations (10^6 by default): wall time of the whole run,
    first iteration (archive set-up and the random batch) included, for
    I = ceil(H / N_B) iterations, the first one counted (Section 4).

Default workloads: the Rastrigin-projection shape (n = 1000, CVT 10^4) and
the 27-64-64-8 policy shape (T = 250, CVT 1024).  One GPU.  With --seeds S
every (workload, N_B) runs for seeds 0 .. S-1 and the figures are the medians
over seeds (the paper reports medians over replications).  Prints one JSON
line per (workload, N_B) and a summary table on stderr.

  python bench_sweep.py [--workloads NAME ...] [--min 64] [--max 131072]
                        [--gens 100] [--evals 1000000] [--seeds 1]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def log(msg: str):
    print(msg, file=sys.stderr, flush=True)


def measure(w: dict, gens: int, evals: int) -> dict:
    import torch
    from paper_2202_01258_amd import qd

    nb = w["batch"]
    a = qd.Archive(w, device="cuda:0")
    s = a.stream
    # eval/s: a few untimed generations, then N back-to-back, then N with events
    g = 1
    for _ in range(3):
        a.generation(g)
        g += 1
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(gens):
        a.generation(g)
        g += 1
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(gens + 1)]
    ev[0].record(s)
    for k in range(gens):
        a.generation(g)
        g += 1
        ev[k + 1].record(s)
    torch.cuda.synchronize()
    t_n = [ev[k].elapsed_time(ev[k + 1]) * 1e-3 for k in range(gens)]
    del a
    # runtime to `evals` evaluations, the first iteration included
    iters = math.ceil(evals / nb)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    b = qd.Archive(w, device="cuda:0")
    for g in range(1, iters):
        b.generation(g)
    torch.cuda.synchronize()
    runtime = time.perf_counter() - t0
    st = b.stats()
    del b
    return {
        "batch": nb,
        "eval_per_s_paper": sum(nb / t for t in t_n) / len(t_n),
        "eval_per_s_wall": nb * gens / wall,
        "median_step_ms": sorted(t_n)[len(t_n) // 2] * 1e3,
        "iterations_to_budget": iters,
        "runtime_to_budget_s": runtime,
        "coverage_at_budget": st["num_occupied"],
        "qd_score_at_budget": st["qd_score"],
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workloads", nargs="+",
                    default=["rastrigin_proj_cvt_b65536", "mlp64_cvt_b8192"])
    ap.add_argument("--min", type=int, default=64)
    ap.add_argument("--max", type=int, default=131072)
    ap.add_argument("--gens", type=int, default=100)
    ap.add_argument("--evals", type=int, default=1_000_000)
    ap.add_argument("--seeds", type=int, default=1)
    args = ap.parse_args()

    import torch
    from paper_2202_01258_amd import workloads as W

    if not torch.cuda.is_available():
        print("bench_sweep.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    rows = []
    for name in args.workloads:
        nb = args.min
        while nb <= args.max:
            runs = []
            for seed in range(args.seeds):
                log(f"sweep: {name} N_B={nb} seed {seed}")
                runs.append(measure(W.workload(name, batch=nb, seed=seed), args.gens, args.evals))
            r = {k: (sorted(x[k] for x in runs)[len(runs) // 2] if isinstance(runs[0][k], float)
                     else runs[0][k]) for k in runs[0]}
            r.update(workload=name, evals_budget=args.evals, gens=args.gens, seeds=args.seeds,
                     per_seed_eval_per_s=[x["eval_per_s_paper"] for x in runs])
            print(json.dumps(r), flush=True)
            rows.append(r)
            nb *= 2
    log(f"{'workload':28s} {'N_B':>7s} {'eval/s (paper)':>15s} {'eval/s (wall)':>15s} "
        f"{'step ms':>9s} {'I':>6s} {'runtime s':>10s}")
    for r in rows:
        log(f"{r['workload']:28s} {r['batch']:7d} {r['eval_per_s_paper']:15.4g} "
            f"{r['eval_per_s_wall']:15.4g} {r['median_step_ms']:9.4f} "
            f"{r['iterations_to_budget']:6d} {r['runtime_to_budget_s']:10.3f}")


if __name__ == "__main__":
    main()
