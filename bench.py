"""Benchmark of one MAP-Elites generation step on one MI355X.

A step is one qd_generation() call: uniform selection, Iso+LineDD variation,
batched evaluation, descriptor -> cell and insertion, over one batch of N_B
offspring, with the archive resident in HBM.  The default workload is the
Rastrigin-projection configuration at N_B = 65536 (n = 1000, CVT of 10^4
cells).  Prints one JSON line.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                  [--no-cpu-baseline] [--cpu-generations G]

Throughput `value` = N_B * K / (wall time of the K timed steps), bracketed by
device synchronisation, with nothing else on the stream.  The paper's eval/s
(mean over steps of N_B / t_n) and the median step come from a second run of K
steps with a HIP event after each.  The roofline object is for the dominant
kernel, whose per-launch duration comes from start/stop HIP events attached to
each of its launches on its stream (hipExtLaunchKernelGGL) over a third run of
K steps.  Beside the bound the metric names (HBM bytes of the byte model, or
fp32 flops for policies) it carries two figures taken from the committed
rocprofv3 summaries under profiles/, each only while the kernel's sources
still hash to the value recorded with it: `traffic`, the measured HBM bytes
per launch, and `valu`, the kernel's VALU instructions per launch over the
same duration against one wave64 instruction per 2 cycles per SIMD.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "offspring evaluated+inserted/sec at 1 MI355X; % of peak HBM BW"
HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, 8 TB/s
FP32_PEAK_TFLOPS = 157.3     # MI355X fp32 vector (dual-issue / packed) peak
# VALU issue peak: 256 CUs x 4 SIMDs, one wave64 instruction per 2 cycles per
# SIMD at 2.4 GHz -- the rate at which fma alone gives the fp32 figure above
VALU_PEAK_PER_S = 256 * 4 * 2.4e9 / 2


def log(msg: str):
    print(msg, file=sys.stderr, flush=True)


def algorithmic_bytes(w: dict, n: int) -> dict:
    """Bytes each offspring must move at least (byte model).

    vary_eval: both parent rows (8n), objective and descriptor (4 + 4D), two
    parent indices (8), won flag (1).  Whole generation adds the cell index
    write and read (8), the key (8) and the winners' rows, which the
    benchmark reports separately through the measured insertion count."""
    D = w["D"]
    vary = 8 * n + 4 + 4 * D + 8 + 1
    gen = 8 * n + 4 * (1 + D) + 4 + 8
    return dict(vary_eval=vary, generation=gen, winner_row=4 * n + 4 + 4 * D)


def mlp_flops(w: dict) -> float:
    """fp32 flops of one rollout (2 per multiply-add), excluding tanh."""
    o, h, a, T = w["obs"], w["hid"], w["act"], w["T"]
    macs = h * o + h * h + a * h + o * o + o * a + a
    return 2.0 * macs * T


def cpu_baseline(w: dict, gens: int) -> dict:
    """The oracle, single-threaded, on a bounded sample of the same workload."""
    from oracle import oracle as O
    o = O.Oracle(w)
    t0 = time.perf_counter()
    if w["task"] == 3:
        # policies: a sample of individuals of the first batch is the unit
        import numpy as np
        o.setup()
        count = gens
        for j in range(count):
            o.offspring(0, j)
        dt = time.perf_counter() - t0
        return dict(value=count / dt, unit="offspring/s", cores=1, kind="oracle",
                    sample=f"{count} rollouts (T={w['T']}) of the first batch, one thread")
    o.init()
    t_init = time.perf_counter() - t0
    t1 = time.perf_counter()
    for g in range(1, gens + 1):
        o.generation(g)
    dt = time.perf_counter() - t1
    return dict(value=gens * w["batch"] / dt, unit="offspring/s", cores=1, kind="oracle",
                sample=f"{gens} full generations of N_B={w['batch']} after the first batch "
                       f"({t_init:.1f} s, untimed), one thread")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="rastrigin_proj_cvt_b65536")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-generations", type=int, default=4)
    ap.add_argument("--no-kernel-timing", action="store_true")
    ap.add_argument("--cvt-lloyd", type=int, nargs=2, metavar=("SAMPLES", "ITERS"),
                    help="build the CVT with Lloyd iterations over uniform points instead of "
                         "keeping the uniform centroids")
    ap.add_argument("--death", nargs=2, metavar=("MODE", "BELOW"),
                    help="policies: end episodes at failure (MODE 1 truncate, 2 discard) "
                         "when new-state component 0 drops below BELOW")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="also run 3 plain device-to-device copies of MIB MiB (the reference "
                         "kernel for scaling HBM byte counters) and exit after them")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the method shards as described in DESIGN.md, but only one GPU is used here)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2202_01258_amd import qd, workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration:
        nbytes = args.copy_calibration << 20
        src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"bench: copied {nbytes} bytes 3 times (counter calibration)")
        return
    w = W.workload(args.workload)
    if args.cvt_lloyd:
        w.update(cvt_samples=args.cvt_lloyd[0], cvt_iters=args.cvt_lloyd[1])
    if args.death:
        w.update(death_mode=int(args.death[0]), death_below=float(args.death[1]))
    n = W.genotype_len(w)
    nb = w["batch"]
    log(f"bench: workload {args.workload} N_B={nb} n={n} C={w['C']}; setting up")
    torch.cuda.synchronize()
    ts = time.perf_counter()
    a = qd.Archive(w, device="cuda:0")
    stream = a.stream
    stream.synchronize()
    setup_s = time.perf_counter() - ts
    g = 1
    for _ in range(args.warmup):
        a.generation(g)
        g += 1
    stream.synchronize()
    log(f"bench: {args.warmup} warmup steps done; timing {args.steps} steps")

    dominant = "rollout" if w["task"] == 3 else "vary_eval"
    # full name of the dominant kernel in profiler output, and the committed
    # HBM-counter summary for it on this workload (see rocprof_summary --traffic)
    kernel_name = (f"k_rollout<{w['hid']}, false, false>" if w["task"] == 3
                   else f"k_vary_eval<{w['task']}, false, false>")
    traffic_file = os.path.join(ROOT, "profiles", f"k_{dominant}_{args.workload}_hbm_traffic.txt")
    sq_file = os.path.join(ROOT, "profiles", f"k_{dominant}_{args.workload}_sq_counters.txt")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        a.generation(g)
        g += 1
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    wall = t1 - t0
    # Every event recorded on the stream between two kernels delays the second
    # by several microseconds, so the timed run above records none.  Per-step
    # times (for the paper's eval/s) come from a second run of the same number
    # of steps with an event after each step; the dominant kernel's launch
    # duration from a third, whose launches carry start/stop events of their
    # own; every kernel's from a fourth.
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    ev[0].record(stream)
    for k in range(args.steps):
        a.generation(g)
        g += 1
        ev[k + 1].record(stream)
    torch.cuda.synchronize()
    step_ms = [ev[k].elapsed_time(ev[k + 1]) for k in range(args.steps)]
    ktimes, breakdown = {}, {}
    if not args.no_kernel_timing:
        a.set_kernel_timing([dominant])
        a.kernel_times()
        for _ in range(args.steps):
            a.generation(g)
            g += 1
        ktimes = a.kernel_times()
        a.set_kernel_timing(["vary_eval", "rollout", "insert", "regen"])
        for _ in range(args.steps):
            a.generation(g)
            g += 1
        breakdown = a.kernel_times()
    a.set_kernel_timing([])
    st = a.stats()
    log(f"bench: timed region {wall * 1e3:.2f} ms; coverage {st['num_occupied']} cells")

    value = nb * args.steps / wall
    paper_evals = sum(nb / (t / 1e3) for t in step_ms) / len(step_ms)
    ms_per_step = wall * 1e3 / args.steps
    bytes_model = algorithmic_bytes(w, n)
    line = {
        "metric": METRIC, "value": value, "unit": "offspring/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded Philox streams; no dataset)",
        "config": {"workload": args.workload, "task": ["rastrigin", "sphere",
                   "rastrigin_projection", "mlp_policy"][w["task"]],
                   "batch": nb, "genotype_dim": n, "cells": w["C"],
                   "tessellation": "grid" if w["tess"] == 0 else "cvt",
                   "episode_len": w["T"] if w["task"] == 3 else None, "seed": w["seed"],
                   "cvt_lloyd": [w["cvt_samples"], w["cvt_iters"]] if w["cvt_iters"] else None,
                   "death": [w["death_mode"], w["death_below"]] if w["death_mode"] else None},
        "setup_s": setup_s,                       # archive set-up and the first batch
        "paper_eval_per_s": paper_evals,          # second run, per-step events
        "median_step_ms": sorted(step_ms)[len(step_ms) // 2],
        "archive": {"filled_cells": st["num_occupied"], "qd_score": st["qd_score"],
                    "best": st["best"]},
    }
    gen_bytes = bytes_model["generation"] * nb
    line["generation_hbm_frac"] = gen_bytes / (ms_per_step * 1e-3) / (HBM_PEAK_GBS * 1e9)
    if breakdown:
        line["kernel_ms_per_step"] = {k: (v[0] / v[1] if v[1] else 0.0)
                                      for k, v in breakdown.items() if v[1]}
    if ktimes:
        from paper_2202_01258_amd.rocprof_summary import recorded_traffic, recorded_valu
        traffic = recorded_traffic(traffic_file, kernel_name)
        valu_n = recorded_valu(sq_file, kernel_name)
        if w["task"] == 3:
            ms, cnt = ktimes["rollout"]
            avg = ms / cnt
            flops = mlp_flops(w) * nb
            ach = flops / (avg * 1e-3) / 1e12
            line["roofline"] = {"kernel": kernel_name, "bound": "alu", "achieved": ach,
                                "peak": FP32_PEAK_TFLOPS, "unit": "TFLOP/s",
                                "frac": ach / FP32_PEAK_TFLOPS, "traffic": traffic,
                                "kernel_avg_us": avg * 1e3}
        else:
            ms, cnt = ktimes["vary_eval"]
            avg = ms / cnt
            ach = bytes_model["vary_eval"] * nb / (avg * 1e-3) / 1e9
            line["roofline"] = {"kernel": kernel_name, "bound": "hbm", "achieved": ach,
                                "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                "frac": ach / HBM_PEAK_GBS, "traffic": traffic,
                                "kernel_avg_us": avg * 1e3,
                                "algorithmic_bytes_per_launch": bytes_model["vary_eval"] * nb}
        # the same launch against the VALU issue limit, from the committed
        # SQ_INSTS_VALU count of this kernel (null once the sources change)
        line["roofline"]["valu"] = None if valu_n is None else {
            "insts_per_launch": valu_n, "achieved": valu_n / (avg * 1e-3),
            "peak": VALU_PEAK_PER_S, "unit": "wave64 VALU instructions/s",
            "frac": valu_n / (avg * 1e-3) / VALU_PEAK_PER_S}
    if not args.no_cpu_baseline:
        log("bench: CPU baseline (oracle, one thread)")
        cb_w = dict(w)
        line["cpu_baseline"] = cpu_baseline(cb_w, args.cpu_generations if w["task"] != 3 else 4)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
