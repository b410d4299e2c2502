"""Benchmark of one MAP-Elites generation step on one MI355X.

A step is one qd_generation() call: uniform selection, Iso+LineDD variation,
batched evaluation, descriptor -> cell and insertion, over one batch of N_B
offspring, with the archive resident in HBM.  The default workload is the
Rastrigin-projection configuration at N_B = 65536 (n = 1000, CVT of 10^4
cells).  Prints one JSON line.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                  [--no-cpu-baseline] [--cpu-generations G] [--no-populated]

Throughput `value` = N_B * K / (wall time of the K timed steps), bracketed by
device synchronisation, with nothing else on the stream.  Before the W counted
warm-up steps, untimed generations run for at least SETTLE_S seconds (`settle`
in the line) so that the GPU's clocks are steady when the timed region starts.  The paper's eval/s
(mean over steps of N_B / t_n) and the median step come from a second run of K
steps with a HIP event after each.  The roofline object is for the dominant
kernel, whose per-launch duration comes from start/stop HIP events attached to
each of its launches on its stream (hipExtLaunchKernelGGL) over a third run of
K steps.  Its `bound` is the one the counters show: fp32 flops for policy
rollouts; for the test functions the larger of the VALU issue fraction
(SQ_INSTS_VALU per launch) and the measured HBM fraction (FETCH_SIZE +
WRITE_SIZE bytes per launch), both read from the committed rocprofv3
summaries under profiles/ while the kernel's sources still hash to the value
recorded with them (else null); the byte model of the generation is kept as a
secondary, labelled figure, and a plain device copy calibrates what HBM
bandwidth a kernel can reach.  `populated` repeats the measurement on the same
shape with a spread first batch (nearly every cell filled, distinct parents).
`cpu_baseline` is the oracle on every host thread and on one.
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
# untimed generations before the counted warm-up, so that clocks are steady
SETTLE_S = 0.25


def log(msg: str):
    print(msg, file=sys.stderr, flush=True)


def algorithmic_bytes(w: dict, n: int) -> dict:
    """Bytes each offspring must move at least (the byte model: every parent row read from HBM).

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


def host_info() -> dict:
    """The host the CPU baseline ran on: logical CPUs, the model name, and the
    OpenMP thread limit in force."""
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "cpu_model": model,
            "omp_num_threads": os.environ.get("OMP_NUM_THREADS")}


def cpu_baseline(w: dict, gens: int) -> dict:
    """The oracle on a bounded sample of the same workload, on every thread
    OpenMP gives it (the per-offspring loops; insertion stays sequential) and
    on one thread.  `value` is the all-threads rate."""
    from oracle import oracle as O
    import numpy as np
    full = O.set_threads(0)
    out = {}
    for threads in (full, 1):
        O.set_threads(threads)
        o = O.Oracle(w)
        if w["task"] == 3:
            # policies: first-batch rollouts are the unit (a generation of
            # N_B rollouts would take minutes)
            o.setup()
            count = max(8, 4 * threads)
            t0 = time.perf_counter()
            o.offspring_many(0, np.arange(count))
            dt = time.perf_counter() - t0
            rate, sample = count / dt, f"{count} rollouts (T={w['T']}) of the first batch"
        else:
            t0 = time.perf_counter()
            o.init()
            t_init = time.perf_counter() - t0
            g_run = gens if threads == 1 else 2 * gens
            t1 = time.perf_counter()
            for g in range(1, g_run + 1):
                o.generation(g)
            dt = time.perf_counter() - t1
            rate = g_run * w["batch"] / dt
            sample = (f"{g_run} full generations of N_B={w['batch']} after the first batch "
                      f"({t_init:.1f} s, untimed)")
        out[threads] = dict(value=rate, cores=threads, seconds=dt, sample=sample)
        del o
    O.set_threads(full)
    top = out[full]
    return dict(value=top["value"], unit="offspring/s", cores=full, kind="oracle",
                sample=top["sample"] + f", {full} threads",
                single_thread=dict(value=out[1]["value"], cores=1, sample=out[1]["sample"]),
                host=host_info())


def copy_calibration(mib: int = 1024, reps: int = 20) -> dict:
    """Achieved bandwidth of a plain device-to-device copy of `mib` MiB
    (bytes read + written per second), timed with events."""
    import torch
    n = (mib << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    gbs = 2.0 * (mib << 20) / (ms * 1e-3) / 1e9
    del src, dst
    return {"bytes_moved": 2 * (mib << 20), "ms": ms, "achieved_gbs": gbs,
            "frac_of_peak": gbs / HBM_PEAK_GBS}


def kernel_name_of(w: dict) -> tuple[str, str]:
    """(timing key, profiler name) of the dominant kernel of a workload."""
    if w["task"] == 3:
        return "rollout", f"k_rollout<{w['hid']}, false, false>"
    from paper_2202_01258_amd import qd
    return "vary_eval", f"k_vary_eval<{w['task']}, false, false, {qd.offspring_per_wave(w['batch'])}>"


def measure(name: str, w: dict, steps: int, warmup: int, kernel_timing: bool = True) -> dict:
    """Set-up, warm-up, then `steps` timed generations of workload `w`, with
    the per-step, per-kernel and dominant-kernel timings described above."""
    import torch
    from paper_2202_01258_amd import qd, workloads as W
    n = W.genotype_len(w)
    nb = w["batch"]
    log(f"bench: workload {name} N_B={nb} n={n} C={w['C']}; setting up")
    torch.cuda.synchronize()
    ts = time.perf_counter()
    a = qd.Archive(w, device="cuda:0")
    stream = a.stream
    stream.synchronize()
    setup_s = time.perf_counter() - ts
    filled_after_first = a.stats()["num_occupied"]
    g = 1
    # The GPU reaches its steady clocks only after some tens of milliseconds
    # of load (measured: 76.7 us per step after 5 warm-up steps, 66.3 us after
    # 1000, for the Rastrigin-projection configuration), so untimed
    # generations run for at least SETTLE_S seconds before the W counted
    # warm-up steps; the timed region is unchanged (exactly K steps).
    t_set = time.perf_counter()
    settle_gens = 0
    chunk = 1
    while time.perf_counter() - t_set < SETTLE_S:
        a.generations(g, chunk)
        g += chunk
        settle_gens += chunk
        stream.synchronize()
        chunk = min(2 * chunk, 64)
    settle_s = time.perf_counter() - t_set
    for _ in range(warmup):
        a.generation(g)
        g += 1
    stream.synchronize()
    log(f"bench: {warmup} warmup steps done; timing {steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        a.generation(g)
        g += 1
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # Every event recorded on the stream between two kernels delays the second
    # by several microseconds, so the timed run above records none.  Per-step
    # times (for the paper's eval/s) come from a second run of the same number
    # of steps with an event after each step; the dominant kernel's launch
    # duration from a third, whose launches carry start/stop events of their
    # own; every kernel's from a fourth.
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ev[0].record(stream)
    for k in range(steps):
        a.generation(g)
        g += 1
        ev[k + 1].record(stream)
    torch.cuda.synchronize()
    step_ms = [ev[k].elapsed_time(ev[k + 1]) for k in range(steps)]
    dom, _ = kernel_name_of(w)
    ktimes, breakdown = {}, {}
    if kernel_timing:
        a.set_kernel_timing([dom])
        a.kernel_times()
        for _ in range(steps):
            a.generation(g)
            g += 1
        ktimes = a.kernel_times()
        a.set_kernel_timing(["vary_eval", "rollout", "insert", "regen"])
        for _ in range(steps):
            a.generation(g)
            g += 1
        breakdown = a.kernel_times()
    a.set_kernel_timing([])
    st = a.stats()
    log(f"bench: timed region {wall * 1e3:.2f} ms; coverage {st['num_occupied']} cells")
    out = dict(value=nb * steps / wall, ms_per_step=wall * 1e3 / steps, setup_s=setup_s,
               settle={"seconds": settle_s, "generations": settle_gens},
               paper_eval_per_s=sum(nb / (t / 1e3) for t in step_ms) / len(step_ms),
               median_step_ms=sorted(step_ms)[len(step_ms) // 2],
               archive={"filled_cells": st["num_occupied"], "qd_score": st["qd_score"],
                        "best": st["best"], "filled_after_first_batch": filled_after_first})
    if breakdown:
        out["kernel_ms_per_step"] = {k: (v[0] / v[1] if v[1] else 0.0)
                                     for k, v in breakdown.items() if v[1]}
    if ktimes:
        ms, cnt = ktimes[dom]
        out["kernel_avg_ms"] = ms / cnt
    return out


def roofline(name: str, w: dict, kernel_avg_ms: float, copy: dict | None) -> dict:
    """The dominant kernel against the bound its counters show.

    Policies: fp32 flops of the rollouts per launch over the event-timed
    launch duration against 157.3 TFLOP/s.  Test functions: VALU wave64
    instructions per launch (SQ_INSTS_VALU from the committed counter summary
    of this kernel and workload) against the issue peak, and the HBM bytes per
    launch that FETCH_SIZE + WRITE_SIZE measured (committed traffic summary)
    against 8 TB/s; `bound` is whichever fraction is larger.  The byte model
    (two parent rows and the per-offspring records, whether or not the parent
    rows come from HBM) is kept as a labelled secondary figure.  Counter-based
    figures are null once the kernel's sources differ from those profiled."""
    from paper_2202_01258_amd import workloads as W
    from paper_2202_01258_amd.rocprof_summary import recorded_traffic, recorded_valu
    dom, kname = kernel_name_of(w)
    n, nb = W.genotype_len(w), w["batch"]
    avg_s = kernel_avg_ms * 1e-3
    traffic_file = os.path.join(ROOT, "profiles", f"k_{dom}_{name}_hbm_traffic.txt")
    sq_file = os.path.join(ROOT, "profiles", f"k_{dom}_{name}_sq_counters.txt")
    traffic = recorded_traffic(traffic_file, kname)
    valu_n = recorded_valu(sq_file, kname)
    hbm_meas = None if traffic is None else {
        "bytes_per_launch": traffic, "achieved": traffic / avg_s / 1e9, "peak": HBM_PEAK_GBS,
        "unit": "GB/s", "frac": traffic / avg_s / 1e9 / HBM_PEAK_GBS,
        "source": os.path.relpath(traffic_file, ROOT)}
    valu = None if valu_n is None else {
        "insts_per_launch": valu_n, "achieved": valu_n / avg_s, "peak": VALU_PEAK_PER_S,
        "unit": "wave64 VALU instructions/s", "frac": valu_n / avg_s / VALU_PEAK_PER_S,
        "source": os.path.relpath(sq_file, ROOT)}
    if w["task"] == 3:
        flops = mlp_flops(w) * nb
        ach = flops / avg_s / 1e12
        r = {"kernel": kname, "bound": "alu", "achieved": ach, "peak": FP32_PEAK_TFLOPS,
             "unit": "TFLOP/s", "frac": ach / FP32_PEAK_TFLOPS, "traffic": traffic,
             "kernel_avg_us": kernel_avg_ms * 1e3, "flops_per_launch": flops,
             "valu": valu, "hbm_measured": hbm_meas}
    else:
        model = algorithmic_bytes(w, n)["vary_eval"] * nb
        hbm_model = {"bytes_per_launch": model, "achieved": model / avg_s / 1e9,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": model / avg_s / 1e9 / HBM_PEAK_GBS,
                     "note": "byte model: both parent rows per offspring counted as HBM reads"}
        if valu is not None and (hbm_meas is None or valu["frac"] >= hbm_meas["frac"]):
            r = {"kernel": kname, "bound": "alu", "achieved": valu["achieved"],
                 "peak": VALU_PEAK_PER_S, "unit": valu["unit"], "frac": valu["frac"]}
        elif hbm_meas is not None:
            r = {"kernel": kname, "bound": "hbm", "achieved": hbm_meas["achieved"],
                 "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": hbm_meas["frac"]}
        else:
            r = {"kernel": kname, "bound": None, "achieved": None, "peak": None,
                 "unit": None, "frac": None}
        r.update({"traffic": traffic, "kernel_avg_us": kernel_avg_ms * 1e3, "valu": valu,
                  "hbm_measured": hbm_meas, "hbm_model": hbm_model})
    if copy is not None:
        r["copy_calibration"] = copy
    return r


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="rastrigin_proj_cvt_b65536")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-generations", type=int, default=4)
    ap.add_argument("--no-kernel-timing", action="store_true")
    ap.add_argument("--no-populated", action="store_true",
                    help="skip the second measurement on the populated archive")
    ap.add_argument("--cvt-lloyd", type=int, nargs=2, metavar=("SAMPLES", "ITERS"),
                    help="build the CVT with Lloyd iterations over uniform points instead of "
                         "keeping the uniform centroids")
    ap.add_argument("--death", nargs=2, metavar=("MODE", "BELOW"),
                    help="policies: end episodes at failure (MODE 1 truncate, 2 discard) "
                         "when new-state component 0 drops below BELOW")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run 3 plain device-to-device copies of MIB MiB (the reference "
                         "kernel for scaling HBM byte counters) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(this path runs and is measured on a single GPU)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2202_01258_amd import workloads as W

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
    kt = not args.no_kernel_timing
    m = measure(args.workload, w, args.steps, args.warmup, kt)
    copy = copy_calibration() if kt else None
    line = {
        "metric": METRIC, "value": m["value"], "unit": "offspring/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": m["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded Philox streams; no dataset)",
        "config": {"workload": args.workload, "task": ["rastrigin", "sphere",
                   "rastrigin_projection", "mlp_policy"][w["task"]],
                   "batch": nb, "genotype_dim": n, "cells": w["C"],
                   "tessellation": "grid" if w["tess"] == 0 else "cvt",
                   "episode_len": w["T"] if w["task"] == 3 else None, "seed": w["seed"],
                   "init_mode": w["init_mode"],
                   "cvt_lloyd": [w["cvt_samples"], w["cvt_iters"]] if w["cvt_iters"] else None,
                   "death": [w["death_mode"], w["death_below"]] if w["death_mode"] else None},
    }
    for k in ("setup_s", "settle", "paper_eval_per_s", "median_step_ms", "archive",
              "kernel_ms_per_step"):
        if k in m:
            line[k] = m[k]
    if "kernel_avg_ms" in m:
        line["roofline"] = roofline(args.workload, w, m["kernel_avg_ms"], copy)
    # The same generation step on an archive whose cells are nearly all
    # filled (the configuration's shape with a spread first batch): parents
    # are distinct rows, and winners are regenerated in every generation.
    spread = args.workload + "_spread"
    if not args.no_populated and spread in W.WORKLOADS:
        ws = W.workload(spread)
        mp = measure(spread, ws, args.steps, args.warmup, kt)
        pop = {"workload": spread, "value": mp["value"], "unit": "offspring/s",
               "ms_per_step": mp["ms_per_step"], "median_step_ms": mp["median_step_ms"],
               "settle": mp["settle"], "archive": mp["archive"]}
        if "kernel_ms_per_step" in mp:
            pop["kernel_ms_per_step"] = mp["kernel_ms_per_step"]
        if "kernel_avg_ms" in mp:
            pop["roofline"] = roofline(spread, ws, mp["kernel_avg_ms"], None)
        line["populated"] = pop
    if not args.no_cpu_baseline:
        log("bench: CPU baseline (the oracle, all threads then one thread)")
        line["cpu_baseline"] = cpu_baseline(dict(w), args.cpu_generations)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
