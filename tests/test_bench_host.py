"""Host logic of bench.py, on the CPU: the one-GPU contract, the kernel
instance it names, and the roofline object built from committed profiles."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2202_01258_amd import rocprof_summary as R, workloads as W  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)


@pytest.mark.parametrize("name", W.ORDER)
def test_kernel_instance_names(name):
    """Test functions name the generation kernel's instance by its offspring per
    wave (one up to 2048 offspring, two up to 8192, four above); policies the
    rollout by its hidden width."""
    w = W.workload(name)
    dom, kname = bench.kernel_name_of(w)
    if w["task"] == W.MLP_SYNTH:
        assert (dom, kname) == ("rollout", f"k_rollout<{w['hid']}, false, false>")
    else:
        per = 1 if w["batch"] <= 2048 else (2 if w["batch"] <= 8192 else 4)
        assert (dom, kname) == ("vary_eval", f"k_vary_eval<{w['task']}, false, false, {per}>")


def test_committed_profiles_name_the_benchmarked_instance():
    """The counter summaries of the benchmark configuration record the kernel
    instance bench.py looks them up by."""
    for name in ("rastrigin_proj_cvt_b65536", "rastrigin_proj_cvt_b65536_spread"):
        w = W.workload(name)
        _, kname = bench.kernel_name_of(w)
        for kind in ("hbm_traffic", "sq_counters"):
            path = os.path.join(ROOT, "profiles", f"k_vary_eval_{name}_{kind}.txt")
            with open(path) as fh:
                tags = [ln.split(maxsplit=3) for ln in fh
                        if ln.startswith((R.TRAFFIC_TAG, R.VALU_TAG))]
            assert tags and all(t[3].strip() == kname for t in tags), path


def test_roofline_object_shape():
    """With a stand-in launch time the roofline object has the contract's fields;
    `bound` is the larger of the VALU and measured-HBM fractions when the
    recorded counters match the sources, and the byte model is secondary."""
    w = W.workload("rastrigin_proj_cvt_b65536")
    r = bench.roofline("rastrigin_proj_cvt_b65536", w, 0.060, None)
    for key in ("kernel", "bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert key in r
    assert r["hbm_model"]["note"].startswith("byte model")
    if r["valu"] is not None and r["hbm_measured"] is not None:
        fr = {"alu": r["valu"]["frac"], "hbm": r["hbm_measured"]["frac"]}
        assert r["bound"] == max(fr, key=fr.get)
        assert r["frac"] == pytest.approx(fr[r["bound"]])
    json.dumps(r)
