"""GPU parity on the cases random inputs never reach, through the C ABI.

* Ties (Algorithm 1, Appendix A.4 ii): many offspring with the same
  objective in one empty cell -- the lowest batch index must take it; and
  offspring that copy their parents exactly (sigma_1 = sigma_2 = 0) tie with
  the incumbents, which must keep their cells (strictly greater replaces),
  leaving the archive bit-identical.
* Four-dimensional CVTs with the policy descriptors spread over the whole
  unit box (the box narrowed around where they lie): the LDS insertion at
  2048 cells, the ring search at 2049 and 10^4 cells, every cell against the
  oracle's brute-force nearest centroid.
* Repeatability: the same generations on a stream restricted to a few
  compute units (a different schedule of workgroups and atomics) give the
  same archive bit for bit.
* Checkpoint and resume: the archive region of the workspace and g copied
  out, restored into a fresh archive, continued -- bit-identical to a run
  that was never interrupted (the archive is static arrays, Appendix A.1).
"""
import ctypes as C

import numpy as np
import pytest

from oracle import oracle as O
from paper_2202_01258_amd import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def qd():
    from paper_2202_01258_amd import qd as Q
    return Q


def say(msg):
    print(msg, flush=True)


def assert_archive_equal(gpu, ora, n, what=""):
    np.testing.assert_array_equal(gpu["occ"], ora["occ"], err_msg=f"occupancy {what}")
    filled = ora["occ"] == 1
    np.testing.assert_array_equal(gpu["fit"][filled], ora["fit"][filled], err_msg=f"fit {what}")
    np.testing.assert_array_equal(gpu["desc"][filled], ora["desc"][filled], err_msg=f"desc {what}")
    np.testing.assert_array_equal(gpu["geno"][filled, :n], ora["geno"][filled, :n],
                                  err_msg=f"genotypes {what}")


def check_first_batch(w):
    a = qd().Archive(w, keep_offspring=True)
    o = O.Oracle(w)
    o.init()
    gb, ob = a.last_batch(), o.last_batch()
    np.testing.assert_array_equal(gb["geno"], o.last_offspring())
    np.testing.assert_array_equal(gb["fit"].view(np.uint32), ob["fit"].view(np.uint32))
    np.testing.assert_array_equal(gb["cell"], ob["cell"])
    np.testing.assert_array_equal(gb["won"], ob["won"])
    assert_archive_equal(a.snapshot(), o.archive(), o.n, "first batch")
    return a, o, gb


# ----------------------------------------------------------------- ties
# the fp32 number one step above 0.3: a first-batch box one fp32 step wide
ONE_STEP = float(np.nextafter(np.float32(0.3), np.float32(1.0)))


@pytest.mark.parametrize("name,kw", [
    # Sphere, n = 2, genes 0.3 or one fp32 step above: three objective values
    # (272 offspring tie at the top), every offspring in one grid cell
    ("sphere_grid_b16384", dict(n=2, batch=1000, init_lo=0.3, init_hi=ONE_STEP)),
    # Rastrigin, n = 4, the same: three objective values, 400 tied at the top
    ("rastrigin_grid_b128", dict(n=4, batch=3001, init_lo=0.3, init_hi=ONE_STEP)),
    # Sphere at 0 with denormal genes: every objective is -0.0
    ("sphere_grid_b16384", dict(n=8, batch=777, init_lo=0.0, init_hi=1e-45)),
])
def test_ties_in_an_empty_cell_go_to_the_lowest_index(name, kw):
    w = W.workload(name, **kw)
    say(f"ties in an empty cell: {name} {kw}")
    a, o, gb = check_first_batch(w)
    cells = np.unique(gb["cell"])
    assert cells.size == 1, cells                     # one cell for the whole batch
    best = gb["fit"].max()
    tied = np.nonzero(gb["fit"] == best)[0]
    assert tied.size >= 2                             # a real tie at the top
    assert np.nonzero(gb["won"])[0].tolist() == [tied[0]]
    # a generation from that archive, driven, still bit-exact
    pre = a.snapshot()
    a.generation(1)
    g1 = a.last_batch()
    o.set_archive(pre["geno"], pre["fit"], pre["desc"], pre["occ"])
    cell, won = o.insert_driven(g1["fit"], g1["desc"], g1["geno"])
    np.testing.assert_array_equal(g1["cell"], cell)
    np.testing.assert_array_equal(g1["won"], won)
    assert_archive_equal(a.snapshot(), o.archive(), o.n, "after a generation")


@pytest.mark.parametrize("name,kw", [
    ("rastrigin_proj_cvt_b65536", dict(n=64, batch=2000, C=500, init_mode=1, seed=5)),
    ("sphere_grid_b16384", dict(batch=3000, init_lo=-5.12, init_hi=5.12, seed=7)),
    ("mlp64_cvt_b8192", dict(batch=48, T=8, C=64, seed=3, lo=(0.4994, 0.4952, 0.4951, 0.4984),
                             hi=(0.5039, 0.5010, 0.4995, 0.5030))),
])
def test_ties_with_incumbents_keep_the_archive(name, kw):
    """sigma_1 = sigma_2 = 0: every offspring is a copy of its first parent,
    evaluates to the parent's objective and descriptor, lands in the
    parent's cell and ties with the incumbent -- which keeps it."""
    w = W.workload(name, iso_sigma=0.0, line_sigma=0.0, **kw)
    say(f"ties with incumbents: {name} {kw}")
    a = qd().Archive(w, keep_offspring=True)
    o = O.Oracle(w)
    o.init()
    before = a.snapshot()
    assert_archive_equal(before, o.archive(), o.n, "first batch")
    assert before["occ"].sum() >= 2
    for g in (1, 2, 3):
        a.generation(g)
        o.generation(g)
        gb = a.last_batch()
        par = gb["parents"][:, 0]
        np.testing.assert_array_equal(gb["cell"], par)             # its parent's cell
        np.testing.assert_array_equal(gb["fit"], before["fit"][par])
        assert not gb["won"].any()
        np.testing.assert_array_equal(gb["won"], o.last_batch()["won"])
        now = a.snapshot()
        for k in ("key", "fit", "desc", "geno", "slot", "occ_list"):
            np.testing.assert_array_equal(now[k], before[k], err_msg=f"{k} g={g}")


# ----------------------------------------------------------- 4-D CVT spread
# the 0.5% and 99.5% quantiles per dimension of the first-batch policy
# descriptors (27-64-64-8, T = 8, seed 3; the oracle's): normalised by this
# box they cover [0, 1]^4 and, two generations on, [-0.9, 1.8]^4
SPREAD_LO = (0.4994, 0.4952, 0.4951, 0.4984)
SPREAD_HI = (0.5039, 0.5010, 0.4995, 0.5030)


@pytest.mark.parametrize("C", [2048, 2049, 10000])
def test_four_dimensional_cvt_over_the_whole_box(C):
    w = W.workload("mlp64_cvt_b8192", batch=512, T=8, C=C, lo=SPREAD_LO, hi=SPREAD_HI, seed=3)
    say(f"4-D CVT spread C={C}")
    a, o, gb = check_first_batch(w)
    u = (gb["desc"] - np.float32(SPREAD_LO)) / (np.float32(SPREAD_HI) - np.float32(SPREAD_LO))
    assert (u.min(0) < 0.15).all() and (u.max(0) > 0.85).all(), (u.min(0), u.max(0))
    assert np.unique(gb["cell"]).size > 150
    cent = o.centroids()
    for g in (1, 2):
        pre = a.snapshot()
        a.generation(g)
        g1 = a.last_batch()
        o.set_archive(pre["geno"], pre["fit"], pre["desc"], pre["occ"])
        cell, won = o.insert_driven(g1["fit"], g1["desc"], g1["geno"])
        np.testing.assert_array_equal(g1["cell"], cell)         # brute-force nearest centroid
        np.testing.assert_array_equal(g1["won"], won)
        assert_archive_equal(a.snapshot(), o.archive(), o.n, f"generation {g}")
    # spot check of the brute force itself against an fp64 argmin
    un = (g1["desc"] - np.float32(SPREAD_LO)) / (np.float32(SPREAD_HI) - np.float32(SPREAD_LO))
    d2 = ((un[:64, None, :].astype(np.float64) - cent[None, :, :]) ** 2).sum(-1)
    agree = np.argmin(d2, 1) == g1["cell"][:64]
    assert agree.mean() > 0.95


# ----------------------------------------------------------- repeatability
def masked_stream(n_cus):
    """A HIP stream whose kernels run on compute units 0 .. n_cus - 1 only
    (hipExtStreamCreateWithCUMask), at the default priority."""
    hip = C.CDLL("libamdhip64.so")
    hip.hipExtStreamCreateWithCUMask.argtypes = [C.POINTER(C.c_void_p), C.c_uint32,
                                                 C.POINTER(C.c_uint32)]
    words = 8
    mask = (C.c_uint32 * words)()
    for c in range(n_cus):
        mask[c // 32] |= 1 << (c % 32)
    s = C.c_void_p()
    torch.cuda.synchronize()
    assert hip.hipExtStreamCreateWithCUMask(C.byref(s), words, mask) == 0
    return hip, s


@pytest.mark.parametrize("name,kw", [("rastrigin_proj_cvt_b65536", {}),
                                     ("mlp64_cvt_b8192", {}),
                                     ("rastrigin_proj_cvt_b65536", dict(init_mode=1)),
                                     # one and two offspring per wave, whole-box first batch
                                     ("rastrigin_grid_b128", dict(batch=2000, init_lo=-5.12,
                                                                  init_hi=5.12, seed=8)),
                                     ("sphere_grid_b16384", dict(batch=6000, init_lo=-5.12,
                                                                 init_hi=5.12, seed=9))])
def test_generations_repeat_on_a_few_compute_units(name, kw):
    w = W.workload(name, **kw)
    say(f"repeatability on 16 compute units: {name} {kw}")
    ref = qd().Archive(w)
    ref.generations(1, 2)
    hip, s = masked_stream(16)
    try:
        ext = torch.cuda.ExternalStream(s.value)
        a = qd().Archive(w, stream=ext)
        a.generations(1, 2)
        ext.synchronize()
        sa, sr = a.snapshot(), ref.snapshot()
        for k in ("key", "fit", "desc", "geno", "slot", "occ_list"):
            np.testing.assert_array_equal(sa[k], sr[k], err_msg=k)
        la, lr = a.last_batch(), ref.last_batch()
        for k in ("parents", "fit", "desc", "cell", "won"):
            np.testing.assert_array_equal(la[k], lr[k], err_msg=k)
        del a
    finally:
        torch.cuda.synchronize()
        hip.hipStreamDestroy.argtypes = [C.c_void_p]
        hip.hipStreamDestroy(s)


# ------------------------------------------------------ checkpoint / resume
STATE = ("key", "fit", "desc", "slot", "geno", "occ_list", "counters")


@pytest.mark.parametrize("name,kw", [("rastrigin_proj_cvt_b65536", dict(batch=3000, n=300)),
                                     ("rastrigin_proj_cvt_b65536", dict(batch=2000, n=64, C=500,
                                                                        init_mode=1)),
                                     ("mlp64_cvt_b8192", dict(batch=40, T=30))])
def test_checkpoint_and_resume(name, kw):
    w = W.workload(name, **kw)
    say(f"checkpoint/resume: {name} {kw}")
    whole = qd().Archive(w)
    whole.generations(1, 6)
    part = qd().Archive(w)
    part.generations(1, 3)
    part.stream.synchronize()
    saved = {k: part.views()[k].cpu().clone() for k in STATE}
    g_next = 4
    del part
    fresh = qd().Archive(w, device="cuda:0")          # its own first batch, then overwritten
    fresh.stream.synchronize()
    v = fresh.views()
    for k in STATE:
        v[k].copy_(saved[k].to(v[k].device))
    torch.cuda.synchronize()
    fresh.generations(g_next, 3)
    sf, sw = fresh.snapshot(), whole.snapshot()
    for k in ("key", "fit", "desc", "geno", "slot", "occ_list"):
        np.testing.assert_array_equal(sf[k], sw[k], err_msg=k)
    lf, lw = fresh.last_batch(), whole.last_batch()
    for k in ("parents", "fit", "desc", "cell", "won"):
        np.testing.assert_array_equal(lf[k], lw[k], err_msg=k)
    assert fresh.stats()["qd_score"] == whole.stats()["qd_score"]


CHILD = r"""
import sys, numpy as np
sys.path.insert(0, sys.argv[1])
from paper_2202_01258_amd import qd, workloads as W
out = {}
for k, (name, kw) in enumerate([("rastrigin_proj_cvt_b65536", {}), ("mlp64_cvt_b8192", {})]):
    a = qd.Archive(W.workload(name, **kw))
    a.generations(1, 2)
    s, b = a.snapshot(), a.last_batch()
    for f in ("key", "fit", "desc", "geno", "slot", "occ_list"):
        out[f"{k}_{f}"] = s[f]
    for f in ("parents", "fit", "desc", "cell", "won"):
        out[f"{k}_b{f}"] = b[f]
import time, torch
a = qd.Archive(W.workload("rastrigin_proj_cvt_b65536"))
a.generations(1, 5)
torch.cuda.synchronize()
t0 = time.perf_counter()
a.generations(6, 20)
torch.cuda.synchronize()
out["seconds_20"] = np.float64(time.perf_counter() - t0)
np.savez(sys.argv[2], **out)
print("child done", flush=True)
"""


def test_generations_repeat_in_a_fresh_process_on_few_cus(tmp_path):
    """The benchmark configuration and the 27-64-64-8 policy configuration,
    two generations each, in a fresh process whose queues may use compute
    units 0 .. 15 only (HSA_CU_MASK), against this process on the whole
    chip: the same archives and batches, bit for bit."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    dst = str(tmp_path / "child.npz")
    say("fresh process on 16 compute units: configuration 3 and the 27-64-64-8 policies")
    env = dict(os.environ, HSA_CU_MASK="0:0-15")
    r = subprocess.run([sys.executable, "-c", CHILD, root, dst], env=env, capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    got = np.load(dst)
    for k, (name, kw) in enumerate([("rastrigin_proj_cvt_b65536", {}), ("mlp64_cvt_b8192", {})]):
        a = qd().Archive(W.workload(name, **kw))
        a.generations(1, 2)
        s, b = a.snapshot(), a.last_batch()
        for f in ("key", "fit", "desc", "geno", "slot", "occ_list"):
            np.testing.assert_array_equal(got[f"{k}_{f}"], s[f], err_msg=f"{name} {f}")
        for f in ("parents", "fit", "desc", "cell", "won"):
            np.testing.assert_array_equal(got[f"{k}_b{f}"], b[f], err_msg=f"{name} batch {f}")
    # the mask took effect: the same 20 generations are several times slower there
    import time
    a = qd().Archive(W.workload("rastrigin_proj_cvt_b65536"))
    a.generations(1, 5)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    a.generations(6, 20)
    torch.cuda.synchronize()
    here = time.perf_counter() - t0
    say(f"20 generations: {float(got['seconds_20']) * 1e3:.2f} ms on 16 CUs, {here * 1e3:.2f} ms here")
    assert float(got["seconds_20"]) > 4.0 * here
