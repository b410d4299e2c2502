"""The oracle's parallel per-offspring loops change nothing.

Each offspring of a generation depends only on the archive before it, and
insertion stays Algorithm 1's sequential loop, so the OpenMP build must give
the single-threaded build's archive and batch bit for bit, at any thread
count.  The single-threaded build is the same source compiled without OpenMP
(its pragmas ignored).
"""
import numpy as np
import pytest

from oracle import build as OB
from oracle import oracle as O
from paper_2202_01258_amd import workloads as W


@pytest.fixture(scope="module")
def single_thread_lib(tmp_path_factory):
    return OB.build(openmp=False, path=str(tmp_path_factory.mktemp("st") / "liboracle_st.so"))


CASES = [
    ("rastrigin_proj_cvt_b65536", dict(batch=300, C=500, n=200)),
    ("rastrigin_proj_cvt_b65536", dict(batch=400, C=700, n=64, init_mode=1, seed=2)),
    ("sphere_grid_b16384", dict(batch=500, init_lo=-5.12, init_hi=5.12, seed=1)),
    ("mlp64_cvt_b8192", dict(batch=24, T=30, C=64)),
    ("mlp64_cvt_b8192", dict(batch=32, T=40, C=64, death_mode=1, death_below=-0.05)),
]


def run(o, G):
    o.init()
    for g in range(1, G + 1):
        o.generation(g)
    return o.archive(), o.last_batch(), o.last_offspring()


@pytest.mark.parametrize("name,kw", CASES)
def test_threads_give_the_single_threaded_result(single_thread_lib, name, kw):
    w = W.workload(name, **kw)
    ref = run(O.Oracle(w, path=single_thread_lib), 3)
    prev = O.set_threads(0)
    try:
        assert O.set_threads(4) == 4
        got = run(O.Oracle(w), 3)
    finally:
        O.set_threads(prev)
    for a, b in zip(ref, got):
        if isinstance(a, dict):
            for k in a:
                np.testing.assert_array_equal(a[k].view(np.uint8), b[k].view(np.uint8), err_msg=k)
        else:
            np.testing.assert_array_equal(a.view(np.uint32), b.view(np.uint32))


def test_offspring_many_equals_one_by_one():
    w = W.workload("mlp64_cvt_b8192", batch=40, T=20, C=64)
    o = O.Oracle(w)
    o.init()
    js = np.array([0, 39, 5, 5, 17, 23], np.int32)
    prev = O.set_threads(0)
    try:
        O.set_threads(3)
        fit, desc, par = o.offspring_many(1, js)
    finally:
        O.set_threads(prev)
    for i, j in enumerate(js):
        _, f, d, p = o.offspring(1, int(j))
        assert fit[i].view(np.uint32) == np.float32(f).view(np.uint32)
        np.testing.assert_array_equal(desc[i], d)
        np.testing.assert_array_equal(par[i], p)
