"""Pins of the oracle's objectives, descriptors and cell mapping.

Closed forms of Rastrigin and Sphere (Appendix B.2), agreement with the
literal fp64 formula to the 1e-5 relative tolerance, exact projection means,
clamping, grid edges and monotonicity, and CVT against an fp64 KD-tree, a
lattice that reduces to the grid, and constructed equidistant ties.
"""
import numpy as np
import pytest
from scipy.spatial import cKDTree

from oracle import oracle as O
from paper_2202_01258_amd.workloads import RASTRIGIN, RASTRIGIN_PROJ, SPHERE


def rastrigin64(x):
    x = x.astype(np.float64)
    return -10.0 * x.size - np.sum(x * x - 10.0 * np.cos(2.0 * np.pi * x))


@pytest.mark.parametrize("n", [1, 2, 5, 100, 257, 1000])
def test_rastrigin_closed_forms(n):
    f, _ = O.eval_testfn(RASTRIGIN, np.zeros(n, np.float32))
    assert f == 0.0                                   # global optimum
    rng = np.random.default_rng(n)
    k = rng.integers(-5, 6, n).astype(np.float32)     # integers: cos(2 pi k) = 1
    f, _ = O.eval_testfn(RASTRIGIN, k)
    assert f == -np.float32(np.sum(k.astype(np.float64) ** 2))
    h = k + np.float32(0.5)                           # half-integers: cos = -1
    f, _ = O.eval_testfn(RASTRIGIN, h)
    ref = -np.sum(h.astype(np.float64) ** 2 + 20.0)
    assert abs(f - ref) <= 1e-6 * abs(ref)


@pytest.mark.parametrize("scale", [0.1, 1.0, 5.12])
def test_rastrigin_matches_literal_fp64(scale):
    rng = np.random.default_rng(11)
    for n in (100, 1000):
        for _ in range(20):
            x = rng.uniform(-scale, scale, n).astype(np.float32)
            f, _ = O.eval_testfn(RASTRIGIN, x)
            ref = rastrigin64(x)
            assert abs(f - ref) <= 1e-5 * abs(ref), (f, ref)
            assert f <= 0.0


def test_sphere():
    rng = np.random.default_rng(5)
    for n in (1, 100, 1000):
        x = rng.normal(0, 1, n).astype(np.float32)
        f, d = O.eval_testfn(SPHERE, x)
        ref = -np.sum(x.astype(np.float64) ** 2)
        assert abs(f - ref) <= 1e-6 * abs(ref)
        assert d[0] == x[0] and (n < 2 or d[1] == x[1])
    ints = np.arange(-3, 4, dtype=np.float32)
    assert O.eval_testfn(SPHERE, ints)[0] == -28.0


def test_descriptor_first_two_genes_clipped():
    x = np.array([7.0, -9.0, 1.0, 2.0], np.float32)
    _, d = O.eval_testfn(RASTRIGIN, x)
    np.testing.assert_array_equal(d, np.float32([5.12, -5.12]))
    x = np.array([0.25, -3.5, 8.0], np.float32)
    _, d = O.eval_testfn(SPHERE, x)
    np.testing.assert_array_equal(d, np.float32([0.25, -3.5]))


def test_projection_descriptor():
    n = 1000
    for c in (0.5, -2.0, 0.0, 3.25):
        x = np.full(n, c, np.float32)
        _, d = O.eval_testfn(RASTRIGIN_PROJ, x)
        np.testing.assert_array_equal(d, np.float32([c, c]))
    x = np.concatenate([np.full(500, 9.0), np.full(500, -7.0)]).astype(np.float32)
    _, d = O.eval_testfn(RASTRIGIN_PROJ, x)
    # 5.12 is not a dyadic number, so its 500-term fp32 sum rounds
    np.testing.assert_allclose(d, [5.12, -5.12], rtol=5e-7)
    rng = np.random.default_rng(2)
    x = rng.uniform(-8, 8, n).astype(np.float32)
    _, d = O.eval_testfn(RASTRIGIN_PROJ, x)
    cl = np.clip(x.astype(np.float64), -5.12, 5.12)
    ref = [cl[:500].mean(), cl[500:].mean()]
    assert np.max(np.abs(d - ref)) < 1e-5


@pytest.mark.parametrize("dist", ["init", "box", "beyond"])
def test_projection_and_objective_at_n1000_match_plain_and_fp64(dist):
    """The two-half projection descriptor and the objective at n = 1000, in
    the R64 order, against the plainest fp32 order (one running sum in gene
    order) and against fp64: within 1e-5 of the box (hi - lo = 10.24) for
    the descriptor and 1e-5 relative for the objective, for genes from the
    configuration's first batch, over the whole box, and partly beyond it
    (clipped)."""
    n, lo, hi = 1000, np.float32(-5.12), np.float32(5.12)
    rng = np.random.default_rng({"init": 1, "box": 2, "beyond": 3}[dist])
    span = float(hi - lo)
    for _ in range(50):
        if dist == "init":
            x = rng.uniform(-0.1, 0.1, n)
        elif dist == "box":
            x = rng.uniform(-5.12, 5.12, n) * rng.uniform(0, 1) + rng.uniform(-4, 4)
        else:
            x = rng.normal(rng.uniform(-6, 6), 3.0, n)
        x = x.astype(np.float32)
        f, d = O.eval_testfn(RASTRIGIN_PROJ, x)
        cl = np.clip(x, lo, hi)
        # plain fp32: a running sum in gene order, then the IEEE quotient
        plain = [np.add.accumulate(cl[:500], dtype=np.float32)[-1] / np.float32(500),
                 np.add.accumulate(cl[500:], dtype=np.float32)[-1] / np.float32(500)]
        ref = [cl[:500].astype(np.float64).mean(), cl[500:].astype(np.float64).mean()]
        assert np.max(np.abs(d - np.float32(plain))) <= 1e-5 * span
        assert np.max(np.abs(d - np.array(ref))) <= 1e-5 * span
        assert np.max(np.abs(np.float32(plain) - np.array(ref))) <= 1e-5 * span
        x64 = x.astype(np.float64)
        terms32 = (x * x + np.float32(20.0) * np.sin(np.pi * x64).astype(np.float32) ** 2)
        plain_f = -np.add.accumulate(terms32.astype(np.float32), dtype=np.float32)[-1]
        ref_f = rastrigin64(x)
        assert abs(f - ref_f) <= 1e-5 * abs(ref_f)
        assert abs(plain_f - ref_f) <= 1e-5 * abs(ref_f)


def test_grid_edges_and_layout():
    lo, hi, grid = [-5.12, -5.12], [5.12, 5.12], [100, 100]
    assert O.grid_cell([-5.12, -5.12], grid, lo, hi) == 0
    assert O.grid_cell([5.12, 5.12], grid, lo, hi) == 9999
    assert O.grid_cell([5.12, -5.12], grid, lo, hi) == 99 * 100       # first dim is slowest
    assert O.grid_cell([-5.12, 5.12], grid, lo, hi) == 99
    assert O.grid_cell([0.0, 0.0], grid, lo, hi) == 50 * 100 + 50
    assert O.grid_cell([-1e-5, -1e-5], grid, lo, hi) == 49 * 100 + 49
    assert O.grid_cell([-100.0, 100.0], grid, lo, hi) == 99            # clamps
    assert O.grid_cell([np.nan, 0.0], grid, lo, hi) == -1
    assert O.grid_cell([0.0, np.inf], grid, lo, hi) == 50 * 100 + 99


def test_grid_matches_fp64_away_from_edges_and_is_monotone():
    rng = np.random.default_rng(9)
    lo, hi = np.float32([-5.12, -1.0]), np.float32([5.12, 3.0])
    grid = [100, 7]
    d = rng.uniform(lo - 0.5, hi + 0.5, (20000, 2)).astype(np.float32)
    cells = np.array([O.grid_cell(v, grid, lo, hi) for v in d])
    t = (d.astype(np.float64) - lo) / (hi.astype(np.float64) - lo) * grid
    frac = t - np.floor(t)
    safe = np.all((frac > 1e-4) & (frac < 1 - 1e-4), axis=1)
    b = np.clip(np.floor(t), 0, np.array(grid) - 1).astype(int)
    ref = b[:, 0] * grid[1] + b[:, 1]
    np.testing.assert_array_equal(cells[safe], ref[safe])
    xs = np.sort(rng.uniform(-6, 6, 5000)).astype(np.float32)
    bins = [O.grid_cell([x, 0.0], grid, lo, hi) // grid[1] for x in xs]
    assert np.all(np.diff(bins) >= 0)


def test_cvt_matches_kdtree_on_unique_nearest():
    rng = np.random.default_rng(4)
    for D, C in ((2, 500), (4, 300)):
        cent = rng.uniform(0, 1, (C, D)).astype(np.float32)
        lo, hi = np.zeros(D, np.float32), np.ones(D, np.float32)
        q = rng.uniform(0, 1, (3000, D)).astype(np.float32)
        dist, idx = cKDTree(cent.astype(np.float64)).query(q.astype(np.float64), k=2)
        unique = dist[:, 1] ** 2 - dist[:, 0] ** 2 > 1e-5 * dist[:, 1] ** 2
        got = np.array([O.cvt_cell(v, lo, hi, cent) for v in q])
        np.testing.assert_array_equal(got[unique], idx[unique, 0])
        # the normalisation into the unit box
        lo2, hi2 = np.full(D, -5.12, np.float32), np.full(D, 5.12, np.float32)
        got2 = np.array([O.cvt_cell(v * np.float32(10.24) - np.float32(5.12), lo2, hi2, cent)
                         for v in q[:300]])
        assert np.mean(got2 == got[:300]) > 0.99


def test_cvt_lattice_is_grid_and_ties_go_low():
    # centroids at the centres of an 8x8 lattice: nearest centroid = grid bin
    g = 8
    cc = (np.arange(g) + 0.5) / g
    cent = np.array([[a, b] for a in cc for b in cc], np.float32)
    rng = np.random.default_rng(8)
    q = rng.uniform(0, 1, (2000, 2)).astype(np.float32)
    got = np.array([O.cvt_cell(v, [0, 0], [1, 1], cent) for v in q])
    grid = np.array([O.grid_cell(v, [g, g], [0, 0], [1, 1]) for v in q])
    frac = q * g - np.floor(q * g)
    safe = np.all((frac > 1e-3) & (frac < 1 - 1e-3), axis=1)
    np.testing.assert_array_equal(got[safe], grid[safe])
    # a query exactly between two centroids goes to the lower index
    cent = np.array([[0.75, 0.5], [0.25, 0.5], [0.5, 0.9]], np.float32)
    assert O.cvt_cell([0.5, 0.5], [0, 0], [1, 1], cent) == 0
    cent = cent[[1, 0, 2]]
    assert O.cvt_cell([0.5, 0.5], [0, 0], [1, 1], cent) == 0
    assert O.cvt_cell([np.nan, 0.5], [0, 0], [1, 1], cent) == -1
