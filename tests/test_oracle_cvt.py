"""Pins of the oracle's Lloyd construction of the CVT centroids.

* One Lloyd step equals a k-means step written here with numpy: points from
  Philox (the published generator, checked bit for bit against rocRAND in
  test_oracle_rng), fp64 nearest centroids, exact integer means.
* The quantisation energy (mean squared distance of the points to their
  nearest centroid) never increases over the iterations -- the defining
  property of Lloyd's algorithm.
* No iterations leave the uniform centroids; centroids that receive no point
  stay where they are.
"""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2202_01258_amd import workloads as W

TAG_CVT_SAMPLE = 5


def cvt_workload(C, D, samples, iters, seed=0):
    if D == 2:
        return W.workload("rastrigin_proj_cvt_b65536", C=C, batch=8, seed=seed,
                          cvt_samples=samples, cvt_iters=iters)
    return W.workload("mlp64_cvt_b8192", C=C, batch=8, seed=seed, cvt_samples=samples,
                      cvt_iters=iters)


def centroids(w):
    o = O.Oracle(w)
    o.setup()
    return o.centroids().astype(np.float64)


def sample_numerators(w):
    i = np.arange(w["cvt_samples"], dtype=np.uint32)
    z = np.zeros_like(i)
    ctr = np.stack([i, z, z, np.full_like(i, TAG_CVT_SAMPLE)], axis=1)
    key = [w["seed"] & 0xFFFFFFFF, w["seed"] >> 32]
    return (O.philox(ctr, key)[:, : w["D"]] >> 8).astype(np.int64)


def assign(points, cent):
    d2 = ((points[:, None, :] - cent[None, :, :]) ** 2).sum(-1)
    order = np.argsort(d2, axis=1, kind="stable")
    best, second = order[:, 0], order[:, 1]
    rows = np.arange(len(points))
    close = d2[rows, second] - d2[rows, best] <= 1e-6 * d2[rows, second]
    return best, close


@pytest.mark.parametrize("C,D,S", [(64, 2, 3000), (37, 4, 2000)])
def test_one_lloyd_step_is_a_kmeans_step(C, D, S):
    w0 = cvt_workload(C, D, 0, 0)
    w1 = cvt_workload(C, D, S, 1)
    c0, c1 = centroids(w0), centroids(w1)
    m = sample_numerators(w1)
    pts = m.astype(np.float64) * 2.0**-24
    best, close = assign(pts, c0)
    assert not close.any(), "a near tie would make the fp64 assignment ambiguous"
    for b in range(C):
        mine = best == b
        if not mine.any():
            np.testing.assert_array_equal(c1[b], c0[b])
            continue
        sums = m[mine].sum(axis=0)
        want = np.float32(sums.astype(np.float64) / mine.sum() * 2.0**-24)
        np.testing.assert_array_equal(np.float32(c1[b]), want, err_msg=f"centroid {b}")


def test_quantisation_energy_never_increases():
    C, D, S = 50, 2, 4000
    m = sample_numerators(cvt_workload(C, D, S, 1))
    pts = m.astype(np.float64) * 2.0**-24
    energies = []
    for it in range(0, 9):
        c = centroids(cvt_workload(C, D, S, it))
        d2 = ((pts[:, None, :] - c[None, :, :]) ** 2).sum(-1).min(axis=1)
        energies.append(d2.mean())
    diffs = np.diff(energies)
    assert np.all(diffs <= 1e-7 * energies[0]), energies
    assert energies[-1] < 0.9 * energies[0]


def test_zero_iterations_and_empty_cells():
    c_uniform = centroids(cvt_workload(20, 2, 0, 0))
    np.testing.assert_array_equal(centroids(cvt_workload(20, 2, 500, 0)), c_uniform)
    # three points for twenty centroids: at most three move, each onto a point
    w = cvt_workload(20, 2, 3, 1)
    c = centroids(w)
    moved = np.any(c != c_uniform, axis=1)
    assert 1 <= moved.sum() <= 3
    pts = np.float32(sample_numerators(w).astype(np.float64) * 2.0**-24)
    for b in np.nonzero(moved)[0]:
        inside = [np.all(np.float32(c[b]) == p) for p in pts]
        mean_of_two = False
        if not any(inside):
            best, _ = assign(pts.astype(np.float64), c_uniform)
            mine = pts[best == b].astype(np.float64)
            mean_of_two = np.all(np.float32(mine.mean(axis=0)) == np.float32(c[b]))
        assert any(inside) or mean_of_two
