"""Pins of the oracle's archive logic: insertion, selection, variation, stats.

* Insertion (Algorithm 1's sequential loop) against the four masked steps of
  Appendix A.4 written here with numpy, and against the maximum of packed
  keys, on tiny batches with forced ties, over every batch permutation.
* Archive invariants over many generations: per-cell objective, occupancy and
  best never decrease; every stored genotype re-evaluates to its stored
  objective and descriptor, and its descriptor maps to its cell.
* Selection: only filled cells, uniform over them (chi-square).
* Variation (Algorithm 2): sigma = 0 copies parent 1; the offspring residual
  is N(0, sigma1^2 + sigma2^2 (theta2 - theta1)^2) per gene.
* QD-score, coverage, best objective (Eq. 1, Appendix B.1).
"""
import itertools

import numpy as np
import pytest
from scipy import stats

from oracle import oracle as O
from paper_2202_01258_amd.workloads import workload


def four_step_addition(arch_fit, arch_occ, fit, cell):
    """Appendix A.4: (i) drop death-flagged offspring, (ii) keep only the best
    offspring of each cell (others -> -inf; the lowest index among equals),
    (iii) mask offspring not better than the incumbent, (iv) scatter."""
    fit = np.asarray(fit, np.float64).copy()
    alive = ~np.isnan(fit) & (cell >= 0)                          # (i)
    keep = np.zeros(fit.size, bool)
    for c in np.unique(cell[alive]):                              # (ii)
        idx = np.nonzero(alive & (cell == c))[0]
        best = idx[np.argmax(fit[idx])]                           # argmax: first of equals
        keep[best] = True
    better = keep.copy()
    for j in np.nonzero(keep)[0]:                                 # (iii)
        c = cell[j]
        better[j] = (not arch_occ[c]) or fit[j] > arch_fit[c]
    new_fit, new_occ = arch_fit.copy(), arch_occ.copy()           # (iv)
    winner = np.full(arch_fit.size, -1)
    for j in np.nonzero(better)[0]:
        new_fit[cell[j]] = fit[j]
        new_occ[cell[j]] = 1
        winner[cell[j]] = j
    return new_fit, new_occ, winner


def tiny_oracle(C, nb):
    # a 1-D grid of C cells over [0, C) used as an insertion harness
    w = workload("rastrigin_grid_b128", batch=nb, D=1, grid=(C, 0), C=C, lo=(0.0,), hi=(float(C),))
    return O.Oracle(w)


@pytest.mark.parametrize("seed", range(6))
def test_insertion_matches_four_steps_and_keys(seed):
    rng = np.random.default_rng(seed)
    C, nb = 3, 5
    base_fit = rng.choice([-1.0, 0.0, 1.0], nb).astype(np.float32)
    base_cell = rng.integers(0, C, nb)
    if seed % 2:
        base_fit[rng.integers(0, nb)] = np.nan                    # a death flag
    inc_occ = rng.integers(0, 2, C).astype(np.uint8)
    inc_fit = np.where(inc_occ == 1, rng.choice([-1.0, 0.0, 1.0], C), np.nan).astype(np.float32)
    for perm in itertools.permutations(range(nb)):
        fit, cell = base_fit[list(perm)], base_cell[list(perm)]
        o = tiny_oracle(C, nb)
        o.set_archive(np.zeros((C, o.n), np.float32), inc_fit, np.zeros((C, 1), np.float32), inc_occ)
        desc = (cell.astype(np.float32) + np.float32(0.5)).reshape(nb, 1)
        got_cell, won = o.insert_driven(fit, desc)
        np.testing.assert_array_equal(got_cell, np.where(np.isnan(fit), -1, cell))
        a = o.archive()
        ref_fit, ref_occ, winner = four_step_addition(inc_fit.astype(np.float64), inc_occ, fit, got_cell)
        np.testing.assert_array_equal(a["occ"], ref_occ)
        np.testing.assert_array_equal(a["fit"][ref_occ == 1], ref_fit[ref_occ == 1].astype(np.float32))
        np.testing.assert_array_equal(np.nonzero(won)[0], np.sort(winner[winner >= 0]))
        # the packed-key maximum reaches the same winners
        for c in range(C):
            keys = [O.key(inc_fit[c], -1, nb)] if inc_occ[c] else [0]
            keys += [O.key(fit[j], j, nb) for j in range(nb) if got_cell[j] == c]
            kmax = max(keys)
            if kmax != 0 and (kmax & 0xFFFFFFFF) != 0xFFFFFFFF:
                assert winner[c] == nb - 1 - (kmax & 0xFFFFFFFF)
            else:
                assert winner[c] == -1


def test_key_order():
    nb = 10
    assert O.key(1.0, 3, nb) > O.key(0.5, 0, nb)
    assert O.key(-0.0, 2, nb) == O.key(0.0, 2, nb)               # -0 is +0
    assert O.key(1.0, 2, nb) > O.key(1.0, 5, nb)                 # lower index wins ties
    assert O.key(1.0, -1, nb) > O.key(1.0, 0, nb)                # incumbent wins ties
    assert O.key(-np.inf, 9, nb) > 0                             # -inf still fills a cell
    assert O.key(-3.0, 0, nb) < O.key(-2.0, 9, nb)


def run_generations(name, G, **kw):
    o = O.Oracle(workload(name, **kw))
    o.init()
    hist = [o.archive()]
    for g in range(1, G + 1):
        o.generation(g)
        hist.append(o.archive())
    return o, hist


@pytest.mark.parametrize("name,kw,G", [
    ("rastrigin_grid_b128", {}, 40),
    ("sphere_grid_b16384", dict(batch=256), 25),
    ("rastrigin_proj_cvt_b65536", dict(batch=64, n=200, C=400), 8),
])
def test_archive_invariants(name, kw, G):
    o, hist = run_generations(name, G, **kw)
    w = o.w
    for prev, cur in zip(hist, hist[1:]):
        assert np.all(cur["occ"] >= prev["occ"])
        both = prev["occ"] == 1
        assert np.all(cur["fit"][both] >= prev["fit"][both])
        assert np.nanmax(cur["fit"]) >= np.nanmax(prev["fit"])
    last = hist[-1]
    filled = np.nonzero(last["occ"])[0]
    assert np.all(np.isnan(last["fit"][last["occ"] == 0]))
    assert not np.any(np.isnan(last["fit"][filled]))
    cent = o.centroids()
    for c in filled:
        f, d = O.eval_testfn(w["task"], last["geno"][c], w["lo"], w["hi"])
        assert f == last["fit"][c]
        np.testing.assert_array_equal(d, last["desc"][c])
        if w["tess"] == 0:
            assert O.grid_cell(d, w["grid"], w["lo"], w["hi"]) == c
        else:
            assert O.cvt_cell(d, w["lo"], w["hi"], cent) == c
    s = o.stats()
    assert s["coverage"] == len(filled)
    assert s["qd_score"] == pytest.approx(float(np.sum(last["fit"][filled].astype(np.float64))),
                                          rel=1e-12)
    assert s["best"] == float(np.max(last["fit"][filled]))
    s2 = o.stats(offset=100.0)
    assert s2["qd_score"] == pytest.approx(s["qd_score"] + 100.0 * len(filled), rel=1e-12)


def test_reinserting_a_batch_changes_nothing():
    o = O.Oracle(workload("rastrigin_grid_b128"))
    o.init()
    o.generation(1)
    lb = o.last_batch()
    geno = o.last_offspring()
    before = o.archive()
    o.insert_driven(lb["fit"], lb["desc"], geno)
    after = o.archive()
    for k in before:
        np.testing.assert_array_equal(before[k], after[k])


def test_first_batch_is_uniform_init():
    o = O.Oracle(workload("sphere_grid_b16384", batch=512))
    o.init()
    x = o.last_offspring()
    assert x.min() >= -0.1 and x.max() < 0.1
    assert abs(x.mean()) < 2e-3
    assert abs(x.std() - 0.2 / np.sqrt(12)) < 2e-3


def test_spread_first_batch():
    """init_mode 1: individual j adds one level per genotype half, uniform over
    that descriptor dimension's box, to the usual U[lo, hi) genes; the
    projection descriptors of the first batch then cover the box, so a
    65536-sized batch fills almost every one of 10^4 centroids' cells."""
    w = workload("rastrigin_proj_cvt_b65536", batch=4096, n=40, init_mode=1, C=400)
    o = O.Oracle(w)
    o.init()
    x = o.last_offspring().astype(np.float64)
    h = x.shape[1] // 2
    lev0 = x[:, :h].mean(1)
    lev1 = x[:, h:].mean(1)
    for lev, part in ((lev0, x[:, :h]), (lev1, x[:, h:])):
        # every gene of a half within [level - 0.1, level + 0.1): the half's
        # spread is that of the usual first batch
        width = part.max(1) - part.min(1)
        assert width.max() < 0.2 + 1e-5
        u = (lev + 5.12) / 10.24
        assert stats.kstest(np.clip(u, 0, 1), "uniform").pvalue > 1e-3
    assert abs(np.corrcoef(lev0, lev1)[0, 1]) < 0.1
    filled = int(o.archive()["occ"].sum())
    assert filled >= 390                    # 4096 draws over 400 cells
    plain = O.Oracle(workload("rastrigin_proj_cvt_b65536", batch=4096, n=40, C=400))
    plain.init()
    assert int(plain.archive()["occ"].sum()) < 10


def test_selection_only_filled_cells_and_uniform():
    o = O.Oracle(workload("sphere_grid_b16384", batch=4096, n=8))
    o.init()
    filled = set(np.nonzero(o.archive()["occ"])[0].tolist())
    o.generation(1)
    par = o.last_batch()["parents"]
    assert set(par.ravel().tolist()) <= filled
    counts = np.array([np.sum(par == c) for c in sorted(filled)])
    assert len(filled) >= 2
    assert stats.chisquare(counts).pvalue > 1e-3


def test_selection_single_cell():
    # one filled cell: every parent is that cell, and theta1 == theta2 leaves
    # only the iso term of Algorithm 2.
    w = workload("sphere_grid_b16384", batch=2048, n=8, init_lo=0.3, init_hi=0.30000001)
    o = O.Oracle(w)
    o.init()
    filled = np.nonzero(o.archive()["occ"])[0]
    assert filled.size == 1
    par_row = o.archive()["geno"][filled[0]]
    o.generation(1)
    assert np.all(o.last_batch()["parents"] == filled[0])
    res = (o.last_offspring() - par_row) / np.float32(0.005)
    for col in range(res.shape[1]):
        assert stats.kstest(res[:, col].astype(np.float64), "norm").pvalue > 1e-3


def test_variation_zero_sigma_copies_first_parent():
    o = O.Oracle(workload("rastrigin_grid_b128", iso_sigma=0.0, line_sigma=0.0))
    o.init()
    a = o.archive()
    o.generation(1)
    par = o.last_batch()["parents"]
    np.testing.assert_array_equal(o.last_offspring(), a["geno"][par[:, 0]])


def test_variation_residual_distribution():
    w = workload("sphere_grid_b16384", batch=8192, n=16, init_lo=-2.0, init_hi=2.0,
                 iso_sigma=0.02, line_sigma=0.3)
    o = O.Oracle(w)
    o.init()
    a = o.archive()
    o.generation(1)
    par = o.last_batch()["parents"]
    x = o.last_offspring().astype(np.float64)
    t1, t2 = a["geno"][par[:, 0]].astype(np.float64), a["geno"][par[:, 1]].astype(np.float64)
    sd = np.sqrt(0.02**2 + 0.3**2 * (t2 - t1) ** 2)
    z = (x - t1) / sd
    for col in (0, 5, 15):     # one gene per offspring: genes share eps2
        assert stats.kstest(z[:, col], "norm").pvalue > 1e-3
    assert np.all(np.abs(z) < 7)
