"""Pins of the oracle's policy rollout on the synthetic dynamics.

* Zero weights from a zero state: a = 0, s = 0 forever, return 0 and
  descriptor sigmoid(0) = 1/2 exactly.
* Against an fp64 numpy rollout built from matrix products and np.tanh
  (a transposed weight block, a wrong bias slice or reward sign fails it).
* Glorot-uniform first batch within its limits, zero biases; environment
  entries 0.1 N(0,1).
"""
import numpy as np
import pytest
from scipy import stats

from oracle import oracle as O
from paper_2202_01258_amd.workloads import genotype_len, workload


def split(w, obs, hid, act):
    i = 0
    out = []
    for shape in ((hid, obs), (hid,), (hid, hid), (hid,), (act, hid), (act,)):
        k = int(np.prod(shape))
        out.append(w[i:i + k].reshape(shape))
        i += k
    assert i == w.size
    return out


def rollout64(w, obs, hid, act, T, A, B, s0):
    W1, b1, W2, b2, W3, b3 = [x.astype(np.float64) for x in split(w, obs, hid, act)]
    A, B, s = A.astype(np.float64), B.astype(np.float64), s0.astype(np.float64)
    ret, dsum = 0.0, np.zeros(4)
    for _ in range(T):
        a = np.tanh(W3 @ np.tanh(W2 @ np.tanh(W1 @ s + b1) + b2) + b3)
        s = np.tanh(A @ s + B @ a)
        ret += s[0] - 0.5 * a @ a
        dsum += 1.0 / (1.0 + np.exp(-s[1:5]))
    return ret, dsum / T


def test_zero_policy_zero_state():
    obs, hid, act, T = 27, 16, 8, 30
    n = hid * obs + hid + hid * hid + hid + act * hid + act
    rng = np.random.default_rng(0)
    A = rng.normal(0, 0.3, (obs, obs)).astype(np.float32)
    B = rng.normal(0, 0.3, (obs, act)).astype(np.float32)
    f, d = O.mlp_rollout(np.zeros(n, np.float32), obs, hid, act, T, A, B, np.zeros(obs, np.float32))
    assert f == 0.0
    np.testing.assert_array_equal(d, np.float32([0.5] * 4))


@pytest.mark.parametrize("hid,T", [(8, 5), (64, 25), (128, 10)])
def test_rollout_matches_fp64(hid, T):
    obs, act = 27, 8
    n = hid * obs + hid + hid * hid + hid + act * hid + act
    rng = np.random.default_rng(hid + T)
    for trial in range(3):
        w = rng.normal(0, 0.6 / np.sqrt(hid), n).astype(np.float32)
        A = rng.normal(0, 0.3, (obs, obs)).astype(np.float32)
        B = rng.normal(0, 0.5, (obs, act)).astype(np.float32)
        s0 = rng.normal(0, 0.5, obs).astype(np.float32)
        f, d = O.mlp_rollout(w, obs, hid, act, T, A, B, s0)
        rf, rd = rollout64(w, obs, hid, act, T, A, B, s0)
        assert abs(f - rf) <= 1e-4 * max(1.0, abs(rf)), (f, rf)
        np.testing.assert_allclose(d, rd, atol=2e-6)


def test_first_batch_glorot_and_environment():
    w = workload("mlp64_cvt_b8192", batch=64, T=3)
    o = O.Oracle(w)
    o.init()
    x = o.last_offspring()
    obs, hid, act = w["obs"], w["hid"], w["act"]
    assert x.shape[1] == genotype_len(w) == 6472
    parts = [split(row, obs, hid, act) for row in x]
    W1, b1, W2, b2, W3, b3 = [np.stack([p[i] for p in parts]) for i in range(6)]
    for W, fi, fo in ((W1, obs, hid), (W2, hid, hid), (W3, hid, act)):
        lim = np.sqrt(6.0 / (fi + fo))
        assert np.all(W >= -lim - 1e-7) and np.all(W < lim + 1e-7)
        assert abs(np.std(W) - lim / np.sqrt(3)) < 0.02 * lim
    for b in (b1, b2, b3):
        assert np.all(b == 0)
    env = o.env().astype(np.float64)
    assert env.size == obs * obs + obs * act + obs
    assert abs(env.std() - 0.1) < 0.01
    assert stats.kstest(env / 0.1, "norm").pvalue > 1e-3
    # the first batch's stored results re-evaluate identically
    A = o.env()[: obs * obs].reshape(obs, obs)
    B = o.env()[obs * obs: obs * obs + obs * act].reshape(obs, act)
    s0 = o.env()[obs * obs + obs * act:]
    lb = o.last_batch()
    for j in (0, 17, 63):
        f, d = O.mlp_rollout(x[j], obs, hid, act, w["T"], A, B, s0)
        assert f == lb["fit"][j]
        np.testing.assert_array_equal(d, lb["desc"][j])


def rollout64_death(w, obs, hid, act, T, A, B, s0, mode, thr):
    """fp64 rollout with the failure rule: stop at the first new state whose
    component 0 is below thr; that step and the rest count for nothing."""
    W1, b1, W2, b2, W3, b3 = [x.astype(np.float64) for x in split(w, obs, hid, act)]
    A, B, s = A.astype(np.float64), B.astype(np.float64), s0.astype(np.float64)
    ret, dsum, valid, failed, lows = 0.0, np.zeros(4), 0, False, []
    for _ in range(T):
        a = np.tanh(W3 @ np.tanh(W2 @ np.tanh(W1 @ s + b1) + b2) + b3)
        sn = np.tanh(A @ s + B @ a)
        lows.append(sn[0])
        if sn[0] < thr:
            failed = True
            break
        ret += sn[0] - 0.5 * a @ a
        dsum += 1.0 / (1.0 + np.exp(-sn[1:5]))
        valid += 1
        s = sn
    fit = np.nan if (mode == 2 and failed) or valid == 0 else ret
    return fit, (dsum / valid if valid else np.zeros(4)), valid, np.array(lows)


def random_policy(rng, obs, hid, act):
    n = hid * obs + hid + hid * hid + hid + act * hid + act
    w = rng.normal(0, 0.6 / np.sqrt(hid), n).astype(np.float32)
    A = rng.normal(0, 0.3, (obs, obs)).astype(np.float32)
    B = rng.normal(0, 0.5, (obs, act)).astype(np.float32)
    s0 = rng.normal(0, 0.5, obs).astype(np.float32)
    return w, A, B, s0


@pytest.mark.parametrize("mode", [1, 2])
def test_death_never_and_always(mode):
    obs, hid, act, T = 27, 16, 8, 20
    rng = np.random.default_rng(11)
    w, A, B, s0 = random_policy(rng, obs, hid, act)
    f0, d0 = O.mlp_rollout(w, obs, hid, act, T, A, B, s0)
    f, d = O.mlp_rollout(w, obs, hid, act, T, A, B, s0, mode, -np.inf)   # never fails
    assert f == f0
    np.testing.assert_array_equal(d, d0)
    f, d = O.mlp_rollout(w, obs, hid, act, T, A, B, s0, mode, np.inf)    # fails at once
    assert np.isnan(f)
    np.testing.assert_array_equal(d, np.zeros(4, np.float32))


@pytest.mark.parametrize("mode", [1, 2])
def test_death_truncates_like_fp64(mode):
    obs, hid, act, T = 27, 32, 8, 40
    rng = np.random.default_rng(5 + mode)
    checked = 0
    for trial in range(12):
        w, A, B, s0 = random_policy(rng, obs, hid, act)
        _, _, _, lows = rollout64_death(w, obs, hid, act, T, A, B, s0, 0, -np.inf)
        thr = np.sort(lows)[len(lows) // 4]          # fails somewhere inside the episode
        fit, desc, valid, seen = rollout64_death(w, obs, hid, act, T, A, B, s0, mode, thr)
        if np.min(np.abs(seen - thr)) < 1e-4 or not 0 < valid < T:
            continue                                  # the fp32 rollout could fail elsewhere
        f, d = O.mlp_rollout(w, obs, hid, act, T, A, B, s0, mode, thr)
        if mode == 2:
            assert np.isnan(f)
        else:
            assert abs(f - fit) <= 1e-4 * max(1.0, abs(fit)), (f, fit)
        np.testing.assert_allclose(d, desc, atol=2e-6)
        checked += 1
    assert checked >= 6
