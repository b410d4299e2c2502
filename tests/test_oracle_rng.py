"""Pins of the oracle's random-number layer against things other than itself.

* Philox4x32-10 against rocRAND's open-source engine compiled on the host
  (a library routine), over random counters and keys.
* The 24-bit uniforms at their exact end points.
* The quarter-turn sine/cosine against numpy's fp64 sin/cos.
* Box-Muller against the fp64 formula sqrt(-2 ln u1) (cos, sin)(2 pi u2) and
  against N(0,1) by moments and a Kolmogorov-Smirnov test.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest
from scipy import stats

from oracle import oracle as O

HELPER = os.path.join(os.path.dirname(__file__), "helpers", "rocrand_philox_ref.cpp")
ROCM_INC = "/opt/rocm/include"


@pytest.fixture(scope="module")
def rocrand_ref(tmp_path_factory):
    if shutil.which("g++") is None or not os.path.exists(
            os.path.join(ROCM_INC, "rocrand", "rocrand_philox4x32_10.h")):
        pytest.skip("rocRAND headers or g++ not available")
    exe = str(tmp_path_factory.mktemp("rr") / "rr")
    subprocess.run(["g++", "-O1", "-D__HIP_PLATFORM_AMD__", "-I", ROCM_INC, HELPER, "-o", exe],
                   check=True)
    return exe


def test_philox_matches_rocrand(rocrand_ref):
    rng = np.random.default_rng(1234)
    m = 4000
    keys = rng.integers(0, 2**32, size=(m, 2), dtype=np.uint64).astype(np.uint32)
    ctrs = rng.integers(0, 2**32, size=(m, 4), dtype=np.uint64).astype(np.uint32)
    # edge words: zeros, all ones, the counter layout actually used (small ints)
    keys[:3] = [[0, 0], [0xFFFFFFFF, 0xFFFFFFFF], [0, 0]]
    ctrs[:3] = [[0, 0, 0, 0], [0xFFFFFFFF] * 4, [5, 17, 3, 2]]
    text = "\n".join(" ".join(str(int(v)) for v in (*k, *c)) for k, c in zip(keys, ctrs))
    out = subprocess.run([rocrand_ref], input=text, capture_output=True, text=True, check=True)
    ref = np.array([[int(t) for t in line.split()] for line in out.stdout.strip().splitlines()],
                   dtype=np.uint64).astype(np.uint32)
    mine = np.stack([O.philox(c, k)[0] for c, k in zip(ctrs, keys)])
    np.testing.assert_array_equal(mine, ref)


def test_philox_bits_are_balanced():
    # 2^16 blocks from the counter layout the method uses; every output bit
    # must be set about half the time (a dropped xor or key word breaks this).
    j = np.arange(1 << 16, dtype=np.uint32)
    ctr = np.stack([j & 255, j >> 8, np.full_like(j, 7), np.full_like(j, 2)], axis=1)
    out = O.philox(ctr, [0, 0])
    bits = ((out[:, :, None] >> np.arange(32, dtype=np.uint32)) & 1).astype(np.float64)
    frac = bits.mean(axis=0)
    assert np.all(np.abs(frac - 0.5) < 0.01), frac


def test_u24_end_points():
    assert O.u24(0) == 0.0
    assert O.u24(0xFFFFFFFF) == 1.0 - 2.0**-24
    assert O.u24(0x000000FF) == 0.0           # low 8 bits are ignored
    assert O.u24p(0) == 2.0**-24
    assert O.u24p(0xFFFFFFFF) == 1.0
    assert O.u24(0x80000000) == 0.5


def test_turn_sincos_against_fp64():
    m = np.concatenate([
        np.arange(0, 1 << 24, 97, dtype=np.uint32),
        # around every quarter turn and the half-way points between them
        np.array([(q << 22) + d for q in range(4) for d in (-1, 0, 1)] +
                 [(q << 22) + (1 << 21) + d for q in range(4) for d in (-1, 0, 1)],
                 dtype=np.int64).astype(np.uint32) & 0xFFFFFF,
    ])
    cs = O.turn_sincos(m).astype(np.float64)
    ang = 2.0 * np.pi * m.astype(np.float64) / 2.0**24
    assert np.max(np.abs(cs[:, 0] - np.cos(ang))) < 2.5e-7
    assert np.max(np.abs(cs[:, 1] - np.sin(ang))) < 2.5e-7
    exact = O.turn_sincos(np.array([0, 1 << 22, 2 << 22, 3 << 22], dtype=np.uint32))
    np.testing.assert_array_equal(exact, [[1, 0], [0, 1], [-1, 0], [0, -1]])


def test_table_turn_sincos_against_fp64():
    # the table-driven (cos, sin) of 2 pi m / 2^24 that the sampler uses
    m = np.concatenate([np.arange(0, 1 << 24, 37, dtype=np.uint32),
                        (np.arange(256, dtype=np.uint32) << 16),           # table points
                        (np.arange(256, dtype=np.uint32) << 16) + 0xFFFF])  # bin ends
    cs = O.turn_sincos_tab(m).astype(np.float64)
    ang = 2.0 * np.pi * m.astype(np.float64) / 2.0**24
    assert np.max(np.abs(cs[:, 0] - np.cos(ang))) < 2.0e-7
    assert np.max(np.abs(cs[:, 1] - np.sin(ang))) < 2.0e-7
    # at a table point the remainder is 0 and the entry comes back unchanged
    pts = (np.arange(256, dtype=np.uint32) << 16)
    np.testing.assert_array_equal(O.turn_sincos_tab(pts), O.turn_sincos(pts))


def test_box_muller_against_fp64_formula():
    rng = np.random.default_rng(7)
    xa = rng.integers(0, 2**32, size=200000, dtype=np.uint64).astype(np.uint32)
    xb = rng.integers(0, 2**32, size=200000, dtype=np.uint64).astype(np.uint32)
    z = O.box_muller(xa, xb).astype(np.float64)
    u1 = ((xa >> 8).astype(np.float64) + 1.0) / 2.0**24
    u2 = (xb >> 8).astype(np.float64) / 2.0**24
    r = np.sqrt(-2.0 * np.log(u1))
    ref = np.stack([r * np.cos(2 * np.pi * u2), r * np.sin(2 * np.pi * u2)], axis=1)
    err = np.abs(z - ref) / np.maximum(1.0, np.abs(ref))
    assert err.max() < 1e-6, err.max()


def test_box_muller_is_standard_normal():
    j = np.arange(1 << 19, dtype=np.uint32)
    ctr = np.stack([j, np.zeros_like(j), np.ones_like(j), np.full_like(j, 2)], axis=1)
    x = O.philox(ctr, [12345, 678])
    z = np.concatenate([O.box_muller(x[:, 0], x[:, 1]), O.box_muller(x[:, 2], x[:, 3])])
    z = z.astype(np.float64)
    for col in range(2):
        v = z[:, col]
        assert abs(v.mean()) < 5e-3
        assert abs(v.var() - 1.0) < 1e-2
        assert abs(stats.skew(v)) < 1e-2
        assert abs(stats.kurtosis(v)) < 2e-2
        assert stats.kstest(v, "norm").pvalue > 1e-3
    # the two members of a pair are uncorrelated
    assert abs(np.corrcoef(z[:, 0], z[:, 1])[0, 1]) < 5e-3
