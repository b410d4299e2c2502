"""Pins of the oracle's random-number layer against things other than itself.

* Philox4x32-10 against rocRAND's open-source engine compiled on the host
  (a library routine), over random counters and keys.
* The 24-bit uniforms at their exact end points.
* The inverse-CDF Gaussian sampler: its fp64 quantile against scipy's ndtri
  (Cephes) and textbook points, every one of its 2^24 magnitudes against
  ndtri, its table against the quantile at the interpolation points, and its
  output on Philox words against N(0,1) by moments and a Kolmogorov-Smirnov
  test.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest
from scipy import stats
from scipy.special import erfc, ndtri

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


def test_normal_quantile_against_scipy_and_closed_forms():
    # the fp64 source of the table: Phi^-1(1 - p/2) = -ndtri(p/2) (Cephes)
    for p in np.concatenate([np.logspace(-9, -1e-9, 300), [0.05, 0.01, 0.5, 0.999]]):
        ref = -ndtri(p / 2.0)
        assert abs(O.normal_quantile(p) - ref) <= 1e-13 * max(1.0, ref), p
    # textbook two-sided points and P(|Z| >= 1) = erfc(1/sqrt 2)
    assert abs(O.normal_quantile(0.05) - 1.959963984540054) < 1e-14
    assert abs(O.normal_quantile(0.01) - 2.5758293035489004) < 1e-14
    assert abs(O.normal_quantile(erfc(1.0 / np.sqrt(2.0))) - 1.0) < 1e-14


def test_normal_exhaustive_against_scipy():
    # every magnitude the sampler can return: k = 1..2^24, p = k 2^-24,
    # |z| = Phi^-1(1 - p/2) = -ndtri(k 2^-25); k - 1 is the low 24 bits of
    # the word, bits 24..30 are ignored, bit 31 is the sign
    k = np.arange(1, (1 << 24) + 1, dtype=np.uint64)
    mid = np.random.default_rng(3).integers(0, 128, size=k.size, dtype=np.uint64) << 24
    x = ((k - 1) | mid).astype(np.uint32)
    z = O.normal(x).astype(np.float64)
    ref = -ndtri(k.astype(np.float64) * 2.0**-25)
    err = np.abs(z - ref)
    assert err.max() <= 5e-7, err.max()
    spacing = np.spacing(np.maximum(np.abs(z), 2.0**-7).astype(np.float32)).astype(np.float64)
    assert (err / spacing).max() <= 4.0
    assert z[-1] == 0.0 and z[0] > 5.41                 # p = 1 and p = 2^-24
    assert np.all(np.diff(z) <= 0.0)                    # |z| falls as p grows
    neg = O.normal(x | np.uint32(0x80000000)).astype(np.float64)
    np.testing.assert_array_equal(neg[:-1], -z[:-1])


def test_normal_table_interpolates_at_chebyshev_points():
    # row 16 E + j covers p = 2^(E-24) (1 + (j + t)/16), t in [0, 1); its
    # stored cubic in t 2^19 meets the fp64 quantile at the four Chebyshev
    # points of [0, 1] up to the fp32 rounding of the coefficients
    tab = O.normal_table().astype(np.float64)
    assert tab.shape == (385, 4) and np.all(tab[384] == 0.0)
    nodes = (1.0 - np.cos((2 * np.arange(4) + 1) * np.pi / 8)) / 2.0
    for r in range(0, 384, 7):
        e, j = r >> 4, r & 15
        for t in nodes:
            q = O.normal_quantile(2.0 ** (e - 24) * (1.0 + (j + t) / 16.0))
            u = t * 2.0**19
            got = tab[r, 0] + u * (tab[r, 1] + u * (tab[r, 2] + u * tab[r, 3]))
            assert abs(got - q) <= 4e-7 * max(1.0, q), (r, t, got, q)


def test_normal_is_standard_normal():
    j = np.arange(1 << 19, dtype=np.uint32)
    ctr = np.stack([j, np.zeros_like(j), np.ones_like(j), np.full_like(j, 2)], axis=1)
    x = O.philox(ctr, [12345, 678])
    z = O.normal(x.ravel()).astype(np.float64).reshape(-1, 4)
    for col in range(4):
        v = z[:, col]
        assert abs(v.mean()) < 5e-3
        assert abs(v.var() - 1.0) < 1e-2
        assert abs(stats.skew(v)) < 1e-2
        assert abs(stats.kurtosis(v)) < 2e-2
        assert stats.kstest(v, "norm").pvalue > 1e-3
    # normals from the words of one block are uncorrelated
    c = np.corrcoef(z.T)
    assert np.max(np.abs(c - np.eye(4))) < 5e-3
    # signs balanced, and the magnitude independent of the sign bit
    sgn = z < 0
    assert abs(sgn.mean() - 0.5) < 2e-3
    assert abs(np.abs(z[sgn]).mean() - np.abs(z[~sgn]).mean()) < 5e-3
