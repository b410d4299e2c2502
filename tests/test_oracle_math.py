"""Pins of the oracle's own fp32 transcendental functions against fp64 numpy.

Each function is checked over a dense sweep of its reachable domain, with an
error bound in units of the fp32 spacing of the exact result, plus the exact
special values the mathematics fixes.
"""
import numpy as np

from oracle import oracle as O


def ulp_err(got, ref):
    got = got.astype(np.float64)
    spacing = np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64)
    return np.abs(got - ref) / spacing


def test_scaled_sinpi():
    # sqrt(20) sin(pi x) up to sign, the Rastrigin term's sine
    x = np.linspace(-12, 12, 480001).astype(np.float32)
    got = np.abs(O.map_f32(O.MAP_RSINPI, x).astype(np.float64))
    ref = np.sqrt(20.0) * np.abs(np.sin(np.pi * x.astype(np.float64)))
    assert np.max(np.abs(got - ref)) < 1.2e-6
    ints = np.arange(-50, 51, dtype=np.float32)
    assert np.all(O.map_f32(O.MAP_RSINPI, ints) == 0.0)
    halves = ints + np.float32(0.5)
    assert np.max(np.abs(np.abs(O.map_f32(O.MAP_RSINPI, halves)) - np.sqrt(20.0))) < 1.2e-6
    # near 0 the relative error stays within two ulp
    small = (2.0 ** np.linspace(-30, -2, 2001)).astype(np.float32)
    exact = np.sqrt(20.0) * np.sin(np.pi * small.astype(np.float64))
    rel = O.map_f32(O.MAP_RSINPI, small) / exact - 1
    assert np.max(np.abs(rel)) < 2.0**-22


def test_scaled_sinpi_coefficients_are_rounded_taylor_terms():
    # each coefficient is the fp32 rounding of sqrt(20) (-1)^k pi^(2k+1)/(2k+1)!,
    # worked out here in 60-digit decimal arithmetic
    import math
    from decimal import Decimal, getcontext
    getcontext().prec = 60
    pi = Decimal("3.14159265358979323846264338327950288419716939937510582097494459")
    s20 = Decimal(20).sqrt()
    got = O.rsin_coef()
    for k in range(6):
        exact = s20 * pi ** (2 * k + 1) / math.factorial(2 * k + 1) * (-1) ** k
        f = np.float32(float(exact))
        # rounding through double can only differ from direct rounding at a tie
        lo, hi = np.nextafter(f, np.float32(-np.inf)), np.nextafter(f, np.float32(np.inf))
        assert abs(Decimal(float(f)) - exact) <= min(abs(Decimal(float(lo)) - exact),
                                                   abs(Decimal(float(hi)) - exact))
        assert got[k] == f, (k, got[k], f)


def test_exp():
    x = np.linspace(-87, 88, 700001).astype(np.float32)
    got = O.map_f32(O.MAP_EXP, x)
    ref = np.exp(x.astype(np.float64))
    assert ulp_err(got, ref).max() <= 3.0
    assert O.map_f32(O.MAP_EXP, [0.0])[0] == 1.0
    # the input clamp keeps the result finite and positive
    big = O.map_f32(O.MAP_EXP, [1000.0, -1000.0])
    assert np.isfinite(big).all() and (big > 0).all()


def test_tanh():
    x = np.concatenate([np.linspace(-20, 20, 400001), np.linspace(-0.31, 0.31, 200001),
                        2.0 ** np.arange(-40, 0)]).astype(np.float32)
    got = O.map_f32(O.MAP_TANH, x)
    ref = np.tanh(x.astype(np.float64))
    nz = ref != 0
    assert ulp_err(got[nz], ref[nz]).max() <= 4.0
    assert O.map_f32(O.MAP_TANH, [0.0])[0] == 0.0
    # odd symmetry is exact and the range is closed
    np.testing.assert_array_equal(O.map_f32(O.MAP_TANH, -x), -got)
    assert np.all(np.abs(got) <= 1.0)


def test_sigmoid():
    x = np.linspace(-30, 30, 300001).astype(np.float32)
    got = O.map_f32(O.MAP_SIGMOID, x)
    ref = 1.0 / (1.0 + np.exp(-x.astype(np.float64)))
    assert ulp_err(got, ref).max() <= 4.0
    assert O.map_f32(O.MAP_SIGMOID, [0.0])[0] == 0.5


def test_r64_sum_exact_cases():
    # distinct powers of two: any dropped, repeated or misplaced term changes the sum
    for n in (1, 3, 4, 63, 64, 255, 256, 257, 1000):
        t = (2.0 ** -(np.arange(n) % 20)).astype(np.float32) * (1 + np.arange(n) // 20)
        t = t.astype(np.float32)
        exact = np.sum(t.astype(np.float64))
        if exact == np.float64(np.float32(exact)):
            assert O.r64_sum(t) == np.float32(exact)
    # sub-ranges
    t = np.arange(1000, dtype=np.float32)
    assert O.r64_sum(t, 0, 500) == np.float32(np.arange(500).sum())
    assert O.r64_sum(t, 500, 1000) == np.float32(np.arange(500, 1000).sum())
    assert O.r64_sum(t, 7, 7) == 0.0


def test_r64_sum_rounding_bound():
    rng = np.random.default_rng(3)
    for n in (100, 1000, 6472):
        t = rng.uniform(0, 1, n).astype(np.float32)
        exact = np.sum(t.astype(np.float64))
        # fp32 partial sums: error below (n/64 + 6) * eps * sum
        bound = (n / 64 + 6) * 2.0**-24 * exact
        assert abs(float(O.r64_sum(t)) - exact) <= bound
