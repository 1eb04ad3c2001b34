"""Pins for the oracle's Gaussian probe generator.

* The Box-Muller series coefficients are the fp32 values nearest to
  (pi/2)^n / n!, checked against an exact rational computation with pi taken
  from Machin's formula at 60 digits.
* The own fp32 logarithm and sine/cosine are checked exhaustively against
  fp64 libm over every input they can receive (all 2^24 grid points), and at
  special values that are exact by construction.
* The resulting z has the N(0,1) law (moments and a Kolmogorov-Smirnov test).
"""
import math
from decimal import Decimal, getcontext
from fractions import Fraction

import numpy as np
import pytest


def _machin_pi(digits=60):
    getcontext().prec = digits + 10

    def arctan_inv(x):
        x = Decimal(x)
        x2 = x * x
        term = Decimal(1) / x
        total = term
        n = 1
        while True:
            term /= -x2
            n += 2
            d = term / n
            if abs(d) < Decimal(10) ** -(digits + 5):
                break
            total += d
        return total

    return 16 * arctan_inv(5) - 4 * arctan_inv(239)


def _nearest_f32(x: Fraction) -> np.float32:
    f = np.float32(float(x))
    best, err = f, abs(Fraction(float(f)) - x)
    for cand in (np.nextafter(f, np.float32(np.inf)), np.nextafter(f, np.float32(-np.inf))):
        e = abs(Fraction(float(cand)) - x)
        if e < err:
            best, err = cand, e
    return best


def test_series_constants_are_correctly_rounded(oracle_mod):
    pi = Fraction(_machin_pi())
    half_pi = pi / 2
    ours = oracle_mod.series_constants()
    expected = []
    for n in (1, 3, 5, 7, 9, 11):
        v = half_pi ** n / Fraction(math.factorial(n))
        expected.append(_nearest_f32(v if (n // 2) % 2 == 0 else -v))
    for n in (0, 2, 4, 6, 8, 10, 12):
        v = half_pi ** n / Fraction(math.factorial(n))
        expected.append(_nearest_f32(v if (n // 2) % 2 == 0 else -v))
    assert np.array_equal(ours.view(np.uint32), np.array(expected, np.float32).view(np.uint32))


def test_ln_exhaustive_against_libm(oracle_mod):
    m = np.arange(1, (1 << 24) + 1, dtype=np.uint32)
    ours = oracle_mod.ln_u24_array(m).astype(np.float64)
    ref = np.log(m.astype(np.float64) * 2.0 ** -24)
    ulp = np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64)
    ulp[ref == 0] = np.spacing(np.float32(0))
    err_ulp = np.abs(ours - ref) / ulp
    assert err_ulp.max() <= 2.0, err_ulp.max()
    assert ours[-1] == 0.0                      # ln 1 = 0 exactly
    assert np.all(ours[:-1] < 0.0)              # ln u < 0 for u < 1


def test_sincos_exhaustive_against_libm(oracle_mod):
    i = np.arange(0, 1 << 24, dtype=np.uint32)
    c, s = oracle_mod.sincos_2pi_u24_array(i)
    ang = 2.0 * np.pi * i.astype(np.float64) * 2.0 ** -24
    err = max(np.abs(c - np.cos(ang)).max(), np.abs(s - np.sin(ang)).max())
    assert err <= 2.0 ** -23, err
    # exact quarter turns
    q = 1 << 22
    assert (c[0], s[0]) == (1.0, 0.0)
    assert (abs(c[q]), s[q]) == (0.0, 1.0)
    assert (c[2 * q], abs(s[2 * q])) == (-1.0, 0.0)
    assert (abs(c[3 * q]), s[3 * q]) == (0.0, -1.0)
    # cos^2 + sin^2 = 1 to fp32 accuracy
    assert np.abs(c.astype(np.float64) ** 2 + s.astype(np.float64) ** 2 - 1).max() < 4e-7


def test_box_muller_special_values(oracle_mod):
    # u1 = 1 (wa >> 8 = 2^24 - 1) gives r = 0, hence z = +-0
    za, zb = oracle_mod.box_muller(0xFFFFFFFF, 0x12345678)
    assert za == 0.0 and zb == 0.0
    # u2 = 0 gives (r, 0); u2 = 1/4 gives (0, r)
    za, zb = oracle_mod.box_muller(0, 0)
    r = np.float32(np.sqrt(np.float32(-2.0) * oracle_mod.ln_u24(1)))
    assert za == r and zb == 0.0
    za, zb = oracle_mod.box_muller(0, 0x40000000)
    assert abs(za) == 0.0 and zb == r
    # largest radius: u1 = 2^-24
    assert abs(float(r) - np.sqrt(-2 * np.log(2.0 ** -24))) < 1e-5


@pytest.mark.slow
def test_gaussian_law(oracle_mod):
    from scipy import stats
    n = 4_000_000
    z = np.concatenate([oracle_mod.gaussian(0x50A10000, 0, j, 0, n // 4) for j in range(4)]).astype(np.float64)
    assert abs(z.mean()) < 5 / np.sqrt(n)
    assert abs(z.var() - 1) < 5 * np.sqrt(2 / n)
    assert abs(stats.skew(z)) < 5 * np.sqrt(6 / n)
    assert abs(stats.kurtosis(z, fisher=False) - 3) < 5 * np.sqrt(24 / n)
    assert stats.kstest(z, "norm").pvalue > 1e-4


def test_gaussian_streams_are_keyed(oracle_mod):
    a = oracle_mod.gaussian(7, 0, 0, 0, 64)
    assert not np.array_equal(a, oracle_mod.gaussian(8, 0, 0, 0, 64))       # seed
    assert not np.array_equal(a, oracle_mod.gaussian(7, 1, 0, 0, 64))       # step
    assert not np.array_equal(a, oracle_mod.gaussian(7, 0, 1, 0, 64))       # direction
    assert not np.array_equal(a, oracle_mod.gaussian(7, 1 << 32, 0, 0, 64)) # high step word
    # a slice starting mid-quad equals the same indices of a longer slice
    b = oracle_mod.gaussian(7, 0, 0, 3, 61)
    assert np.array_equal(a[3:], b)


def test_gaussian_index_layout(oracle_mod):
    # z[4q + i] comes from Philox(counter = (q, pair, step, 0), key = (seed_lo, seed_hi))
    seed, step, pair, q = 0x1234567890ABCDEF, 5, 3, 1000
    w = oracle_mod.philox([q, pair, step, 0], [seed & 0xFFFFFFFF, seed >> 32])
    za, zb = oracle_mod.box_muller(w[0], w[1])
    zc, zd = oracle_mod.box_muller(w[2], w[3])
    z = oracle_mod.gaussian(seed, step, pair, 4 * q, 4)
    assert np.array_equal(z, np.array([za, zb, zc, zd], np.float32))
