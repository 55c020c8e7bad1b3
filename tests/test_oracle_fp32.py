"""Pins of the exact fp32 helpers (oracle/fp32.py) against exact rational arithmetic."""
from fractions import Fraction

import numpy as np

from oracle import fp32


def _round_fraction_to_f32(x):
    """Correctly rounded fp32 of a Fraction, ties to even, by exact comparison."""
    approx = np.float32(float(x))
    cands = {approx, np.nextafter(approx, np.float32(np.inf)), np.nextafter(approx, np.float32(-np.inf))}
    best = None
    for c in cands:
        d = abs(Fraction(float(c)) - x)
        key = (d, int(np.array(c).view(np.uint32)) & 1)
        if best is None or key < best[0]:
            best = (key, c)
    return best[1]


def test_fma_matches_exact_rounding_random():
    rng = np.random.default_rng(2)
    a = rng.standard_normal(3000).astype(np.float32)
    b = (rng.standard_normal(3000) * 100).astype(np.float32)
    c = (rng.standard_normal(3000) * np.exp2(rng.integers(-30, 10, 3000))).astype(np.float32)
    got = fp32.fma(a, b, c)
    for i in range(len(a)):
        exact = Fraction(float(a[i])) * Fraction(float(b[i])) + Fraction(float(c[i]))
        assert got[i] == _round_fraction_to_f32(exact), i


def test_fma_double_rounding_case():
    # 4097 * 16773121 = 2**36 + 1, so with these exponents a*b = 0.5 + 2**-37.
    a = np.float32(4097 * 2.0 ** -13)
    b = np.float32(16773121 * 2.0 ** -24)
    c = np.float32(2.0 ** 23)
    assert Fraction(float(a)) * Fraction(float(b)) == Fraction(1, 2) + Fraction(1, 2 ** 37)
    # exact a*b + c = 2**23 + 0.5 + 2**-37 lies just above the fp32 midpoint
    # 2**23 + 0.5; fp64 rounds it onto the midpoint, and a second rounding to
    # fp32 would then pick the even neighbour 2**23.  One rounding gives 2**23+1.
    assert float(a) * float(b) + float(c) == 2.0 ** 23 + 0.5
    assert fp32.fma(a, b, c) == np.float32(2.0 ** 23 + 1)
    assert fp32.fma(-a, b, -c) == np.float32(-(2.0 ** 23 + 1))
    # without the tail the tie goes to even
    assert fp32.fma(np.float32(0.5), np.float32(1.0), c) == np.float32(2.0 ** 23)


def test_mul_is_numpy_fp32_product():
    rng = np.random.default_rng(3)
    a = rng.standard_normal(10000).astype(np.float32)
    b = rng.standard_normal(10000).astype(np.float32)
    assert np.array_equal(fp32.mul(a, b), a * b)
