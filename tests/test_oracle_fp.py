"""Pins for the exact float helpers: fma32 against rational arithmetic."""
from fractions import Fraction

import numpy as np

from oracle.fp import fma32, fp16_sat, halving_tree


def _round_f32(fr):
    """Nearest float32 (ties to even) of a Fraction, by exhaustive neighbour check."""
    x = np.float32(float(fr))          # within an ulp or so
    cands = {x, np.nextafter(x, np.float32(np.inf)), np.nextafter(x, np.float32(-np.inf))}
    best = None
    for c in cands:
        d = abs(Fraction(float(c)) - fr)
        key = (d, int(np.frombuffer(np.float32(c).tobytes(), np.uint32)[0]) & 1)
        if best is None or key < best[0]:
            best = (key, c)
    return np.float32(best[1])


def test_fma32_random_matches_rational():
    rng = np.random.default_rng(1)
    a = rng.standard_normal(3000).astype(np.float32)
    b = rng.standard_normal(3000).astype(np.float32) * np.float32(2.0) ** rng.integers(-30, 30, 3000)
    c = rng.standard_normal(3000).astype(np.float32)
    r = fma32(a, b, c)
    for i in range(3000):
        ex = Fraction(float(a[i])) * Fraction(float(b[i])) + Fraction(float(c[i]))
        assert r[i] == _round_f32(ex), i


def test_fma32_double_rounding_midpoint():
    # a*b = 1 - 2^-46 exactly; c = 2^24 + 2.  The float64 sum rounds to
    # 2^24 + 3, a float32 midpoint, which a float64-then-float32 evaluation
    # rounds to the even 2^24 + 4; the exact value lies below the midpoint.
    a = np.float32(1.0 + 2.0 ** -23)
    b = np.float32(1.0 - 2.0 ** -23)
    c = np.float32(2.0 ** 24 + 2)
    ex = Fraction(float(a)) * Fraction(float(b)) + Fraction(float(c))
    naive = np.float32(np.float64(a) * np.float64(b) + np.float64(c))
    assert naive == np.float32(2.0 ** 24 + 4)
    assert _round_f32(ex) == np.float32(2.0 ** 24 + 2)
    assert fma32(a, b, c) == np.float32(2.0 ** 24 + 2)
    # mirrored case above the midpoint
    assert fma32(-a, b, -c) == np.float32(-(2.0 ** 24 + 2))


def test_fma32_exact_midpoint_ties_even():
    # a*b + c exactly equal to a float32 midpoint: ties to even
    a = np.float32(2.0 ** -24)
    b = np.float32(1.0)
    c = np.float32(1.0)
    assert fma32(a, b, c) == np.float32(1.0)
    c2 = np.float32(1.0 + 2.0 ** -23)
    assert fma32(a, b, c2) == np.float32(1.0 + 2.0 ** -22)


def test_fp16_saturates_and_rounds_even():
    assert fp16_sat(np.float32(1e6)) == np.float16(65504)
    assert fp16_sat(np.float32(65519.0)) == np.float16(65504)
    assert fp16_sat(np.float32(1.0 + 2.0 ** -11)) == np.float16(1.0)
    assert fp16_sat(np.float32(1.0 + 3 * 2.0 ** -11)) == np.float16(1.0 + 2.0 ** -9)


def test_halving_tree_order():
    p = [np.float32(x) for x in (1e8, 1.0, -1e8, 1.0)]
    # (p0 + p2) + (p1 + p3) = 0 + 2 = 2 ; a left fold would give 1
    assert halving_tree(p) == np.float32(2.0)
