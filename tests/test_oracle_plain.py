"""Pins of the plain validity checks (oracle/plain.py).

The checks must accept exactly the optimal width vectors (brute force over
every vector on tiny scopes), agree with exact rational arithmetic on the
clip-factor argmin, accept the float32 contract's outputs, and reject
planted mistakes: a bit moved to a less valuable row, another candidate's
scale, a code off by one, a flipped sign bit.
"""
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import alloc, plain, quant

F32 = np.float32


def test_fp16_rounding_is_exact():
    rng = np.random.default_rng(0)
    v = np.exp(rng.uniform(np.log(1e-7), np.log(7e4), 4000))
    h = plain.fp16_sat(v)
    for a, b in zip(v[:600], h[:600]):
        assert b == plain.fp16_of_fraction(Fraction(float(a)))
    assert plain.fp16_sat(np.array([1e6]))[0] == 65504.0
    # a midpoint between two FP16 values rounds to the even one
    assert plain.fp16_of_fraction(Fraction(2049, 2048)) == 1.0
    assert plain.fp16_of_fraction(Fraction(2051, 2048)) == float(np.float16(1.0 + 2 ** -9))


def test_group_rms_plain():
    R = np.array([[3.0, 4.0, 2.0, 2.0]], F32)
    rms = plain.group_rms(R, 2)
    assert np.allclose(rms, [[math.sqrt(12.5)] * 2 + [2.0] * 2], rtol=0, atol=0)
    c = plain.keys(np.full((1, 4), 2.5), np.full((1, 4), 7.0, F32), 4)
    assert np.all(c == 2.5)


def _proxy(c, b):
    return sum(Fraction(float(ci)) * Fraction(1, 4 ** int(bi)) for ci, bi in zip(c, b))


@pytest.mark.parametrize("seed", range(40))
def test_widths_accept_exactly_the_minimisers(seed):
    rng = np.random.default_rng(seed)
    N = int(rng.integers(2, 6))
    b_min, b_max = (1, 4) if seed % 2 else (2, 5)
    mean = float(rng.integers(b_min * 4, b_max * 4 + 1)) / 4.0
    c = np.exp(rng.normal(0, 2, N))
    if seed % 5 == 0:
        c[1] = c[0]                      # a tie
    if seed % 7 == 0:
        c[-1] = 0.0                      # a zero key
    K = alloc.budget(mean, N)
    vecs = [b for b in itertools.product(range(b_min, b_max + 1), repeat=N) if sum(b) == K]
    best = min(_proxy(c, b) for b in vecs)
    for b in vecs:
        res = plain.check_widths(c, np.array(b), mean, b_min, b_max)
        assert res["ok"] == (_proxy(c, b) == best), (c, b)
        if res["ok"]:
            assert res["exempt"] == 0


def test_widths_accept_the_allocator_and_reject_a_moved_bit():
    rng = np.random.default_rng(1)
    c = np.exp(rng.normal(0, 3, 4096))
    b = alloc.allocate(c, 4.0, 2, 8)
    res = plain.check_widths(c, b, 4.0, 2, 8)
    assert res["ok"] and res["exempt"] == 0
    # move one bit from the most valuable granted slot to the least valuable open one
    last = np.ldexp(c, -2 * b)
    nxt = np.ldexp(c, -2 * (b + 1))
    i = int(np.argmax(np.where(b > 2, last, -np.inf)))
    j = int(np.argmin(np.where(b < 8, nxt, np.inf)))
    b2 = b.copy()
    b2[i] -= 1
    b2[j] += 1
    assert not plain.check_widths(c, b2, 4.0, 2, 8)["ok"]
    # a budget violation
    b3 = b.copy()
    b3[j] += 1
    assert not plain.check_widths(c, b3, 4.0, 2, 8)["ok"]


@pytest.mark.parametrize("seed", range(12))
def test_fit_argmin_matches_rational_arithmetic(seed):
    rng = np.random.default_rng(100 + seed)
    L = 12
    for _ in range(6):
        b = int(rng.integers(2, 7))
        x = (rng.standard_normal(L) * np.exp(rng.normal(0, 1))).astype(F32)
        if seed % 3 == 0:
            x[0] *= 6                                  # a clipped outlier
        m = plain.fit_exact_rational(x, b)
        _, d = plain.candidate_scales(np.array([np.max(np.abs(x))], F32), b)
        n = (1 << (b - 1)) - 1
        E = [plain.errors(x[None], d[:, k], n)[0] for k in range(16)]
        assert int(np.argmin(E)) == m or E[int(np.argmin(E))] == E[m]
        codes, _ = plain.nearest_codes(x[None], d[:, m], n)
        res = plain.check_fit(x[None], np.array([b]), d[:, m].astype(np.float16),
                              codes.astype(np.int64))
        assert res["bad_scale"] == res["bad_fit"] == res["bad_codes"] == 0


@pytest.mark.parametrize("b", [1, 2, 3, 4, 6, 8])
def test_fit_accepts_the_contract(b):
    rng = np.random.default_rng(b)
    x = rng.standard_normal((300, 128)).astype(F32)
    x[:20] *= np.exp(rng.normal(0, 4, (20, 1))).astype(F32)
    x[20] = 0.0
    widths = np.full(300, b)
    codes, scale, _ = quant.quantize_rows(x, widths)
    res = plain.check_fit(x, widths, scale, codes)
    assert res["bad_scale"] == res["bad_fit"] == res["bad_codes"] == 0, plain.summary("c", res)
    assert res["exempt_fit"] + res["exempt_scale"] <= 3
    assert res["exempt_codes"] <= 5


def test_fit_rejects_planted_mistakes():
    rng = np.random.default_rng(7)
    x = rng.standard_normal((64, 128)).astype(F32)
    widths = np.full(64, 4)
    codes, scale, mstar = quant.quantize_rows(x, widths)
    # another candidate's scale (with its own nearest codes): at least the
    # candidates far from the optimum must be rejected
    R = np.max(np.abs(x), axis=1)
    _, d = plain.candidate_scales(R, 4)
    far = (mstar + 8) % 16
    d2 = d[np.arange(64), far]
    c2, _ = plain.nearest_codes(x, d2, 7)
    res = plain.check_fit(x, widths, d2.astype(np.float16), c2.astype(np.int64))
    assert res["bad_fit"] >= 60
    # a scale that is no candidate's
    sc = scale.copy()
    sc[3] = np.float16(float(sc[3]) * 1.01)
    assert plain.check_fit(x, widths, sc, codes)["bad_scale"] >= 1
    # a code off by one away from a midpoint
    cc = codes.copy()
    j = int(np.argmin(np.abs(np.abs(x[5]) - 0.3)))
    cc[5, j] += 1 if cc[5, j] < 7 else -1
    assert plain.check_fit(x, widths, scale, cc)["bad_codes"] == 1
    # one-bit rows: a flipped sign bit and a wrong mean
    w1 = np.ones(64, np.int64)
    c1, s1, _ = quant.quantize_rows(x, w1)
    assert plain.check_fit(x, w1, s1, c1)["bad_codes"] == 0
    c1[2, 9] ^= 1
    assert plain.check_fit(x, w1, s1, c1)["bad_codes"] == 1
    s1[4] = np.float16(float(s1[4]) * 1.01)
    assert plain.check_fit(x, w1, s1, quant.quantize_rows(x, w1)[0])["bad_scale"] == 1


def test_block_groups_accept_the_contract():
    # head units: scale groups of 32 rows of one column, checked as rows of 32
    rng = np.random.default_rng(3)
    x = rng.standard_normal((64, 32)).astype(F32)
    for b in (2, 5):
        codes, bscale, _ = quant.quantize_blocks(x, b)
        g = x.reshape(2, 32, 32).transpose(0, 2, 1).reshape(-1, 32)
        cg = codes.reshape(2, 32, 32).transpose(0, 2, 1).reshape(-1, 32)
        res = plain.check_fit(g, np.full(64, b), bscale.reshape(-1), cg)
        assert res["bad_scale"] == res["bad_fit"] == res["bad_codes"] == 0


def test_double_rounded_scales_are_exempt_not_failed():
    """Rows of +-R where the contract's float32 product R fl32(f/n) lands on
    an FP16 midpoint the exact f R / n does not: the contract stores the
    other FP16 neighbour; the check counts it as exempt."""
    rng = np.random.default_rng(3)
    b, m = 5, 15
    phi = quant.phi_table(b)[m]
    R = np.float32(0.37)
    rows = []
    while len(rows) < 4:
        R = np.nextafter(R, np.float32(np.inf))
        p = np.float32(R * phi)
        h = np.float16(p)
        v = Fraction(float(R)) * Fraction(5 + m, 20 * 15)
        if float(h) != plain.fp16_of_fraction(v):
            rows.append(R)
    x = np.stack([np.where(rng.random(64) < 0.5, -1.0, 1.0).astype(F32) * r for r in rows])
    widths = np.full(len(rows), b)
    codes, scale, mstar = quant.quantize_rows(x, widths)
    res = plain.check_fit(x, widths, scale, codes)
    assert res["bad_scale"] == res["bad_fit"] == res["bad_codes"] == 0
    assert res["exempt_scale"] >= 1
