"""Pins for the fitted row quantiser (Sec. 3, Levels and storage)."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import quant


def _rows(rng, n, dv=128, dist="normal"):
    if dist == "uniform":
        return rng.uniform(-1, 1, (n, dv)).astype(np.float32)
    if dist == "t3":
        return rng.standard_t(3, (n, dv)).astype(np.float32)
    return rng.standard_normal((n, dv)).astype(np.float32)


@pytest.mark.parametrize("b", [2, 3, 4, 6, 8])
def test_p16_fit_is_argmin_of_exact_error(b):
    rng = np.random.default_rng(16 + b)
    x = _rows(rng, 12, 64, "t3")
    codes, scale, mstar = quant.quantize_rows(x, np.full(12, b))
    R = np.max(np.abs(x), axis=1)
    for r in range(12):
        exact = []
        for m in range(16):
            c, d, _ = quant.candidate(x[r:r + 1], R[r:r + 1], b, m)
            D = Fraction(float(d[0]))
            exact.append(sum((Fraction(float(xx)) - int(cc) * D) ** 2 for xx, cc in zip(x[r], c[0])))
        lo = min(exact)
        assert exact[mstar[r]] <= lo * (1 + Fraction(1, 2 ** 16))
        # scale is the FP16 of f R / n for the chosen clip factor
        n = 2 ** (b - 1) - 1
        f = quant.clip_factor(mstar[r])
        assert float(scale[r]) == pytest.approx(f * float(R[r]) / n, rel=2 ** -10)


@pytest.mark.parametrize("b", [2, 3, 5, 8, 12])
def test_p14_codes_are_nearest_clamped_levels(b):
    rng = np.random.default_rng(140 + b)
    x = _rows(rng, 40, 128)
    codes, scale, _ = quant.quantize_rows(x, np.full(40, b))
    n = 2 ** (b - 1) - 1
    assert codes.min() >= -n and codes.max() <= n
    d = scale.astype(np.float64)[:, None]
    err = np.abs(x - codes * d)
    for delta in (-1, 1):
        alt = np.clip(codes + delta, -n, n)
        assert np.all(err <= np.abs(x - alt * d) + 1e-6 * np.abs(x))
    inside = np.abs(x) <= n * d
    assert np.all(err[inside] <= 0.5 * np.broadcast_to(d, x.shape)[inside] * (1 + 1e-5))


def test_p14_ternary_and_one_bit():
    rng = np.random.default_rng(141)
    x = _rows(rng, 10, 64)
    codes, _, _ = quant.quantize_rows(x, np.full(10, 2))
    assert set(np.unique(codes)) <= {-1, 0, 1}
    x[0, 3] = -0.0
    codes1, scale1, _ = quant.quantize_rows(x, np.full(10, 1))
    assert codes1[0, 3] == 0
    np.testing.assert_allclose(scale1.astype(np.float64), np.mean(np.abs(x), axis=1), rtol=1e-3)
    xh = quant.dequantize_rows(codes1, scale1, np.full(10, 1))
    assert np.all(np.sign(xh[x != 0]) == np.sign(x[x != 0]))
    assert np.all(np.abs(xh) == scale1.astype(np.float32)[:, None])


@pytest.mark.parametrize("b", [6, 8])
def test_p13_single_writeback_mse_is_delta2_over_12(b):
    rng = np.random.default_rng(13 + b)
    x = _rows(rng, 3000, 128, "uniform")
    codes, scale, _ = quant.quantize_rows(x, np.full(3000, b))
    xh = quant.dequantize_rows(codes, scale, np.full(3000, b)).astype(np.float64)
    d = scale.astype(np.float64)
    ratio = np.mean(np.mean((x - xh) ** 2, axis=1) / (d ** 2 / 12))
    assert ratio == pytest.approx(1.0, abs=0.03)


def test_zero_row_and_saturation():
    x = np.zeros((2, 64), np.float32)
    x[1, 0] = 1e6
    codes, scale, mstar = quant.quantize_rows(x, np.array([4, 2]))
    assert np.all(codes[0] == 0) and scale[0] == 0 and mstar[0] == 0
    assert scale[1] == np.float16(65504)


def test_first_strict_minimum_tie_break():
    # a row whose every element is exactly representable by two candidates
    # with zero error: the smaller clip factor wins
    x = np.zeros((1, 64), np.float32)
    codes, scale, mstar = quant.quantize_rows(x, np.array([3]))
    assert mstar[0] == 0
