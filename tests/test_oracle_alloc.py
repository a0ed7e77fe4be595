"""Pins for range normalisation and bit allocation (Sec. 3, eq. weight, eq. alloc)."""
import numpy as np
import pytest

from oracle import alloc


def test_p9_real_valued_budget_and_am_gm():
    rng = np.random.default_rng(9)
    c = np.exp(rng.normal(0, 2, 50))
    b = alloc.real_allocation(c, 4.0)
    assert np.sum(b) == pytest.approx(50 * 4.0, rel=1e-13)
    # distortion ratio uniform / optimal equals AM(c)/GM(c)
    uni = np.sum(c * 2.0 ** (-2 * 4.0))
    opt = np.sum(c * 2.0 ** (-2 * b))
    assert uni / opt == pytest.approx(alloc.am_gm_gain(c), rel=1e-12)


@pytest.mark.parametrize("trial", range(60))
def test_p10_integer_allocation_equals_bruteforce(trial):
    rng = np.random.default_rng(100 + trial)
    N = int(rng.integers(2, 6))
    b_min, b_max = [(1, 8), (2, 8), (1, 4)][trial % 3]
    mean = [2.0, 3.0, 2.5, 4.0][trial % 4]
    if mean > b_max:
        mean = b_max - 0.5
    c = np.exp(rng.normal(0, 3, N))
    if trial % 7 == 0:
        c[0] = 0.0
    b = alloc.allocate(c, mean, b_min, b_max)
    K = alloc.budget(mean, N)
    assert b.sum() == K and b.min() >= b_min and b.max() <= b_max
    best, _ = alloc.allocate_bruteforce(c, mean, b_min, b_max)
    assert alloc.proxy(c, b) == pytest.approx(best, rel=1e-12, abs=0)


def test_p10_budget_errors():
    with pytest.raises(alloc.BudgetError):
        alloc.allocate(np.ones(4), 1.5, 2, 8)
    with pytest.raises(alloc.BudgetError):
        alloc.allocate(np.ones(4), 9.0, 2, 8)


def test_p11_scale_invariance():
    rng = np.random.default_rng(11)
    c = np.exp(rng.normal(0, 2, 300))
    b = alloc.allocate(c, 3.0, 1, 8)
    for kappa in (2.0 ** -7, 4.0, 2.0 ** 30):
        assert np.array_equal(alloc.allocate(c * kappa, 3.0, 1, 8), b)
    assert np.array_equal(alloc.allocate(c * 3.7, 3.0, 1, 8), b)


def test_ties_go_to_lower_row():
    b = alloc.allocate(np.ones(4), 2.5, 2, 8)
    assert list(b) == [3, 3, 2, 2]
    b = alloc.allocate(np.zeros(4), 2.25, 2, 8)
    assert list(b) == [3, 2, 2, 2]


def test_p12_normalized_ranges():
    rng = np.random.default_rng(12)
    R = np.abs(rng.standard_normal((3, 128))).astype(np.float32)
    Rt = alloc.normalized_ranges(R, 64)
    for g in range(2):
        rms = np.sqrt(np.mean(Rt[:, 64 * g:64 * g + 64] ** 2, axis=1))
        np.testing.assert_allclose(rms, 1.0, rtol=1e-14)
    assert np.all(alloc.normalized_ranges(np.full((1, 32), 5.0, np.float32), 32) == 1.0)
    assert np.all(alloc.normalized_ranges(np.zeros((1, 32), np.float32), 32) == 0.0)


def test_allocation_orders_by_weight():
    # more weight never gets fewer bits
    rng = np.random.default_rng(13)
    c = np.exp(rng.normal(0, 2, 500))
    b = alloc.allocate(c, 4.0, 2, 8)
    o = np.argsort(c)
    assert np.all(np.diff(b[o]) >= 0)


def test_p12_groups_spanning_heads():
    # Mamba-2 normalises over groups of several heads: the RMS of R~ is 1 over
    # each group of consecutive rows, whichever heads they belong to
    rng = np.random.default_rng(14)
    B, H, dk = 2, 6, 16
    R = np.abs(rng.standard_normal((B, H * dk))).astype(np.float32)
    Rt = alloc.normalized_ranges(R, 3 * dk)
    for g in range(2):
        rms = np.sqrt(np.mean(Rt[:, 3 * dk * g:3 * dk * (g + 1)] ** 2, axis=1))
        np.testing.assert_allclose(rms, 1.0, rtol=1e-14)


def test_group_rms_runs():
    # the group sum of squares is formed in runs of 64 rows: for groups of at
    # most 64 rows that is the plain row-order sum; for a group of 12 heads of
    # 128 rows (1536) it stays within a few units of the exactly rounded sum
    import math
    rng = np.random.default_rng(15)
    R = np.abs(rng.standard_normal((2, 1536)) * np.exp(rng.normal(0, 2, (2, 1536)))).astype(np.float32)
    for G in (16, 64):
        Rt = alloc.normalized_ranges(R, G)
        for g0 in range(0, 1536, G):
            acc = 0.0
            for j in range(g0, g0 + G):
                acc = acc + float(R[0, j]) * float(R[0, j])
            assert np.array_equal(Rt[0, g0:g0 + G], R[0, g0:g0 + G].astype(np.float64) / np.sqrt(acc / G))
    Rt = alloc.normalized_ranges(R, 1536)
    for b in range(2):
        exact = math.sqrt(math.fsum(float(r) * float(r) for r in R[b]) / 1536)
        got = float(R[b, 0]) / Rt[b, 0]
        assert abs(got - exact) <= 8 * np.spacing(exact)
