"""Pins for the Gramian weights, EMAs and rate codes (Prop. 1, Sec. 2-3)."""
import json
import os

import numpy as np
import pytest

from oracle import stats

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))


def _closed_finite(lam, W):
    return (lam / (1 - lam)) * ((W - 1) - lam * (1 - lam ** (W - 1)) / (1 - lam)) / W


@pytest.mark.parametrize("s", [0.05, 0.003, 0.7])
def test_p5_no_erasure_closed_form(s):
    W = 1024
    q = np.ones((W, 3), np.float32)
    sv = np.full((W, 3), s, np.float32)
    k = np.zeros((W, 3), np.float32)
    beta = np.zeros(W, np.float32)
    g = stats.window_gamma(q, sv, k, beta, C=1)
    lam = np.exp(-2 * np.float64(np.float32(s)))
    np.testing.assert_allclose(g, _closed_finite(lam, W), rtol=1e-12)
    # W -> infinity: 1/expm1(2 s) = DAMP's 1/(1-a^2) times exp(-2 s)
    a = np.exp(-np.float64(s))
    lim = 1 / np.expm1(2 * np.float64(s))
    assert lim == pytest.approx(np.exp(-2 * s) / (1 - a * a), rel=1e-12)
    gl = stats.window_gamma(np.ones((20000, 1), np.float32), np.full((20000, 1), s, np.float32),
                            np.zeros((20000, 1), np.float32), np.zeros(20000, np.float32), C=1)
    assert gl[0] == pytest.approx(lim * (1 - 1 / 20000 / (1 - lam)), rel=1e-3)


def test_p5_window_writeback_interval():
    # with write-backs every C tokens the diagonal sum carries the 1/C of eq. gram
    W, s = 4096, 0.01
    args = (np.ones((W, 1), np.float32), np.full((W, 1), s, np.float32),
            np.zeros((W, 1), np.float32), np.zeros(W, np.float32))
    g1 = stats.window_gamma(*args, C=1)
    g8 = stats.window_gamma(*args, C=8)
    assert g8[0] == pytest.approx(g1[0] / 8, rel=0.02)


def test_p6_worked_example_matches_paper():
    ex = GOLD["worked_example"]
    for dk in (2, 8):
        k = np.zeros(dk); k[:2] = 1 / np.sqrt(2)
        F = stats.transition(k, 0.01, 0.5)
        g = stats.stationary_gamma(F, np.eye(dk))
        assert round(g[0], 1) == ex["exact_gamma"]
        # the paper's approximation, r = E[beta (2-beta) k_i^2] / 2
        r = 0.5 * 0.5 * 1.5 * 0.5
        approx = stats.gamma_hat(0.01, r)
        assert round(float(approx), 2) == ex["approx_gamma"]


def test_p7_fixed_key_series_equals_lyapunov():
    for beta in (0.5, 1.0, 1.7):
        k = np.zeros(6); k[:3] = 1 / np.sqrt(3)
        s = 0.02
        g = stats.stationary_gamma(stats.transition(k, s, beta), np.eye(6))
        L = np.arange(1, 20000)
        cl = 1 - (1 - beta) ** L
        for i in (0, 4):
            series = np.sum(np.exp(-2 * s * L) * (1 - 2 * cl * k[i] ** 2 + cl ** 2 * k[i] ** 2))
            assert g[i] == pytest.approx(series, rel=1e-9)


def test_p8_per_head_bound_random_keys():
    rng = np.random.default_rng(8)
    dk, W, s = 8, 400, 0.02
    for C in (1, 4):
        qs = rng.standard_normal((W, dk)); qs /= np.linalg.norm(qs, axis=1, keepdims=True)
        ks = rng.standard_normal((W, dk)); ks /= np.linalg.norm(ks, axis=1, keepdims=True)
        betas = rng.uniform(0, 2, W)
        Fs = np.stack([stats.transition(ks[t], s, betas[t]) for t in range(W)])
        g = stats.exact_window_gamma(qs, Fs, C)
        assert np.all(g <= 1.0 / (C * np.expm1(2 * s)) * (1 + 1e-12))


def test_window_gamma_equals_exact_without_erasure():
    rng = np.random.default_rng(9)
    dk, W = 4, 300
    qs = rng.standard_normal((W, dk)).astype(np.float32)
    s = np.exp(rng.uniform(-6, 0, (W, dk))).astype(np.float32)
    Fs = np.stack([np.diag(np.exp(-s[t].astype(np.float64))) for t in range(W)])
    for C in (1, 3):
        g = stats.window_gamma(qs, s, np.zeros((W, dk), np.float32), np.zeros(W, np.float32), C)
        ge = stats.exact_window_gamma(qs.astype(np.float64), Fs, C)
        np.testing.assert_allclose(g, ge, rtol=1e-11)


def test_window_gamma_diagonal_erase_term():
    # A fixed key along basis vector 0: the exact squared per-token factor of
    # row 0 is exp(-2 s) (1 - beta)^2 = exp(-2 s) (1 - beta (2 - beta)); the
    # weight's erase term replaces 1 - x by exp(-x).  So the diagonal sum is
    # an upper bound there and agrees to first order in beta; row 1 (never
    # erased) is exact.
    W, s = 500, 0.01
    for beta in (0.6, 0.02):
        q = np.ones((W, 2), np.float32)
        k = np.zeros((W, 2), np.float32); k[:, 0] = 1
        g = stats.window_gamma(q, np.full((W, 2), s, np.float32), k,
                               np.full(W, beta, np.float32), 1)
        a = np.exp(-np.float64(np.float32(s)))
        b = np.float64(np.float32(beta))
        Fs = np.stack([np.diag([a * (1 - b), a])] * W)
        ge = stats.exact_window_gamma(np.ones((W, 2)), Fs, 1)
        assert g[1] == pytest.approx(ge[1], rel=1e-10)
        assert g[0] >= ge[0]
        if beta < 0.1:
            # per-token factors differ by O(x^2), x = beta (2 - beta); summed
            # over the ~1/(2 s + x) effective lags the gap stays small
            assert g[0] == pytest.approx(ge[0], rel=0.02)


def test_p17_logq_monotone_half_step():
    s = np.exp(np.linspace(np.log(2.0 ** -19.9), np.log(2.0 ** 4.9), 50001))
    z = stats.logq_encode(s)
    assert np.all(np.diff(z.astype(np.int64)) >= 0)
    d = stats.logq_decode(z)
    assert np.max(np.abs(np.log2(d) - np.log2(s))) <= 0.5 * 25 / 65535 * (1 + 1e-9)
    lv = np.log2(stats.logq_decode(np.arange(0, 65536, 997, dtype=np.uint16)))
    np.testing.assert_allclose(np.diff(lv), 997 * 25 / 65535, rtol=1e-9)
    assert stats.logq_encode(0.0) == 0 and stats.logq_encode(1e9) == 65535


def test_p18_ema_constant_and_span_one():
    s = np.full(5, 0.03, np.float32)
    k = np.full(5, 0.3, np.float32)
    m, e = stats.ema_init(s, k, np.float32(0.4))
    m0, e0 = m.copy(), e.copy()
    for _ in range(50):
        m, e = stats.ema_update(m, e, s, k, np.float32(0.4), 64)
    np.testing.assert_allclose(m, m0, rtol=1e-14)
    np.testing.assert_allclose(e, e0, rtol=1e-14)
    m1, e1 = stats.ema_update(m, e, np.full(5, 0.5, np.float32), k, np.float32(0.9), 1)
    assert np.array_equal(m1, stats.decay_sample(np.full(5, 0.5, np.float32)))
    assert np.array_equal(e1, stats.erase_sample(k, np.float32(0.9)))
    sh, r = stats.ema_rates(m0, e0)
    np.testing.assert_allclose(sh, 0.03, rtol=1e-6)
    np.testing.assert_allclose(r, 0.5 * 0.4 * 1.6 * 0.09, rtol=1e-6)


@pytest.mark.parametrize("s", [0.05, 0.5])
def test_no_erasure_window_weights_are_the_closed_form(s):
    # Prop. 1: constant diagonal decay without erasure gives rho / expm1(2 s);
    # with a = 0 the keys and beta must drop out of the window weights
    W = 1024
    rng = np.random.default_rng(23)
    k = rng.standard_normal((W, 4)).astype(np.float32)
    beta = rng.uniform(0, 2, W).astype(np.float32)
    g = stats.window_gamma(np.ones((W, 4), np.float32), np.full((W, 4), s, np.float32), k, beta,
                           C=1, erase=False)
    lam = np.exp(-2 * np.float64(np.float32(s)))
    np.testing.assert_allclose(g, _closed_finite(lam, W), rtol=1e-12)


@pytest.mark.parametrize("C", [1, 3])
def test_no_erasure_exact_gramian_is_the_diagonal_recursion(C):
    # F = diag(exp(-s)) has a diagonal Gramian: the matrix recursion and the
    # per-row recursion are two computations of the same numbers
    rng = np.random.default_rng(24)
    W, dk = 40, 5
    qs = rng.standard_normal((W, dk)).astype(np.float32)
    ss = np.exp(rng.uniform(np.log(1e-3), 0, (W, dk))).astype(np.float32)
    ks = rng.standard_normal((W, dk)).astype(np.float32)
    bs = rng.uniform(0, 1, W).astype(np.float32)
    Fs = np.stack([stats.transition(ks[t], ss[t].astype(np.float64), bs[t], erase=False)
                   for t in range(W)])
    ge = stats.exact_window_gamma(qs.astype(np.float64), Fs, C)
    gw = stats.window_gamma(qs, ss, ks, bs, C, erase=False)
    np.testing.assert_allclose(ge, gw, rtol=1e-12)
