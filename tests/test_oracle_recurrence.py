"""Pins for the gated delta rule (Sec. 2, eq. rule)."""
import numpy as np

from oracle import recurrence as rec


def _inputs(rng, dk=64, dv=64):
    q = rng.standard_normal(dk); q /= np.linalg.norm(q)
    k = rng.standard_normal(dk); k /= np.linalg.norm(k)
    v = rng.standard_normal(dv)
    s = np.exp(rng.uniform(np.log(1e-3), 0, dk))
    beta = 1 / (1 + np.exp(-rng.standard_normal()))
    return q, k, v, s, beta


def test_p1_rowform_equals_dense_definition():
    rng = np.random.default_rng(0)
    S = rng.standard_normal((64, 64))
    for _ in range(5):
        q, k, v, s, beta = _inputs(rng)
        Sd, od = rec.truth_step(S, q, k, v, s, beta)
        Sr, orow = rec.truth_step_rowform(S, q, k, v, s, beta)
        np.testing.assert_allclose(Sr, Sd, rtol=0, atol=1e-12)
        np.testing.assert_allclose(orow, od, rtol=0, atol=1e-12)
        S = Sd


def test_p1_mirror_tracks_truth_within_float32():
    rng = np.random.default_rng(1)
    S = rng.standard_normal((2, 3, 64, 64)).astype(np.float32)
    q = rng.standard_normal((2, 3, 64)); q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k = rng.standard_normal((2, 3, 64)); k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((2, 3, 64))
    s = np.exp(rng.uniform(-5, 0, (2, 3, 64)))
    beta = rng.uniform(0, 1, (2, 3))
    args = [a.astype(np.float32) for a in (q, k, v, s, beta)]
    Sm, om = rec.mirror_step(S, *args)
    St, ot = rec.truth_step_rowform(S.astype(np.float64), *[a.astype(np.float64) for a in args])
    assert np.max(np.abs(Sm - St)) <= 64 * 2.0 ** -23 * np.max(np.abs(St))
    assert np.max(np.abs(om - ot)) <= 64 * 2.0 ** -23 * np.max(np.abs(St))


def test_p2_pure_decay():
    rng = np.random.default_rng(2)
    S0 = rng.standard_normal((64, 32))
    S = S0.copy()
    tot = np.zeros(64)
    for _ in range(20):
        q, k, v, s, _ = _inputs(rng, 64, 32)
        S, _ = rec.truth_step(S, q, k, v, s, 0.0)
        tot += s
    np.testing.assert_allclose(S, np.exp(-tot)[:, None] * S0, rtol=1e-12, atol=0)


def test_p3_beta0_s0_identity_bit_exact():
    rng = np.random.default_rng(3)
    S = rng.standard_normal((4, 64, 64)).astype(np.float32)
    q = rng.standard_normal((4, 64)).astype(np.float32)
    k = rng.standard_normal((4, 64)).astype(np.float32)
    v = rng.standard_normal((4, 64)).astype(np.float32)
    S1, o = rec.mirror_step(S, q, k, v, np.zeros((4, 64), np.float32), np.zeros(4, np.float32))
    assert np.array_equal(S1, S)
    np.testing.assert_allclose(o, np.einsum("bi,bij->bj", q.astype(np.float64), S), rtol=1e-5, atol=1e-5)


def test_p4_delta_rule_recall():
    rng = np.random.default_rng(4)
    S = rng.standard_normal((64, 64))
    _, k, v, _, _ = _inputs(rng)
    S1, _ = rec.truth_step(S, np.zeros(64), k, v, np.zeros(64), 1.0)
    np.testing.assert_allclose(S1.T @ k, v, rtol=0, atol=1e-12)
    Sm, _ = rec.mirror_step(S.astype(np.float32), np.zeros(64, np.float32), k.astype(np.float32),
                            v.astype(np.float32), np.zeros(64, np.float32), np.float32(1.0))
    np.testing.assert_allclose(Sm.astype(np.float64).T @ k, v, rtol=0, atol=1e-4)


def test_blockdot_order_is_the_contract():
    # block partials combined by halving: with four blocks, (p0+p2)+(p1+p3)
    x = np.ones(128, np.float32)
    M = np.zeros((128, 1), np.float32)
    M[0, 0], M[64, 0], M[32, 0], M[96, 0] = 1e8, -1e8, 1.0, 1.0
    assert rec.blockdot(x, M)[0] == np.float32(2.0)


def test_no_erasure_is_the_decayed_sum_of_writes():
    # without erasure (a = 0, Mamba-2) eq. rule is the linear recurrence
    # S_T = diag(exp(-sum s)) S_0 + sum_t diag(exp(-sum_{tau>t} s_tau)) beta_t k_t v_t^T
    rng = np.random.default_rng(21)
    dk, dv, T = 16, 8, 12
    S0 = rng.standard_normal((dk, dv))
    ins = [_inputs(rng, dk, dv) for _ in range(T)]
    S = S0.copy()
    for q, k, v, s, beta in ins:
        Sd, _ = rec.truth_step(S, q, k, v, s, beta, erase=False)
        Sr, _ = rec.truth_step_rowform(S, q, k, v, s, beta, erase=False)
        np.testing.assert_allclose(Sr, Sd, rtol=0, atol=1e-12)
        S = Sd
    ssum = np.sum([x[3] for x in ins], axis=0)
    want = np.exp(-ssum)[:, None] * S0
    for t, (q, k, v, s, beta) in enumerate(ins):
        later = np.sum([x[3] for x in ins[t + 1:]], axis=0) if t + 1 < T else np.zeros(dk)
        want += np.exp(-later)[:, None] * beta * np.outer(k, v)
    np.testing.assert_allclose(S, want, rtol=1e-12, atol=1e-12)


def test_no_erasure_mirror_tracks_truth():
    rng = np.random.default_rng(22)
    S = rng.standard_normal((2, 64, 64)).astype(np.float32)
    q = rng.standard_normal((2, 64)); q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k = rng.standard_normal((2, 64)); k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((2, 64))
    s = np.exp(rng.uniform(-5, 0, (2, 1)))
    beta = rng.uniform(0, 1, 2)
    args = [a.astype(np.float32) for a in (q, k, v, s, beta)]
    Sm, om = rec.mirror_step(S, *args, erase=False)
    St, ot = rec.truth_step_rowform(S.astype(np.float64), *[a.astype(np.float64) for a in args],
                                    erase=False)
    assert np.max(np.abs(Sm - St)) <= 4 * 2.0 ** -23 * np.max(np.abs(St))
    assert np.max(np.abs(om - ot)) <= 64 * 2.0 ** -23 * np.max(np.abs(St))
