"""GPU parity of kda_alloc_bits and kda_weights against the oracle; widths
also against the plain optimality condition of the allocation
(oracle/plain.py)."""
import numpy as np
import pytest
import torch

import paper_2609_30950_amd as K
import workloads as W
from oracle import alloc, plain, stats
from tests._gpu import dev, host, say


def _plain_widths(gamma, R, G, scope, mean, bmin, bmax, got, label):
    """The GPU's widths minimise sum c 4^-b over each scope unit, with keys
    from plain group sums of squares."""
    B, H, d = gamma.shape
    if G <= d:
        c = plain.keys(gamma, R, G)
    else:
        c = plain.keys(gamma.reshape(B, H * d), R.reshape(B, H * d), G).reshape(B, H, d)
    units = [(b, slice(None)) for b in range(B)] if scope == 0 else \
        [(b, h) for b in range(B) for h in range(H)]
    ex = 0
    for b, h in units:
        res = plain.check_widths(c[b, h], got[b, h], mean, bmin, bmax)
        assert res["ok"], f"{label}: unit {(b, h)} {res}"
        ex += res["exempt"]
    say(f"plain widths {label}: exempt rows {ex}")

pytestmark = pytest.mark.gpu


def _oracle_bits(gamma, R, G, scope, mean, bmin, bmax):
    B, H, d = gamma.shape
    c = alloc.weights(gamma, alloc.normalized_ranges(R, G))
    if scope == 0:
        return np.stack([alloc.allocate(c[b].reshape(-1), mean, bmin, bmax).reshape(H, d)
                         for b in range(B)])
    return np.stack([[alloc.allocate(c[b, h], mean, bmin, bmax) for h in range(H)]
                     for b in range(B)])


CASES = [
    (2, 3, 64, 64, 0, 4.0, 2, 8),
    (2, 32, 128, 64, 0, 4.0, 2, 8),
    (1, 32, 128, 128, 0, 2.0, 1, 8),
    (3, 4, 128, 128, 1, 3.0, 1, 8),
    (1, 8, 64, 32, 0, 5.5, 1, 16),
]


@pytest.mark.parametrize("case", CASES)
def test_alloc_bits_bit_exact(case):
    B, H, d, G, scope, mean, bmin, bmax = case
    say("alloc case", case)
    rng = np.random.default_rng(7 * d + H)
    gamma = np.exp(rng.normal(0, 3, (B, H, d)))
    R = np.abs(rng.standard_normal((B, H, d))).astype(np.float32)
    R[0, 0, :5] = 0.0                       # zero rows
    gamma[0, 1, :] = 1.0                    # ties inside a head
    R[0, 1, :] = 0.5
    if H > 2:
        R[0, 2, :] = 0.0                    # a whole zero head
    cfg = K.Config(B=B, H=H, d_k=d, d_v=d, group_rows=G, scope=scope, mean_bits=mean,
                   b_min=bmin, b_max=bmax)
    bits = torch.zeros(B * H * d, dtype=torch.uint8, device="cuda")
    ws = K.new_workspace(cfg)
    K.kda_alloc_bits(cfg, dev(gamma), dev(R), bits, ws)
    got = host(bits).reshape(B, H, d).astype(np.int64)
    want = _oracle_bits(gamma, R, G, scope, mean, bmin, bmax)
    assert np.array_equal(got, want), f"{np.sum(got != want)} widths differ"
    _plain_widths(gamma, R, G, scope, mean, bmin, bmax, got, str(case))


def test_alloc_all_zero_weights_fill_in_row_order():
    B, H, d = 1, 2, 64
    cfg = K.Config(B=B, H=H, d_k=d, d_v=d, group_rows=64, scope=0, mean_bits=2.3, b_min=2, b_max=8)
    bits = torch.zeros(B * H * d, dtype=torch.uint8, device="cuda")
    K.kda_alloc_bits(cfg, dev(np.zeros((B, H, d))), dev(np.zeros((B, H, d), np.float32)), bits,
                     K.new_workspace(cfg))
    want = alloc.allocate(np.zeros(H * d), 2.3, 2, 8)
    assert np.array_equal(host(bits).astype(np.int64), want)


@pytest.mark.parametrize("C", [1, 4])
def test_window_weights_match_oracle(C):
    w = W.sized(W.WORKLOADS["tiny"], B=2, H=3)
    x = W.tokens(w, 0, 96)
    cfg = K.Config(B=2, H=3, d_k=64, d_v=64)
    g = torch.zeros(2 * 3 * 64, dtype=torch.float64, device="cuda")
    K.kda_weights(cfg, 96, C, dev(x["q"]), dev(x["s"]), dev(x["beta"]), dev(x["k"]), g)
    # oracle takes [W, ..., dk] time-major
    want = stats.window_gamma(np.moveaxis(x["q"], 1, 0), np.moveaxis(x["s"], 1, 0),
                              np.moveaxis(x["k"], 1, 0), np.moveaxis(x["beta"], 1, 0), C)
    np.testing.assert_allclose(host(g).reshape(2, 3, 64), want, rtol=1e-12)


def _exact_oracle(x, b, h, C, per_head):
    """Oracle exact-Gramian weights of head (b, h): matrices F_t from the
    token's k, s, beta (eq. rule, KDA erase) and the backward recursion."""
    q = x["q"][b, :, h].astype(np.float64)
    ks = x["k"][b, :, h]
    Wn = q.shape[0]
    Fs = np.stack([stats.transition(ks[t], x["s"][b, t, h, 0] if per_head else x["s"][b, t, h],
                                    float(x["beta"][b, t, h])) for t in range(Wn)])
    return stats.exact_window_gamma(q, Fs, C)


@pytest.mark.parametrize("d,C,per_head", [(64, 1, False), (64, 4, True), (128, 1, False),
                                          (128, 3, False)])
def test_exact_weights_match_oracle(d, C, per_head):
    w = W.sized(W.WORKLOADS["gdn2" if per_head else "tiny"], B=2, H=2, dk=d, dv=d)
    Wn = 40
    x = W.tokens(w, 0, Wn)
    cfg = K.Config(B=2, H=2, d_k=d, d_v=d, group_rows=d, decay_per_head=int(per_head))
    g = torch.zeros(2 * 2 * d, dtype=torch.float64, device="cuda")
    s_arg = x["s"][..., 0] if per_head else x["s"]
    K.kda_weights_exact(cfg, Wn, C, dev(x["q"]), dev(s_arg), dev(x["beta"]), dev(x["k"]), g)
    got = host(g).reshape(2, 2, d)
    want = np.stack([[_exact_oracle(x, b, h, C, per_head) for h in range(2)] for b in range(2)])
    err = float(np.max(np.abs(got - want) / np.abs(want)))
    say(f"exact weights d={d} C={C} per_head={per_head}: max rel err {err:.2e}")
    np.testing.assert_allclose(got, want, rtol=1e-9)


def _weights_case(kind, rng, B, H, d):
    gamma = np.exp(rng.normal(0, 3, (B, H, d)))
    R = np.abs(rng.standard_normal((B, H, d))).astype(np.float32)
    if kind == "all_equal":                  # one bucket, identical keys everywhere
        gamma[:] = 0.37
        R[:] = 1.0
    elif kind == "few_values":               # many exact ties between rows
        gamma = np.choose(rng.integers(0, 3, (B, H, d)), [0.5, 1.0, 2.0]).astype(np.float64)
        R[:] = np.choose(rng.integers(0, 2, (B, H, d)), [1.0, 2.0]).astype(np.float32)
    elif kind == "powers_of_two":            # fraction bits all zero
        gamma = np.exp2(rng.integers(-20, 20, (B, H, d))).astype(np.float64)
        R[:] = 1.0
    elif kind == "wide_range":
        gamma = np.exp(rng.uniform(-600, 600, (B, H, d)))
    elif kind == "near_ties":                # keys differing in the last fraction bits
        base = 1.2345678
        gamma = base * (1 + rng.integers(0, 8, (B, H, d)) * 2.0 ** -50)
        R[:] = 1.0
    return gamma, R


@pytest.mark.parametrize("kind", ["all_equal", "few_values", "powers_of_two", "wide_range",
                                  "near_ties"])
@pytest.mark.parametrize("mean", [2.5, 4.0, 6.25])
def test_alloc_ties_and_ranges(kind, mean):
    B, H, d = 2, 32, 128
    rng = np.random.default_rng(hash((kind, mean)) % 2 ** 32)
    gamma, R = _weights_case(kind, rng, B, H, d)
    say("alloc ties", kind, mean)
    cfg = K.Config(B=B, H=H, d_k=d, d_v=d, group_rows=64, scope=0, mean_bits=mean, b_min=2, b_max=8)
    bits = torch.zeros(B * H * d, dtype=torch.uint8, device="cuda")
    K.kda_alloc_bits(cfg, dev(gamma), dev(R), bits, K.new_workspace(cfg))
    got = host(bits).reshape(B, H, d).astype(np.int64)
    want = _oracle_bits(gamma, R, 64, 0, mean, 2, 8)
    assert np.array_equal(got, want), f"{kind}: {np.sum(got != want)} widths differ"
    _plain_widths(gamma, R, 64, 0, mean, 2, 8, got, f"{kind} {mean}")
