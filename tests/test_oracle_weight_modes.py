"""Pins for the allocation-key variants the paper ablates (Sec. 5, Table ablate
and Effect of range normalization for decay-only allocation; Related work for
DAMP's persistence w^(1) = 1/(1 - a^2); Choice of persistence factor for
h^(C) = 1/(1 - exp(-2 C s)))."""
import numpy as np
import pytest

import workloads as W
from oracle import alloc, stats, step


def test_without_erasure_the_weight_is_persistence_times_decay():
    """Related work: without erasure eq. weight is DAMP's uncapped persistence
    times exp(-2 s): 1/expm1(2 s) = exp(-2 s) / (1 - exp(-2 s))."""
    s = np.exp(np.linspace(np.log(1e-6), np.log(5.0), 200))
    g = stats.mode_gamma(s, np.zeros_like(s), "ema")
    w1 = stats.mode_gamma(s, np.zeros_like(s), "persist")
    assert np.allclose(g, w1 * np.exp(-2 * s), rtol=1e-13, atol=0)
    assert np.array_equal(stats.mode_gamma(s, 0.3 + 0 * s, "no_erase_rate"), g)


def test_write_back_factor():
    s = np.exp(np.linspace(np.log(1e-5), np.log(2.0), 50))
    w1 = stats.mode_gamma(s, 0 * s, "persist")
    assert np.allclose(stats.mode_gamma(s, 0 * s, "writeback", C=1), w1, rtol=1e-15)
    h64 = stats.mode_gamma(s, 0 * s, "writeback", C=64)
    assert np.all(h64 <= w1 * (1 + 1e-15)) and np.all(h64 >= 1.0)
    small = s * 64 < 1e-3
    assert np.allclose(h64[small], 1 / (2 * 64 * s[small]), rtol=2e-3)   # slow rows
    assert np.allclose(h64[s * 64 > 20], 1.0, rtol=1e-15)               # fast rows


def _state(erase=True):
    w = W.sized(W.WORKLOADS["tiny"], B=1, H=2)
    oc = step.Cfg(dk=64, dv=64, G=64, mean_bits=3.5, b_min=2, b_max=8, erase=erase)
    xs = W.tokens(w, 0, 24)
    st, S = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    m, e = step.ema_start(st)
    return oc, S.astype(np.float32), m, e, st["ntok"]


def test_uniform_mode_gives_uniform_widths():
    oc, S, m, e, nt = _state()
    oc.weight = "uniform"
    st, _ = step.write_back(S, m, e, nt, oc)
    wd = st["widths"].reshape(-1)
    # 3.5 bits over 128 rows: 64 slots above 3 bits go to the lowest rows
    assert np.array_equal(wd, np.r_[np.full(64, 4), np.full(64, 3)])


def test_range_alone_ignores_decay_and_follows_raw_ranges():
    oc, S, m, e, nt = _state()
    oc.weight = "range"
    a, _ = step.write_back(S, m, e, nt, oc)
    b, _ = step.write_back(S, m * 0.5, e * 3.0, nt, oc)       # other decay statistics
    assert np.array_equal(a["widths"], b["widths"])
    S2 = S.copy()
    S2[0, 1] *= 8.0                                            # head 1 raw ranges x 8
    c, _ = step.write_back(S2, m, e, nt, oc)
    assert c["widths"][0, 1].sum() > a["widths"][0, 1].sum()
    oc.weight = "rel_range"
    d, _ = step.write_back(S, m, e, nt, oc)
    f, _ = step.write_back(S2, m, e, nt, oc)                   # normalised: no change
    assert np.array_equal(d["widths"], f["widths"])


def test_no_erase_rate_mode_equals_ema_without_erasure():
    oc, S, m, e, nt = _state(erase=False)
    ema, _ = step.write_back(S, m, e, nt, oc)
    oc.weight = "no_erase_rate"
    ner, _ = step.write_back(S, m, e + 0.2, nt, oc)            # r ignored
    assert np.array_equal(ema["widths"], ner["widths"])


@pytest.mark.parametrize("mode", stats.WEIGHT_MODES)
def test_every_mode_meets_the_budget(mode):
    oc, S, m, e, nt = _state()
    oc.weight = mode
    st, _ = step.write_back(S, m, e, nt, oc, C=16)
    assert int(st["widths"].sum()) == alloc.budget(3.5, 128)


def test_decay_only_ignores_ranges_and_equals_ema_at_equal_ranges():
    """Decay-only keys are Gamma^ itself: widths do not move when the state's
    rows are rescaled, and they equal the paper's key when every row of a
    group has the same range (R~ = 1)."""
    oc, S, m, e, nt = _state()
    oc.weight = "decay"
    a, _ = step.write_back(S, m, e, nt, oc)
    rng = np.random.default_rng(5)
    S2 = (S * rng.uniform(0.1, 10.0, S.shape[:-1] + (1,))).astype(np.float32)
    b, _ = step.write_back(S2, m, e, nt, oc)
    assert np.array_equal(a["widths"], b["widths"])
    # rows of equal range: scale every row to range 1, then R~ = 1 exactly
    R = np.max(np.abs(S), axis=-1, keepdims=True)
    S3 = (S / np.where(R > 0, R, 1)).astype(np.float32)
    S3[..., 0] = np.where(np.max(np.abs(S3), axis=-1) < 1, 1.0, S3[..., 0])
    assert np.all(np.max(np.abs(S3), axis=-1) == 1.0)
    c, _ = step.write_back(S3, m, e, nt, oc)
    oc.weight = "ema"
    d, _ = step.write_back(S3, m, e, nt, oc)
    assert np.array_equal(c["widths"], d["widths"])
    assert not np.array_equal(a["widths"], step.write_back(S, m, e, nt, oc)[0]["widths"])
