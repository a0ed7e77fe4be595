"""Pins for the write-back protocol drivers (Sec. 2-3, Sec. 5 Protocol)."""
import numpy as np
import pytest

import workloads as W
from oracle import alloc, record, stats, step


def _cfg(w):
    return step.Cfg(dk=w.dk, dv=w.dv, G=w.G, mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max)


def test_decode_steps_budget_and_outputs():
    w = W.WORKLOADS["tiny"]
    cfg = _cfg(w)
    st = step.zero_state(w.B, w.H, cfg)
    base = W.base_rates(w)
    for t in range(6):
        x = W.token(w, t, base=base)
        X = step.dequantize(st)
        new, o, d = step.mirror_decode_step(st, x["q"], x["k"], x["v"], x["s"], x["beta"], cfg)
        # layer budget: sum of widths over all heads of a sequence
        assert new["widths"][0].sum() == alloc.budget(cfg.mean_bits, w.H * w.dk)
        assert new["widths"].min() >= cfg.b_min and new["widths"].max() <= cfg.b_max
        # outputs precede quantisation: o comes from the float32 state
        ot = step.truth_outputs(X, x["q"], x["k"], x["v"], x["s"], x["beta"])
        err = np.max(np.abs(o - ot)) / np.max(np.abs(ot))
        assert err < 1e-5
        assert np.all(new["ntok"] == t + 1)
        st = new


def test_prefill_C1_equals_decode_steps():
    w = W.sized(W.WORKLOADS["tiny"], T=5)
    cfg = _cfg(w)
    xs = W.tokens(w, 0, 5)
    st = step.zero_state(w.B, w.H, cfg)
    outs = []
    for t in range(5):
        st, o, _ = step.mirror_decode_step(st, xs["q"][:, t], xs["k"][:, t], xs["v"][:, t],
                                           xs["s"][:, t], xs["beta"][:, t], cfg)
        outs.append(o)
    st2, o2, _ = step.mirror_prefill(step.zero_state(w.B, w.H, cfg), xs["q"], xs["k"], xs["v"],
                                     xs["s"], xs["beta"], 1, cfg)
    assert np.array_equal(np.stack(outs, 1), o2)
    for key in st:
        assert np.array_equal(st[key], st2[key]), key


def test_prefill_chunked_writeback_count_and_ema_chunk_invariance():
    w = W.sized(W.WORKLOADS["tiny"], T=11)
    cfg = _cfg(w)
    xs = W.tokens(w, 0, 11)
    st, o, diags = step.mirror_prefill(step.zero_state(w.B, w.H, cfg), xs["q"], xs["k"], xs["v"],
                                       xs["s"], xs["beta"], 4, cfg)
    assert len(diags) == 3                       # after tokens 4, 8 and the last (11)
    assert np.all(st["ntok"] == 11)
    # without write-backs in between, the EMA after 4 tokens equals the
    # token-sequential EMA (chunk-aware: independent of C)
    m, e = stats.ema_init(xs["s"][:, 0], xs["k"][:, 0], xs["beta"][:, 0][..., None])
    for t in range(1, 4):
        m, e = stats.ema_update(m, e, xs["s"][:, t], xs["k"][:, t], xs["beta"][:, t][..., None], 64)
    sh, r = stats.ema_rates(m, e)
    np.testing.assert_array_equal(diags[0]["s_hat"], sh)


def test_record_bytes_roundtrip_of_step_state():
    w = W.WORKLOADS["tiny"]
    cfg = _cfg(w)
    st = step.zero_state(w.B, w.H, cfg)
    x = W.token(w, 0)
    st, _, _ = step.mirror_decode_step(st, x["q"], x["k"], x["v"], x["s"], x["beta"], cfg)
    for h in range(w.H):
        buf = record.pack(st["ntok"][0, h], st["widths"][0, h], st["scale"][0, h], st["z"][0, h],
                          st["r16"][0, h], st["codes"][0, h], w.dk, w.dv, w.b_max)
        f = record.unpack(buf, w.dk, w.dv, w.b_max)
        assert np.array_equal(f["codes"], st["codes"][0, h])


def test_head_scope_budget_per_head():
    w = W.WORKLOADS["tiny"]
    cfg = step.Cfg(dk=w.dk, dv=w.dv, G=w.G, scope="head", mean_bits=3.0, b_min=1, b_max=8)
    st = step.zero_state(w.B, w.H, cfg)
    x = W.token(w, 0)
    st, _, _ = step.mirror_decode_step(st, x["q"], x["k"], x["v"], x["s"], x["beta"], cfg)
    assert np.all(st["widths"].sum(-1) == 3 * w.dk)


def test_decay_weighting_gives_slow_rows_more_bits():
    # equal ranges, slow vs fast decay: slower rows (larger Gamma) get wider codes
    cfg = step.Cfg(dk=64, dv=64, G=64, scope="head", mean_bits=4.0, b_min=2, b_max=8)
    S = np.ones((1, 1, 64, 64), np.float32)
    s = np.where(np.arange(64) < 32, 1e-3, 0.5)[None, None].astype(np.float32)
    m, e = stats.ema_init(s, np.zeros((1, 1, 64), np.float32), np.zeros((1, 1, 1), np.float32))
    st, _ = step.write_back(S, m, e, np.ones((1, 1), np.int64), cfg)
    assert st["widths"][0, 0, :32].min() > st["widths"][0, 0, 32:].max()


def test_no_erasure_stores_zero_erase_rates_and_spans_heads():
    # without erasure the erase statistic is 0, so the stored rate r is 0; the
    # normalisation groups may span heads (G = 2 d_k)
    w = W.sized(W.WORKLOADS["tiny"], B=1, H=4, dk=32, dv=32)
    cfg = step.Cfg(dk=32, dv=32, G=64, mean_bits=3.0, b_min=1, b_max=8, erase=False)
    xs = W.tokens(w, 0, 6)
    st, S = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], cfg)
    assert np.all(st["r16"] == 0)
    R = np.max(np.abs(S.astype(np.float32)), axis=-1).astype(np.float32)
    Rt = alloc.normalized_ranges(R.reshape(1, 4 * 32), 64)
    assert np.allclose(np.sqrt(np.mean(Rt.reshape(2, 64) ** 2, axis=1)), 1.0)
    assert int(st["widths"].sum()) == alloc.budget(3.0, 4 * 32)
