"""Parity at the benchmark's full size and launch configuration.

The decode workload (B=64 sequences, H=32 heads, d=128, 4-bit mean, layer
budget) runs as one kda_step launch exactly as bench.py times it.  Sampled
sequences start from oracle-made records (the others from the zero state:
sequences are independent) and are compared one by one with the oracle.
The long-context shape (Student-t values, 3-bit mean, window Gramian weights
recomputed by kda_weights) is checked the same way at a reduced batch.  The
prefill workload (B=4, H=32, T=8192) runs as one kda_prefill call in both
forms, with sampled write-back intervals checked against the oracle.  The
decode step is also run from the benchmark's own prior records (512 decode
tokens from the zero state on the GPU, as bench.py builds them).  Every
write-back checked here is also checked against the plain definitions of
widths, clip factors, scales and codes (oracle/plain.py) on the GPU's own
float32 state.
"""
import dataclasses

import numpy as np
import pytest
import torch

import paper_2609_30950_amd as K
import workloads as W
from oracle import recurrence, record, stats, step
from tests._gpu import (bytes_to_state, decode_gamma, decode_state_gpu, dev, host, plain_check,
                        plain_check_heads, say, state32_step_gpu, state_to_bytes, ws_state32)

pytestmark = pytest.mark.gpu

SAMPLED = (0, 37, 63)


def _compare(stg, st, label):
    same_w = stg["widths"] == st["widths"]
    dc = int(np.sum((stg["codes"] != st["codes"]) & same_w[..., None])) + \
        int(np.sum(~same_w)) * stg["codes"].shape[-1]
    say(f"{label}: widths {int(np.sum(~same_w))} codes {dc} of {stg['codes'].size}")
    assert np.array_equal(stg["ntok"], st["ntok"])
    assert np.array_equal(stg["widths"], st["widths"])
    assert np.array_equal(stg["scale"].view(np.uint16), st["scale"].view(np.uint16))
    assert np.array_equal(stg["r16"].view(np.uint16), st["r16"].view(np.uint16))
    assert np.sum(stg["z"] != st["z"]) <= 2
    assert dc / stg["codes"].size <= 1e-5


def test_decode_full_batch_sampled_sequences():
    w = W.WORKLOADS["decode"]
    kc = K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.G, mean_bits=w.mean_bits,
                  b_min=w.b_min, b_max=w.b_max)
    oc = step.Cfg(dk=w.dk, dv=w.dv, G=w.G, mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max)
    base = W.base_rates(w)
    sel = list(SAMPLED)
    warm = [W.token(w, t, base=base) for t in range(24)]
    xs = {n: np.stack([x[n][sel] for x in warm], axis=1) for n in warm[0]}
    st0, _ = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    slot = record.record_bytes(w.dk, w.dv, w.b_max)
    recs = np.zeros((w.B, w.H * slot), np.uint8)
    recs[sel] = state_to_bytes(st0, w.dk, w.dv, w.b_max).reshape(len(sel), -1)
    recs_d = dev(recs.reshape(-1))
    x = W.token(w, 24, base=base)
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    ws = K.new_workspace(kc)
    before = recs_d.clone()
    K.kda_step(kc, recs_d, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(x["s"]), dev(x["beta"]), o,
               ws)
    got = host(recs_d).reshape(w.B, w.H * slot)[sel].reshape(-1)
    og = host(o).reshape(w.B, w.H, w.dv)[sel]
    xo = {n: a[sel] for n, a in x.items()}
    X = step.dequantize(st0)
    st1, o_or, _ = step.mirror_decode_step(st0, xo["q"], xo["k"], xo["v"], xo["s"], xo["beta"], oc)
    stg = bytes_to_state(got, len(sel), w.H, w.dk, w.dv, w.b_max)
    plain_check(decode_state_gpu(kc, before, ws, sel), decode_gamma(st0, xo, oc.span), stg,
                G=w.G, scope=0, mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max,
                label="decode B=64 sampled")
    _compare(stg, st1, "decode B=64 sampled")
    ot = step.truth_outputs(X, xo["q"], xo["k"], xo["v"], xo["s"], xo["beta"])
    err = float(np.max(np.abs(og - ot)) / np.max(np.abs(ot)))
    say(f"decode B=64 sampled: o normwise rel err vs float64 {err:.2e}")
    assert err <= 1e-3
    assert np.max(np.abs(og - o_or)) <= 1e-6 * np.max(np.abs(o_or))


def test_long_context_window_weights_student_t():
    w = W.sized(W.WORKLOADS["long"], B=2, H=4, window=64)
    kc = K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.G, mean_bits=w.mean_bits,
                  b_min=w.b_min, b_max=w.b_max)
    oc = step.Cfg(dk=w.dk, dv=w.dv, G=w.G, mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max)
    xs = W.tokens(w, 0, w.window)
    st0, _ = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    # Gramian weights from the query window (C = 1), on the GPU and in the oracle
    g = torch.zeros(w.B * w.H * w.dk, dtype=torch.float64, device="cuda")
    K.kda_weights(kc, w.window, 1, dev(xs["q"]), dev(xs["s"]), dev(xs["beta"]), dev(xs["k"]), g)
    gam = stats.window_gamma(np.moveaxis(xs["q"], 1, 0), np.moveaxis(xs["s"], 1, 0),
                             np.moveaxis(xs["k"], 1, 0), np.moveaxis(xs["beta"], 1, 0), 1)
    np.testing.assert_allclose(host(g).reshape(gam.shape), gam, rtol=1e-12)
    recs = dev(state_to_bytes(st0, w.dk, w.dv, w.b_max))
    ws = K.new_workspace(kc)
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    st = st0
    base = W.base_rates(w)
    for t in range(w.window, w.window + 6):
        x = W.token(w, t, base=base)
        before = recs.clone()
        K.kda_step(kc, recs, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(x["s"]), dev(x["beta"]), o,
                   ws, gamma=dev(gam))
        stg = bytes_to_state(host(recs), w.B, w.H, w.dk, w.dv, w.b_max)
        plain_check(decode_state_gpu(kc, before, ws), gam, stg, G=w.G, scope=0,
                    mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max, label=f"long t={t}")
        st, o_or, _ = step.mirror_decode_step(st, x["q"], x["k"], x["v"], x["s"], x["beta"], oc,
                                              gamma=gam)
        _compare(stg, st, f"long t={t}")


def _prefill_call(kc, w, xs, T):
    """kda_prefill of tokens [0, T) from zero records, as bench.py calls it."""
    recs = K.new_records(kc)
    ws = K.new_workspace(kc)
    o = torch.zeros(w.B * T * w.H * w.dv, dtype=torch.float32, device="cuda")
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a[:, :T])).to(torch.bfloat16).cuda()
    K.kda_prefill(kc, T, w.C, recs, bf(xs["q"]), bf(xs["k"]), bf(xs["v"]),
                  dev(np.ascontiguousarray(xs["s"][:, :T])), dev(np.ascontiguousarray(xs["beta"][:, :T])),
                  o, ws)
    return recs, o, ws


@pytest.mark.parametrize("chunked", [1, 0])
def test_prefill_full_size_sampled_intervals(chunked):
    """The prefill workload (B=4, H=32, d=128, T=8192, write-back every 64
    tokens, bf16 inputs, 4-bit mean) in the launch configuration bench.py
    times: one call over all tokens from the empty state.  Calls that stop
    at an interval boundary must produce the same outputs for the tokens they
    share, bit for bit (the chunked form's groups of chunks change with T);
    the interval after such a boundary (the 64th and the last) is then checked
    against the oracle from the GPU's own record at the boundary: outputs and
    state against the float64 recurrence within 1e-3 (normwise, both forms), and the
    write-back of the GPU's float32 state bit for bit against the oracle's
    allocation and quantiser."""
    w = W.WORKLOADS["prefill"]
    kc = K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.G, mean_bits=w.mean_bits,
                  b_min=w.b_min, b_max=w.b_max, chunked=chunked)
    oc = step.Cfg(dk=w.dk, dv=w.dv, G=w.G, mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max)
    tol = 1e-3
    xs = W.tokens(w, 0, w.T)
    say(f"prefill full size chunked={chunked}: inputs ready")
    _, o_full, _ = _prefill_call(kc, w, xs, w.T)
    o_full = host(o_full).reshape(w.B, w.T, w.H, w.dv)
    for t_end in (64 * 64, w.T):
        t0 = t_end - w.C
        r0, o0, _ = _prefill_call(kc, w, xs, t0)
        r1, o1, ws1 = _prefill_call(kc, w, xs, t_end)
        o1 = host(o1).reshape(w.B, t_end, w.H, w.dv)
        assert np.array_equal(o1.view(np.uint32), o_full[:, :t_end].view(np.uint32))
        assert np.array_equal(host(o0).reshape(w.B, t0, w.H, w.dv).view(np.uint32),
                              o_full[:, :t0].view(np.uint32))
        st0 = bytes_to_state(host(r0), w.B, w.H, w.dk, w.dv, w.b_max)
        X = step.dequantize(st0).astype(np.float64)
        m, e = step.ema_start(st0)
        ot = np.zeros((w.B, w.C, w.H, w.dv))
        for j, t in enumerate(range(t0, t_end)):
            x = {n: a[:, t] for n, a in xs.items()}
            X, ot[:, j] = recurrence.truth_step_rowform(X, x["q"], x["k"], x["v"], x["s"], x["beta"])
            m, e = stats.ema_update(m, e, x["s"], x["k"], np.asarray(x["beta"])[..., None], oc.span)
        og = o1[:, t0:t_end]
        Sg = ws_state32(ws1, w)
        es = np.max(np.abs(Sg - X), axis=(2, 3)) / np.max(np.abs(X), axis=(2, 3))
        eo = np.max(np.abs(og - ot), axis=(1, 3)) / np.max(np.abs(ot), axis=(1, 3))
        say(f"interval [{t0}, {t_end}): state err {es.max():.2e}, output err {eo.max():.2e} "
            f"(bound {tol:.1e})")
        assert np.all(np.isfinite(Sg)) and es.max() <= tol and eo.max() <= tol
        exp, _ = step.write_back(Sg, m, e, st0["ntok"] + w.C, oc)
        got = bytes_to_state(host(r1), w.B, w.H, w.dk, w.dv, w.b_max)
        s_hat, r = stats.ema_rates(m, e)
        plain_check(Sg, stats.mode_gamma(s_hat, r), got, G=w.G, scope=0, mean_bits=w.mean_bits,
                    b_min=w.b_min, b_max=w.b_max, label=f"prefill interval [{t0}, {t_end})")
        for f in ("ntok", "widths", "z", "r16", "codes"):
            assert np.array_equal(got[f], exp[f]), f
        assert np.array_equal(got["scale"].view(np.uint16), exp["scale"].view(np.uint16))


@pytest.mark.parametrize("name,heads", [("gdn2", 0), ("gdn6", 0), ("gdn2", 1), ("gdn6", 1)])
def test_gdn_decode_full_batch_sampled_sequences(name, heads):
    """The Gated-DeltaNet-shaped decode workloads (B=16, H=16, d=256, one
    decay rate per head and token, mean 2 or 6 bits) as one kda_step launch,
    with per-row widths or (heads = 1) one width per head and block scales:
    sequences 0, 7 and 15 start from oracle-made records, the others from the
    zero state, and the sampled ones are compared with the oracle."""
    w = W.WORKLOADS[name]
    if heads:
        w = W.sized(w, b_min=2, G=w.dk)
    kc = K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.G, mean_bits=w.mean_bits,
                  b_min=w.b_min, b_max=w.b_max, decay_per_head=1, head_units=heads)
    oc = step.Cfg(dk=w.dk, dv=w.dv, G=w.G, mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max,
                  unit="head" if heads else "row")
    sel = [0, 7, 15]
    warm = W.tokens(w, 0, 12)
    xs = {n: a[sel] for n, a in warm.items()}
    st0, _ = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    if heads:
        slot = record.record_bytes_heads(w.dk, w.dv, w.b_max)
        packed = np.concatenate([record.pack_heads(st0["ntok"][b, h], st0["width"][b, h],
                                                   st0["bscale"][b, h], st0["z"][b, h],
                                                   st0["r16"][b, h], st0["codes"][b, h], w.dk,
                                                   w.dv, w.b_max)
                                 for b in range(len(sel)) for h in range(w.H)])
    else:
        slot = record.record_bytes(w.dk, w.dv, w.b_max)
        packed = state_to_bytes(st0, w.dk, w.dv, w.b_max)
    recs = np.zeros((w.B, w.H * slot), np.uint8)
    recs[sel] = packed.reshape(len(sel), -1)
    recs_d = dev(recs.reshape(-1))
    x = W.token(w, 12)
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    ws = K.new_workspace(kc)
    before = recs_d.clone()
    K.kda_step(kc, recs_d, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(x["s"][..., 0]),
               dev(x["beta"]), o, ws)
    got = host(recs_d).reshape(w.B, w.H, slot)[sel]
    og = host(o).reshape(w.B, w.H, w.dv)[sel]
    xo = {n: a[sel] for n, a in x.items()}
    X = step.dequantize(st0)
    st1, o_or, _ = step.mirror_decode_step(st0, xo["q"], xo["k"], xo["v"], xo["s"], xo["beta"], oc)
    label = f"{name} B=16 heads={heads} sampled"
    g_sel = decode_gamma(st0, xo, oc.span)
    if heads:
        stg = {k_: np.stack([np.stack([np.asarray(record.unpack_heads(got[b, h], w.dk, w.dv,
                                                                      w.b_max)[k_])
                                       for h in range(w.H)]) for b in range(len(sel))])
               for k_ in ("width", "bscale", "codes")}
        S_sel = state32_step_gpu(dataclasses.replace(kc, B=len(sel)), X, xo)
        plain_check_heads(S_sel, g_sel, stg, mean_bits=w.mean_bits, b_min=w.b_min,
                          b_max=w.b_max, label=label)
    else:
        plain_check(decode_state_gpu(kc, before, ws, sel), g_sel,
                    bytes_to_state(got.reshape(-1), len(sel), w.H, w.dk, w.dv, w.b_max),
                    G=w.G, scope=0, mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max,
                    label=label)
    if heads:
        for b in range(len(sel)):
            for h in range(w.H):
                f = record.unpack_heads(got[b, h], w.dk, w.dv, w.b_max)
                assert int(f["ntok"]) == int(st1["ntok"][b, h])
                assert int(f["width"]) == int(st1["width"][b, h]), (b, h)
                assert np.array_equal(np.asarray(f["bscale"]).view(np.uint16),
                                      st1["bscale"][b, h].view(np.uint16)), (b, h)
                assert np.array_equal(np.asarray(f["codes"]), st1["codes"][b, h]), (b, h)
                assert np.array_equal(np.asarray(f["r16"]).view(np.uint16),
                                      st1["r16"][b, h].view(np.uint16))
                assert int(np.sum(np.asarray(f["z"]) != st1["z"][b, h])) <= 1
        say(f"{label}: head widths {st1['width'].ravel().tolist()}")
    else:
        _compare(bytes_to_state(got.reshape(-1), len(sel), w.H, w.dk, w.dv, w.b_max), st1, label)
    ot = step.truth_outputs(X, xo["q"], xo["k"], xo["v"], xo["s"], xo["beta"])
    err = float(np.max(np.abs(og - ot)) / np.max(np.abs(ot)))
    say(f"{label}: o normwise rel err vs float64 {err:.2e}")
    assert err <= 1e-3
    assert np.max(np.abs(og - o_or)) <= 1e-6 * np.max(np.abs(o_or))


def test_long_context_weights_full_size():
    """Window weights of the long-context layer at full size (B=128, H=32,
    d=128, a window of W=1024 tokens, C=1) as bench.py launches them: two
    sequences' inputs tiled to 128 sequences.  The diagonal-erase estimate
    (kda_weights) of every head against the oracle's float64 recursion, and
    the exact Gramian recursion (kda_weights_exact) of sampled heads against
    the oracle's matrix recursion."""
    w = W.WORKLOADS["long"]
    Wn = w.window
    xs = W.tokens(W.sized(w, B=2), 0, Wn)
    rep = w.B // 2
    d = {n: dev(a).repeat((rep,) + (1,) * (a.ndim - 1)).contiguous() for n, a in xs.items()}
    kc = K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.G, mean_bits=w.mean_bits,
                  b_min=w.b_min, b_max=w.b_max)
    g = torch.zeros(w.B * w.H * w.dk, dtype=torch.float64, device="cuda")
    K.kda_weights(kc, Wn, 1, d["q"], d["s"], d["beta"], d["k"], g)
    got = host(g).reshape(w.B, w.H, w.dk)
    want = stats.window_gamma(np.moveaxis(xs["q"], 1, 0), np.moveaxis(xs["s"], 1, 0),
                              np.moveaxis(xs["k"], 1, 0), np.moveaxis(xs["beta"], 1, 0), 1)
    np.testing.assert_allclose(got, np.tile(want, (rep, 1, 1)), rtol=1e-12)
    g.zero_()
    K.kda_weights_exact(kc, Wn, 1, d["q"], d["s"], d["beta"], d["k"], g)
    got = host(g).reshape(w.B, w.H, w.dk)
    worst = 0.0
    for b, h in ((0, 0), (1, 17), (127, 31)):
        q = xs["q"][b % 2, :, h].astype(np.float64)
        Fs = np.stack([stats.transition(xs["k"][b % 2, t, h], xs["s"][b % 2, t, h],
                                        float(xs["beta"][b % 2, t, h])) for t in range(Wn)])
        ref = stats.exact_window_gamma(q, Fs, 1)
        worst = max(worst, float(np.max(np.abs(got[b, h] - ref) / np.abs(ref))))
    say(f"long-context weights B=128 W=1024: exact Gramian max rel err {worst:.2e} (sampled heads)")
    assert worst <= 1e-9


def test_long_context_decode_full_batch_sampled_sequences():
    """One decode step of the long-context workload at full batch (B=128,
    H=32, d=128, mean 3 bits, widths [2, 8], Student-t values, weights given
    by the caller): sequences 0, 64 and 127 start from oracle-made records
    with window weights from their own inputs, the others from the zero
    state with unit weights; the sampled ones are compared with the oracle."""
    w = W.WORKLOADS["long"]
    kc = K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.G, mean_bits=w.mean_bits,
                  b_min=w.b_min, b_max=w.b_max)
    oc = step.Cfg(dk=w.dk, dv=w.dv, G=w.G, mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max)
    sel = [0, 64, 127]
    ws_ = W.sized(w, B=len(sel))
    xs = W.tokens(ws_, 0, 32)
    st0, _ = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    gam_sel = stats.window_gamma(np.moveaxis(xs["q"], 1, 0), np.moveaxis(xs["s"], 1, 0),
                                 np.moveaxis(xs["k"], 1, 0), np.moveaxis(xs["beta"], 1, 0), 1)
    gam = np.ones((w.B, w.H, w.dk))
    gam[sel] = gam_sel
    slot = record.record_bytes(w.dk, w.dv, w.b_max)
    recs = np.zeros((w.B, w.H * slot), np.uint8)
    recs[sel] = state_to_bytes(st0, w.dk, w.dv, w.b_max).reshape(len(sel), -1)
    recs_d = dev(recs.reshape(-1))
    x1 = W.token(ws_, 32)
    x = {n: np.zeros((w.B,) + a.shape[1:], a.dtype) for n, a in x1.items()}
    for n in x:
        x[n][:] = x1[n][:1]          # unsampled sequences: any valid token
        x[n][sel] = x1[n]
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    ws = K.new_workspace(kc)
    before = recs_d.clone()
    K.kda_step(kc, recs_d, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(x["s"]), dev(x["beta"]), o,
               ws, gamma=dev(gam))
    got = host(recs_d).reshape(w.B, w.H * slot)[sel].reshape(-1)
    og = host(o).reshape(w.B, w.H, w.dv)[sel]
    X = step.dequantize(st0)
    st1, o_or, _ = step.mirror_decode_step(st0, x1["q"], x1["k"], x1["v"], x1["s"], x1["beta"], oc,
                                           gamma=gam_sel)
    stg = bytes_to_state(got, len(sel), w.H, w.dk, w.dv, w.b_max)
    plain_check(decode_state_gpu(kc, before, ws, sel), gam_sel, stg, G=w.G, scope=0,
                mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max, label="long B=128 sampled")
    _compare(stg, st1, "long B=128 sampled")
    ot = step.truth_outputs(X, x1["q"], x1["k"], x1["v"], x1["s"], x1["beta"])
    err = float(np.max(np.abs(og - ot)) / np.max(np.abs(ot)))
    say(f"long B=128 sampled: o normwise rel err vs float64 {err:.2e}")
    assert err <= 1e-3
    assert np.max(np.abs(og - o_or)) <= 1e-6 * np.max(np.abs(o_or))


def test_decode_from_bench_prior_records():
    """The decode workload from the records the benchmark times: 512 decode
    tokens from the zero state run by the library (as bench.py builds its
    prior state), then three more steps; for sampled sequences each step is
    compared with the oracle started from the GPU's own records of that step
    (widths, scales and codes bit for bit, rate codes counted in the
    mismatch rate, outputs against float64), and checked against the plain
    definitions."""
    w = W.WORKLOADS["decode"]
    kc = K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.G, mean_bits=w.mean_bits,
                  b_min=w.b_min, b_max=w.b_max)
    oc = step.Cfg(dk=w.dk, dv=w.dv, G=w.G, mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max)
    base = W.base_rates(w)
    recs = K.new_records(kc)
    ws = K.new_workspace(kc)
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    warm = 512
    for t in range(warm):
        x = {n: torch.from_numpy(a).cuda() for n, a in W.token(w, t, base=base).items()}
        K.kda_step(kc, recs, x["q"], x["k"], x["v"], x["s"], x["beta"], o, ws)
    torch.cuda.synchronize()
    say(f"bench prior: {warm} warm-up decode tokens done")
    sel = [0, 21, 42, 63]
    slot = record.record_bytes(w.dk, w.dv, w.b_max)
    bad = tot = 0
    for t in range(warm, warm + 3):
        x = W.token(w, t, base=base)
        xo = {n: a[sel] for n, a in x.items()}
        st0 = bytes_to_state(host(recs).reshape(w.B, w.H * slot)[sel].reshape(-1), len(sel), w.H,
                             w.dk, w.dv, w.b_max)
        before = recs.clone()
        K.kda_step(kc, recs, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(x["s"]), dev(x["beta"]), o,
                   ws)
        stg = bytes_to_state(host(recs).reshape(w.B, w.H * slot)[sel].reshape(-1), len(sel), w.H,
                             w.dk, w.dv, w.b_max)
        plain_check(decode_state_gpu(kc, before, ws, sel), decode_gamma(st0, xo, oc.span), stg,
                    G=w.G, scope=0, mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max,
                    label=f"bench prior t={t}")
        X = step.dequantize(st0)
        st1, o_or, _ = step.mirror_decode_step(st0, xo["q"], xo["k"], xo["v"], xo["s"],
                                               xo["beta"], oc)
        for j, b in enumerate(sel):
            one = {f: a[j:j + 1] for f, a in stg.items()}
            ref = {f: a[j:j + 1] for f, a in st1.items()}
            assert np.array_equal(one["ntok"], ref["ntok"])
            assert np.array_equal(one["widths"], ref["widths"]), (t, b)
            assert np.array_equal(one["scale"].view(np.uint16), ref["scale"].view(np.uint16)), (t, b)
            assert np.array_equal(one["r16"].view(np.uint16), ref["r16"].view(np.uint16)), (t, b)
            dc = int(np.sum(one["codes"] != ref["codes"]))
            dz = int(np.sum(one["z"] != ref["z"]))
            bad += dc + dz
            tot += one["codes"].size + one["z"].size
        hist = np.bincount(stg["widths"].ravel(), minlength=w.b_max + 1)[w.b_min:]
        og = host(o).reshape(w.B, w.H, w.dv)[sel]
        ot = step.truth_outputs(X, xo["q"], xo["k"], xo["v"], xo["s"], xo["beta"])
        err = float(np.max(np.abs(og - ot)) / np.max(np.abs(ot)))
        say(f"bench prior t={t}: widths {w.b_min}..{w.b_max}: {hist.tolist()}, "
            f"o rel err vs float64 {err:.2e}")
        assert err <= 1e-3
        assert np.max(np.abs(og - o_or)) <= 1e-6 * np.max(np.abs(o_or))
    say(f"bench prior: code and rate-code mismatch rate {bad / tot:.2e} ({bad} of {tot})")
    assert bad / tot <= 1e-5
