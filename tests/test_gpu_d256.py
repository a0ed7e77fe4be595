"""GPU parity at d_k = d_v = 256 (the Gated-DeltaNet head shape: per-head
decay, one-bit floor, widths up to 8) against the oracle.

* codec: pack/unpack bit exact on given states and widths;
* 32-bit mode: float32 contract of the recurrence;
* oracle-forced decode steps on 16 heads x 256 rows (one layer budget of
  4096 rows, the largest the library accepts) at mean 2 and 6 bits, and with
  the per-head budget;
* prefill with write-back every C tokens and a ragged last chunk.
"""
import numpy as np
import pytest
import torch

import paper_2609_30950_amd as K
import workloads as W
from oracle import quant, record, recurrence, stats, step
from tests._gpu import (bytes_to_state, decode_gamma, decode_state_gpu, dev, host,
                        meaningful_equal, plain_check, prefill_gamma, say, state_to_bytes,
                        ws_state32)

pytestmark = pytest.mark.gpu

D = 256


def _cfgs(w, scope=0, state32=0):
    kc = K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.G, scope=scope,
                  mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max,
                  decay_per_head=int(w.decay == "head"), state32=state32)
    oc = step.Cfg(dk=w.dk, dv=w.dv, G=w.G, scope="sequence" if scope == 0 else "head",
                  mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max)
    return kc, oc


def _s_arg(s, w):
    return s if w.decay != "head" else s[..., 0]


def _codes_off(stg, st):
    same_w = stg["widths"] == st["widths"]
    return int(np.sum((stg["codes"] != st["codes"]) & same_w[..., None])) + \
        int(np.sum(~same_w)) * stg["codes"].shape[-1]


@pytest.mark.parametrize("dist", ["normal", "mixed"])
def test_codec_d256_bit_exact(dist):
    B, H, bmin, bmax = 1, 3, 1, 8
    rng = np.random.default_rng(256)
    S = rng.standard_normal((B, H, D, D))
    if dist == "mixed":
        S = S * np.exp(rng.uniform(-30, 12, (B, H, D, 1)))
        S[0, 0, 7] = 0.0
        S[0, 1, 200] = 1e7
    S = S.astype(np.float32)
    bits = rng.integers(bmin, bmax + 1, (B, H, D)).astype(np.uint8)
    s_hat = np.exp(rng.uniform(np.log(1e-6), np.log(30), (B, H, D)))
    r = rng.uniform(0, 0.5, (B, H, D))
    cfg = K.Config(B=B, H=H, d_k=D, d_v=D, group_rows=D, b_min=bmin, b_max=bmax, mean_bits=4.0)
    recs = K.new_records(cfg)
    K.kda_pack_state(cfg, dev(S), dev(bits), dev(s_hat), dev(r), 5, recs)
    want = []
    for b in range(B):
        for h in range(H):
            codes, scale, _ = quant.quantize_rows(S[b, h], bits[b, h])
            want.append(record.pack(5, bits[b, h], scale, stats.logq_encode(s_hat[b, h]),
                                    stats.r_encode(r[b, h]), codes, D, D, bmax))
    want = np.concatenate(want)
    bad = meaningful_equal(host(recs), want, B, H, D, D, bmax)
    say(f"pack d=256 {dist}: {len(bad)} of {B * H} records differ")
    assert not bad
    Sg = torch.zeros(B * H * D * D, dtype=torch.float32, device="cuda")
    bg = torch.zeros(B * H * D, dtype=torch.uint8, device="cuda")
    K.kda_unpack_state(cfg, dev(want), Sg, bg, None, None)
    st = bytes_to_state(want, B, H, D, D, bmax)
    X = quant.dequantize_rows(st["codes"].reshape(-1, D), st["scale"].reshape(-1),
                              st["widths"].reshape(-1))
    assert np.array_equal(host(bg), st["widths"].reshape(-1))
    assert np.array_equal(host(Sg).view(np.uint32), X.astype(np.float32).reshape(-1).view(np.uint32))


def test_state32_step_d256():
    w = W.sized(W.WORKLOADS["gdn2"], B=1, H=2)
    kc, _ = _cfgs(w, state32=1)
    rng = np.random.default_rng(7)
    S = rng.standard_normal((w.B, w.H, D, D)).astype(np.float32)
    recs = dev(S.reshape(-1).view(np.uint8))
    o = torch.zeros(w.B * w.H * D, dtype=torch.float32, device="cuda")
    base = W.base_rates(w)
    X = S
    for t in range(4):
        x = W.token(w, t, base=base)
        K.kda_step(kc, recs, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(_s_arg(x["s"], w)),
                   dev(x["beta"]), o, None)
        X, o_or = recurrence.mirror_step(X, x["q"], x["k"], x["v"], x["s"], x["beta"])
        Sg = host(recs).view(np.float32).reshape(X.shape)
        nbad = int(np.sum(Sg.view(np.uint32) != X.view(np.uint32)))
        assert nbad <= X.size // 10000, f"token {t}: {nbad} state values differ"
        og = host(o).reshape(o_or.shape)
        assert np.max(np.abs(og - o_or)) <= 1e-6 * np.max(np.abs(o_or))
        X = Sg


@pytest.mark.parametrize("name,scope", [("gdn2", 0), ("gdn6", 0), ("gdn2", 1)])
def test_forced_decode_steps_d256(name, scope):
    w = W.sized(W.WORKLOADS[name], B=1)
    kc, oc = _cfgs(w, scope=scope)
    xs = W.tokens(w, 0, 6)
    st, _ = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    ws = K.new_workspace(kc)
    o = torch.zeros(w.B * w.H * D, dtype=torch.float32, device="cuda")
    base = W.base_rates(w)
    bad = tot = 0
    for t in range(6, 8):
        x = W.token(w, t, base=base)
        recs = dev(state_to_bytes(st, D, D, w.b_max))
        before = recs.clone()
        K.kda_step(kc, recs, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(_s_arg(x["s"], w)),
                   dev(x["beta"]), o, ws)
        stg = bytes_to_state(host(recs), w.B, w.H, D, D, w.b_max)
        plain_check(decode_state_gpu(kc, before, ws), decode_gamma(st, x, oc.span), stg, G=w.G,
                    scope=scope, mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max,
                    label=f"{name} scope={scope} t={t}")
        X = step.dequantize(st)
        st, o_or, _ = step.mirror_decode_step(st, x["q"], x["k"], x["v"], x["s"], x["beta"], oc)
        dc = _codes_off(stg, st)
        ds = int(np.sum(stg["scale"].view(np.uint16) != st["scale"].view(np.uint16)))
        say(f"{name} scope={scope} t={t}: widths {int(np.sum(stg['widths'] != st['widths']))} "
            f"scales {ds} codes {dc} of {stg['codes'].size}")
        assert np.array_equal(stg["ntok"], st["ntok"])
        assert np.array_equal(stg["widths"], st["widths"])
        assert ds == 0
        assert np.array_equal(stg["r16"].view(np.uint16), st["r16"].view(np.uint16))
        assert int(np.sum(stg["z"] != st["z"])) <= 1
        bad += dc
        tot += stg["codes"].size
        og = host(o).reshape(o_or.shape)
        ot = step.truth_outputs(X, x["q"], x["k"], x["v"], x["s"], x["beta"])
        assert float(np.max(np.abs(og - ot)) / np.max(np.abs(ot))) <= 1e-3
        assert np.max(np.abs(og - o_or)) <= 1e-6 * np.max(np.abs(o_or))
    # the budget is met exactly
    assert int(stg["widths"].sum()) == int(np.floor(w.mean_bits * w.H * D + 0.5)) or scope == 1
    assert bad / tot <= 1e-5


def test_prefill_d256_ragged():
    w = W.sized(W.WORKLOADS["gdn6"], B=1, H=2, T=20, bf16=True)
    kc, oc = _cfgs(w, scope=1)
    xs = W.tokens(w, 0, 20)
    st0 = step.zero_state(w.B, w.H, oc)
    recs = dev(state_to_bytes(st0, D, D, w.b_max))
    T = 20
    o = torch.zeros(w.B * T * w.H * D, dtype=torch.float32, device="cuda")
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(torch.bfloat16).cuda()
    ws = K.new_workspace(kc)
    K.kda_prefill(kc, T, 8, recs, bf(xs["q"]), bf(xs["k"]), bf(xs["v"]), dev(_s_arg(xs["s"], w)),
                  dev(xs["beta"]), o, ws)
    st, o_or, _ = step.mirror_prefill(st0, xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], 8, oc)
    stg = bytes_to_state(host(recs), w.B, w.H, D, D, w.b_max)
    plain_check(ws_state32(ws, w), prefill_gamma(st0, xs, 8, oc.span), stg, G=w.G, scope=1,
                mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max, label="prefill d=256")
    dc = _codes_off(stg, st)
    say(f"prefill d=256 C=8 T=20: codes {dc} of {stg['codes'].size}")
    assert np.array_equal(stg["ntok"], st["ntok"])
    assert np.array_equal(stg["widths"], st["widths"])
    assert np.array_equal(stg["scale"].view(np.uint16), st["scale"].view(np.uint16))
    assert dc / stg["codes"].size <= 1e-5
    og = host(o).reshape(o_or.shape)
    assert np.max(np.abs(og - o_or)) <= 1e-6 * np.max(np.abs(o_or))
