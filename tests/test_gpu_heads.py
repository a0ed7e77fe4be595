"""GPU parity of head allocation units with block scales (Gated DeltaNet: one
width per head, FP16 scales per 32 rows of a column) against the oracle:
oracle-forced decode steps (d = 64 and the d = 256 Gated-DeltaNet shape at
mean 2 and 6 bits), a ragged bf16 prefill from the empty state, given row
weights, and the entry points this unit type does not support."""
import numpy as np
import pytest
import torch

import paper_2609_30950_amd as K
import workloads as W
from oracle import record, step
from tests._gpu import decode_gamma, dev, host, plain_check_heads, say, state32_step_gpu

pytestmark = pytest.mark.gpu


def _cfgs(w):
    kc = K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.dk, mean_bits=w.mean_bits,
                  b_min=2, b_max=w.b_max, decay_per_head=int(w.decay == "head"), head_units=1)
    oc = step.Cfg(dk=w.dk, dv=w.dv, G=w.dk, mean_bits=w.mean_bits, b_min=2, b_max=w.b_max,
                  unit="head")
    return kc, oc


def _s_arg(s, w):
    return s if w.decay != "head" else s[..., 0]


def _to_bytes(st, w):
    out = [record.pack_heads(st["ntok"][b, h], st["width"][b, h], st["bscale"][b, h],
                             st["z"][b, h], st["r16"][b, h], st["codes"][b, h], w.dk, w.dv,
                             w.b_max)
           for b in range(w.B) for h in range(w.H)]
    return np.concatenate(out)


def _from_bytes(buf, w):
    slot = record.record_bytes_heads(w.dk, w.dv, w.b_max)
    buf = np.asarray(buf, np.uint8).reshape(w.B, w.H, slot)
    fs = [[record.unpack_heads(buf[b, h], w.dk, w.dv, w.b_max) for h in range(w.H)]
          for b in range(w.B)]
    st = {k: np.stack([np.stack([np.asarray(fs[b][h][k]) for h in range(w.H)]) for b in range(w.B)])
          for k in ("ntok", "width", "bscale", "z", "r16", "codes")}
    return st


def _check(stg, st, label):
    same = stg["width"] == st["width"]
    dc = int(np.sum((stg["codes"] != st["codes"]) & same[..., None, None]))
    ds = int(np.sum(stg["bscale"].view(np.uint16) != st["bscale"].view(np.uint16)))
    say(f"{label}: widths {stg['width'].ravel().tolist()} vs {st['width'].ravel().tolist()}, "
        f"scales {ds} codes {dc} of {stg['codes'].size}")
    assert np.array_equal(stg["ntok"], st["ntok"])
    assert np.array_equal(stg["width"], st["width"])
    assert ds == 0
    assert dc == 0
    assert np.array_equal(stg["r16"].view(np.uint16), st["r16"].view(np.uint16))
    assert int(np.sum(stg["z"] != st["z"])) <= 1


@pytest.mark.parametrize("name,dk,H,mean", [("gdn2", 64, 4, 3.0), ("gdn2", 256, 16, 2.0),
                                             ("gdn6", 256, 16, 6.0), ("gdn2", 128, 8, 4.5)])
def test_forced_decode_steps_heads(name, dk, H, mean):
    w = W.sized(W.WORKLOADS[name], B=2 if dk < 256 else 1, H=H, dk=dk, dv=dk, G=dk,
                mean_bits=mean)
    kc, oc = _cfgs(w)
    xs = W.tokens(w, 0, 6)
    st, _ = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    ws = K.new_workspace(kc)
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    base = W.base_rates(w)
    for t in range(6, 9):
        x = W.token(w, t, base=base)
        recs = dev(_to_bytes(st, w))
        K.kda_step(kc, recs, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(_s_arg(x["s"], w)),
                   dev(x["beta"]), o, ws)
        X = step.dequantize(st)
        stg = _from_bytes(host(recs), w)
        plain_check_heads(state32_step_gpu(kc, X, x), decode_gamma(st, x, oc.span), stg,
                          mean_bits=w.mean_bits, b_min=2, b_max=w.b_max,
                          label=f"heads {name} d={dk} mean={mean} t={t}")
        st, o_or, _ = step.mirror_decode_step(st, x["q"], x["k"], x["v"], x["s"], x["beta"], oc)
        _check(stg, st, f"heads {name} d={dk} mean={mean} t={t}")
        og = host(o).reshape(o_or.shape)
        ot = step.truth_outputs(X, x["q"], x["k"], x["v"], x["s"], x["beta"])
        assert float(np.max(np.abs(og - ot)) / np.max(np.abs(ot))) <= 1e-3
        assert np.max(np.abs(og - o_or)) <= 1e-6 * np.max(np.abs(o_or))
    assert int(st["width"].sum()) == w.B * int(np.floor(mean * w.H + 0.5))


def test_decode_chain_from_empty_state():
    """Eight steps chained on the GPU's own records from the zero state."""
    w = W.sized(W.WORKLOADS["gdn2"], B=2, H=4, dk=64, dv=64, G=64, mean_bits=3.0)
    kc, oc = _cfgs(w)
    st = step.zero_state(w.B, w.H, oc)
    recs = dev(_to_bytes(st, w))
    ws = K.new_workspace(kc)
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    base = W.base_rates(w)
    for t in range(8):
        x = W.token(w, t, base=base)
        K.kda_step(kc, recs, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(_s_arg(x["s"], w)),
                   dev(x["beta"]), o, ws)
        st, o_or, _ = step.mirror_decode_step(st, x["q"], x["k"], x["v"], x["s"], x["beta"], oc)
        _check(_from_bytes(host(recs), w), st, f"chain t={t}")
        assert np.max(np.abs(host(o).reshape(o_or.shape) - o_or)) <= 1e-6 * np.max(np.abs(o_or))


def test_prefill_heads_ragged_bf16():
    w = W.sized(W.WORKLOADS["gdn6"], B=1, H=4, dk=128, dv=128, G=128, T=20, bf16=True)
    kc, oc = _cfgs(w)
    xs = W.tokens(w, 0, 20)
    st0 = step.zero_state(w.B, w.H, oc)
    recs = dev(_to_bytes(st0, w))
    T = 20
    o = torch.zeros(w.B * T * w.H * w.dv, dtype=torch.float32, device="cuda")
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(torch.bfloat16).cuda()
    K.kda_prefill(kc, T, 8, recs, bf(xs["q"]), bf(xs["k"]), bf(xs["v"]), dev(_s_arg(xs["s"], w)),
                  dev(xs["beta"]), o, K.new_workspace(kc))
    st, o_or, _ = step.mirror_prefill(st0, xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], 8, oc)
    _check(_from_bytes(host(recs), w), st, "prefill heads C=8 T=20")
    og = host(o).reshape(o_or.shape)
    assert np.max(np.abs(og - o_or)) <= 1e-6 * np.max(np.abs(o_or))


def test_given_row_weights():
    """With given weights the head keys are their row means."""
    w = W.sized(W.WORKLOADS["gdn2"], B=1, H=8, dk=64, dv=64, G=64, mean_bits=4.0)
    kc, oc = _cfgs(w)
    xs = W.tokens(w, 0, 4)
    st, _ = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    rng = np.random.default_rng(3)
    gamma = np.exp(rng.uniform(-6, 6, (w.B, w.H, 1)) + rng.uniform(-1, 1, (w.B, w.H, w.dk)))
    x = W.token(w, 4, base=W.base_rates(w))
    recs = dev(_to_bytes(st, w))
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    K.kda_step(kc, recs, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(_s_arg(x["s"], w)),
               dev(x["beta"]), o, K.new_workspace(kc), gamma=dev(gamma))
    stg = _from_bytes(host(recs), w)
    plain_check_heads(state32_step_gpu(kc, step.dequantize(st), x), gamma, stg,
                      mean_bits=w.mean_bits, b_min=2, b_max=w.b_max, label="given weights")
    st, _, _ = step.mirror_decode_step(st, x["q"], x["k"], x["v"], x["s"], x["beta"], oc,
                                       gamma=gamma)
    _check(stg, st, "given weights")
    assert len(set(st["width"].ravel().tolist())) > 1


def test_head_units_unsupported_entry_points():
    w = W.sized(W.WORKLOADS["gdn2"], B=1, H=2, dk=64, dv=64, G=64)
    kc, _ = _cfgs(w)
    recs = K.new_records(kc)
    S = torch.zeros(w.B * w.H * 64 * 64, dtype=torch.float32, device="cuda")
    with pytest.raises(K.KdaError):
        K.kda_unpack_state(kc, recs, S, None, None, None)
