"""GPU parity of kda_prefill (write-back every C tokens and after the last)
against the oracle, from oracle-made starting records.  The last write-back
of every call is also checked against the plain definitions of widths,
clip factors, scales and codes (oracle/plain.py) on the GPU's own float32
state before it."""
import numpy as np
import pytest
import torch

import paper_2609_30950_amd as K
import workloads as W
from oracle import recurrence, step
from tests._gpu import (bytes_to_state, dev, host, plain_check, prefill_gamma, say,
                        state_to_bytes, ws_state32)

pytestmark = pytest.mark.gpu


def _cfgs(w, scope=0):
    kc = K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.G, scope=scope,
                  mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max,
                  decay_per_head=int(w.decay == "head"))
    oc = step.Cfg(dk=w.dk, dv=w.dv, G=w.G, scope="sequence" if scope == 0 else "head",
                  mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max)
    return kc, oc


def _bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(torch.bfloat16).cuda()


def _run(w, st0, xs, C, scope=0):
    kc, oc = _cfgs(w, scope)
    T = xs["q"].shape[1]
    recs = dev(state_to_bytes(st0, w.dk, w.dv, w.b_max))
    o = torch.zeros(w.B * T * w.H * w.dv, dtype=torch.float32, device="cuda")
    s_arg = xs["s"] if w.decay != "head" else xs["s"][..., 0]
    ws = K.new_workspace(kc)
    K.kda_prefill(kc, T, C, recs, _bf16(xs["q"]), _bf16(xs["k"]), _bf16(xs["v"]), dev(s_arg),
                  dev(xs["beta"]), o, ws)
    st, o_or, diags = step.mirror_prefill(st0, xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], C, oc)
    stg = bytes_to_state(host(recs), w.B, w.H, w.dk, w.dv, w.b_max)
    og = host(o).reshape(o_or.shape)
    plain_check(ws_state32(ws, w), prefill_gamma(st0, xs, C, oc.span), stg, G=w.G, scope=scope,
                mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max,
                label=f"prefill B={w.B} H={w.H} d={w.dk} T={T} C={C}")
    return stg, st, og, o_or


def _check_state(stg, st, label):
    same_w = stg["widths"] == st["widths"]
    dc = int(np.sum((stg["codes"] != st["codes"]) & same_w[..., None])) + \
        int(np.sum(~same_w)) * stg["codes"].shape[-1]
    ds = int(np.sum(stg["scale"].view(np.uint16) != st["scale"].view(np.uint16)))
    say(f"{label}: widths {int(np.sum(~same_w))} scales {ds} codes {dc} of {stg['codes'].size}")
    assert np.array_equal(stg["ntok"], st["ntok"])
    assert np.array_equal(stg["widths"], st["widths"])
    assert ds == 0
    assert dc / stg["codes"].size <= 1e-5




@pytest.mark.parametrize("C", [16, 1])
def test_prefill_tiny_ragged(C):
    w = W.sized(W.WORKLOADS["tiny"], bf16=True)
    kc, oc = _cfgs(w)
    T = 38
    xs = W.tokens(w, 0, T)
    st0 = step.zero_state(w.B, w.H, oc)
    stg, st, og, o_or = _run(w, st0, xs, C)
    _check_state(stg, st, f"prefill tiny C={C}")
    assert np.max(np.abs(og - o_or)) <= 1e-6 * np.max(np.abs(o_or))


def test_prefill_outputs_match_truth_within_chunk():
    """Inside one write-back interval the state is float32; outputs agree with
    the float64 recurrence from the same starting state to 1e-3 (normwise)."""
    w = W.sized(W.WORKLOADS["prefill"], B=1, H=2, dk=64, dv=64, G=64)
    kc, oc = _cfgs(w)
    warm = W.tokens(w, 0, 32)
    st0, _ = step.warm_state(warm["q"], warm["k"], warm["v"], warm["s"], warm["beta"], oc)
    xs = W.tokens(w, 32, 32 + 48)
    stg, st, og, o_or = _run(w, st0, xs, 64)     # one chunk: 48 tokens, one write-back
    _check_state(stg, st, "prefill one chunk")
    X = step.dequantize(st0).astype(np.float64)
    worst = 0.0
    for t in range(48):
        X, ot = recurrence.truth_step_rowform(X, xs["q"][:, t], xs["k"][:, t], xs["v"][:, t],
                                              xs["s"][:, t], xs["beta"][:, t])
        worst = max(worst, float(np.max(np.abs(og[:, t] - ot)) / np.max(np.abs(ot))))
    say(f"prefill o vs float64 truth: worst normwise rel err {worst:.2e}")
    assert worst <= 1e-3


def test_prefill_decode_shape_layer_budget():
    w = W.sized(W.WORKLOADS["prefill"], B=1, T=80)
    kc, oc = _cfgs(w)
    warm = W.tokens(w, 0, 16)
    st0, _ = step.warm_state(warm["q"], warm["k"], warm["v"], warm["s"], warm["beta"], oc)
    xs = W.tokens(w, 16, 16 + 80)
    stg, st, og, o_or = _run(w, st0, xs, 32)     # write-backs after 32, 64 and 80
    _check_state(stg, st, "prefill 32x128 heads C=32")
    assert np.max(np.abs(og - o_or)) <= 1e-6 * np.max(np.abs(o_or))


def test_prefill_per_head_decay_head_scope():
    w = W.sized(W.WORKLOADS["gdn2"], B=1, H=4, dk=64, dv=64, G=64, T=40, bf16=True)
    kc, oc = _cfgs(w, scope=1)
    xs = W.tokens(w, 0, 40)
    st0 = step.zero_state(w.B, w.H, oc)
    stg, st, og, o_or = _run(w, st0, xs, 8, scope=1)
    _check_state(stg, st, "prefill per-head decay, head scope")


def test_prefill_state32():
    w = W.sized(W.WORKLOADS["tiny"], bf16=True)
    kc, _ = _cfgs(w)
    kc.state32 = 1
    T = 20
    xs = W.tokens(w, 0, T)
    rng = np.random.default_rng(9)
    S0 = rng.standard_normal((w.B, w.H, w.dk, w.dv)).astype(np.float32)
    recs = dev(S0.reshape(-1).view(np.uint8))
    o = torch.zeros(w.B * T * w.H * w.dv, dtype=torch.float32, device="cuda")
    K.kda_prefill(kc, T, 4, recs, _bf16(xs["q"]), _bf16(xs["k"]), _bf16(xs["v"]), dev(xs["s"]),
                  dev(xs["beta"]), o, None)
    X = S0
    for t in range(T):
        X, _ = recurrence.mirror_step(X, xs["q"][:, t], xs["k"][:, t], xs["v"][:, t], xs["s"][:, t],
                                      xs["beta"][:, t])
    Sg = host(recs).view(np.float32).reshape(X.shape)
    assert np.sum(Sg.view(np.uint32) != X.view(np.uint32)) <= X.size // 10000
