"""GPU parity without erasure (Mamba-2, eq. rule with a = 0) and with
output-normalisation groups spanning heads (Mamba-2 normalises over 12 heads).

* oracle-forced decode steps on a reduced Mamba-2-shaped layer (groups of 3
  heads) and on the full 24-head layer of one sequence (groups of 12 heads);
* prefill with write-backs every C tokens and a ragged last chunk;
* the 32-bit mode (plain recurrence) and both Gramian weight functions.
"""
import numpy as np
import pytest
import torch

import paper_2609_30950_amd as K
import workloads as W
from oracle import recurrence, stats, step
from tests._gpu import (bytes_to_state, decode_gamma, decode_state_gpu, dev, host, plain_check,
                        prefill_gamma, say, state_to_bytes, ws_state32)

pytestmark = pytest.mark.gpu


def _cfgs(w, state32=0):
    kc = K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.G, mean_bits=w.mean_bits,
                  b_min=w.b_min, b_max=w.b_max, decay_per_head=1, state32=state32, no_erase=1)
    oc = step.Cfg(dk=w.dk, dv=w.dv, G=w.G, mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max,
                  erase=False)
    return kc, oc


def _compare(stg, st, label):
    assert np.array_equal(stg["ntok"], st["ntok"]), label
    dw = int(np.sum(stg["widths"] != st["widths"]))
    ds = int(np.sum(stg["scale"].view(np.uint16) != st["scale"].view(np.uint16)))
    dz = int(np.sum(stg["z"] != st["z"]))
    same = stg["widths"] == st["widths"]
    dc = int(np.sum((stg["codes"] != st["codes"]) & same[..., None]))
    say(f"{label}: widths {dw} scales {ds} zcodes {dz} codes {dc}")
    assert dw == 0 and ds == 0, label
    assert np.all(stg["r16"].view(np.uint16) == 0), label     # no erase statistic
    assert dz <= max(1, stg["z"].size // 100000), label
    return dc, stg["codes"].size


@pytest.mark.parametrize("H,G", [(6, 3 * 128), (24, 12 * 128)])
def test_forced_decode_no_erasure_groups_across_heads(H, G):
    w = W.sized(W.WORKLOADS["mamba2"], B=1 if H == 24 else 2, H=H, G=G)
    kc, oc = _cfgs(w)
    xs = W.tokens(w, 0, 16)
    st, _ = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    ws = K.new_workspace(kc)
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    bad = tot = 0
    for t in range(16, 19):
        x = W.token(w, t)
        recs = dev(state_to_bytes(st, w.dk, w.dv, w.b_max))
        before = recs.clone()
        K.kda_step(kc, recs, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(x["s"][..., 0]),
                   dev(x["beta"]), o, ws)
        plain_check(decode_state_gpu(kc, before, ws), decode_gamma(st, x, oc.span, erase=False),
                    bytes_to_state(host(recs), w.B, w.H, w.dk, w.dv, w.b_max), G=w.G, scope=0,
                    mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max,
                    label=f"mamba2 H={H} G={G} t={t}")
        X = step.dequantize(st)
        st, o_or, _ = step.mirror_decode_step(st, x["q"], x["k"], x["v"], x["s"], x["beta"], oc)
        stg = bytes_to_state(host(recs), w.B, w.H, w.dk, w.dv, w.b_max)
        dc, n = _compare(stg, st, f"mamba2 H={H} G={G} t={t}")
        bad += dc
        tot += n
        og = host(o).reshape(o_or.shape)
        ot = step.truth_outputs(X, x["q"], x["k"], x["v"], x["s"], x["beta"], erase=False)
        assert float(np.max(np.abs(og - ot)) / np.max(np.abs(ot))) <= 1e-3
        assert np.max(np.abs(og - o_or)) <= 1e-6 * np.max(np.abs(o_or))
    assert bad / tot <= 1e-5


def test_prefill_no_erasure_ragged():
    w = W.sized(W.WORKLOADS["mamba2"], B=1, H=6, G=3 * 128, T=40, bf16=True)
    kc, oc = _cfgs(w)
    xs = W.tokens(w, 0, w.T)
    C = 16
    recs = K.new_records(kc)
    ws = K.new_workspace(kc)
    o = torch.zeros(w.B * w.T * w.H * w.dv, dtype=torch.float32, device="cuda")
    K.kda_prefill(kc, w.T, C, recs, dev(xs["q"], torch.bfloat16), dev(xs["k"], torch.bfloat16),
                  dev(xs["v"], torch.bfloat16), dev(xs["s"][..., 0]), dev(xs["beta"]), o, ws)
    st, o_or, _ = step.mirror_prefill(step.zero_state(w.B, w.H, oc), xs["q"], xs["k"], xs["v"],
                                      xs["s"], xs["beta"], C, oc)
    stg = bytes_to_state(host(recs), w.B, w.H, w.dk, w.dv, w.b_max)
    st0 = step.zero_state(w.B, w.H, oc)
    plain_check(ws_state32(ws, w), prefill_gamma(st0, xs, C, oc.span, erase=False), stg, G=w.G,
                scope=0, mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max,
                label="mamba2 prefill")
    dc, n = _compare(stg, st, "mamba2 prefill")
    assert dc / n <= 1e-5
    og = host(o).reshape(o_or.shape)
    assert np.max(np.abs(og - o_or)) <= 1e-5 * np.max(np.abs(o_or))


def test_state32_no_erasure():
    w = W.sized(W.WORKLOADS["mamba2"], B=2, H=3, G=128)
    kc, _ = _cfgs(w, state32=1)
    rng = np.random.default_rng(31)
    S = rng.standard_normal((w.B, w.H, w.dk, w.dv)).astype(np.float32)
    recs = dev(S.reshape(-1).view(np.uint8))
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    X = S
    for t in range(6):
        x = W.token(w, t)
        K.kda_step(kc, recs, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(x["s"][..., 0]),
                   dev(x["beta"]), o, None)
        X, o_or = recurrence.mirror_step(X, x["q"], x["k"], x["v"], x["s"], x["beta"], erase=False)
        Sg = host(recs).view(np.float32).reshape(X.shape)
        assert int(np.sum(Sg.view(np.uint32) != X.view(np.uint32))) <= X.size // 10000
        assert np.max(np.abs(host(o).reshape(o_or.shape) - o_or)) <= 1e-6 * np.max(np.abs(o_or))
        X = Sg


def test_weights_no_erasure():
    w = W.sized(W.WORKLOADS["mamba2"], B=1, H=2, G=128)
    kc, _ = _cfgs(w)
    Wn = 40
    xs = W.tokens(w, 0, Wn)
    g = torch.zeros(w.B * w.H * w.dk, dtype=torch.float64, device="cuda")
    K.kda_weights(kc, Wn, 2, dev(xs["q"]), dev(xs["s"][..., 0]), dev(xs["beta"]), dev(xs["k"]), g)
    want = stats.window_gamma(np.moveaxis(xs["q"], 1, 0), np.moveaxis(xs["s"], 1, 0),
                              np.moveaxis(xs["k"], 1, 0), np.moveaxis(xs["beta"], 1, 0), 2,
                              erase=False)
    np.testing.assert_allclose(host(g).reshape(want.shape), want, rtol=1e-12)
    K.kda_weights_exact(kc, Wn, 2, dev(xs["q"]), dev(xs["s"][..., 0]), dev(xs["beta"]),
                        dev(xs["k"]), g)
    ge = host(g).reshape(want.shape)
    # without erasure the transition is diagonal: the exact Gramian is the
    # per-row recursion (pinned in the oracle)
    np.testing.assert_allclose(ge, want, rtol=1e-9)
