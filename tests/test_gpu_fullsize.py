"""Parity at the benchmark's full size and launch configuration.

The decode workload (B=64 sequences, H=32 heads, d=128, 4-bit mean, layer
budget) runs as one kda_step launch exactly as bench.py times it.  Sampled
sequences start from oracle-made records (the others from the zero state:
sequences are independent) and are compared one by one with the oracle.
The long-context shape (Student-t values, 3-bit mean, window Gramian weights
recomputed by kda_weights) is checked the same way at a reduced batch.
"""
import numpy as np
import pytest
import torch

import paper_2609_30950_amd as K
import workloads as W
from oracle import record, stats, step
from tests._gpu import bytes_to_state, dev, host, say, state_to_bytes

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
    K.kda_step(kc, recs_d, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(x["s"]), dev(x["beta"]), o,
               K.new_workspace(kc))
    got = host(recs_d).reshape(w.B, w.H * slot)[sel].reshape(-1)
    og = host(o).reshape(w.B, w.H, w.dv)[sel]
    xo = {n: a[sel] for n, a in x.items()}
    X = step.dequantize(st0)
    st1, o_or, _ = step.mirror_decode_step(st0, xo["q"], xo["k"], xo["v"], xo["s"], xo["beta"], oc)
    _compare(bytes_to_state(got, len(sel), w.H, w.dk, w.dv, w.b_max), st1, "decode B=64 sampled")
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
        K.kda_step(kc, recs, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(x["s"]), dev(x["beta"]), o,
                   ws, gamma=dev(gam))
        st, o_or, _ = step.mirror_decode_step(st, x["q"], x["k"], x["v"], x["s"], x["beta"], oc,
                                              gamma=gam)
        _compare(bytes_to_state(host(recs), w.B, w.H, w.dk, w.dv, w.b_max), st, f"long t={t}")
