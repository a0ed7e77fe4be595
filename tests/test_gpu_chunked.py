"""GPU parity of the chunked (WY/UT, bf16 MFMA) prefill.

The chunked form evaluates the same recurrence (eq. rule) in another order:
products on bf16 MFMA with float32 accumulation, each operand that is not
exact in bf16 split into hi and lo bf16 parts (relative 2^-18) and multiplied
as three products.  Its state and outputs are compared with the float64
recurrence from the same starting record within 1e-3 (the outputs' accuracy bound) of the
head's largest |S| (state) or largest |o| (outputs), normwise; observed
errors are printed.  Its write-back is compared bit for bit with the oracle's
quantiser applied to the GPU's own float32 state (EMA statistics from the
oracle's token-order recursion), and checked against the plain definitions.
A multi-chunk call must equal the same chunks run one call at a time, bit for
bit.
"""
import numpy as np
import pytest
import torch

import paper_2609_30950_amd as K
import workloads as W
from oracle import recurrence, stats, step
from tests._gpu import bytes_to_state, dev, host, plain_check, say, state_to_bytes, ws_state32

pytestmark = pytest.mark.gpu

TOL = 1e-3


def _cfgs(w, scope=0, no_erase=False):
    kc = K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.G, scope=scope,
                  mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max,
                  decay_per_head=int(w.decay == "head"), no_erase=int(no_erase), chunked=1)
    oc = step.Cfg(dk=w.dk, dv=w.dv, G=w.G, scope="sequence" if scope == 0 else "head",
                  mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max, erase=not no_erase)
    return kc, oc


def _bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(torch.bfloat16).cuda()


_AUX = []


def _aux():
    """The caller's second stream for the preparation of later chunks."""
    if not _AUX:
        _AUX.append(torch.cuda.Stream())
    return _AUX[0]


def _gpu_prefill(kc, w, st0, xs, C):
    T = xs["q"].shape[1]
    recs = dev(state_to_bytes(st0, w.dk, w.dv, w.b_max))
    o = torch.zeros(w.B * T * w.H * w.dv, dtype=torch.float32, device="cuda")
    ws = K.new_workspace(kc)
    s_arg = xs["s"] if w.decay != "head" else xs["s"][..., 0]
    K.kda_prefill(kc, T, C, recs, _bf16(xs["q"]), _bf16(xs["k"]), _bf16(xs["v"]), dev(s_arg),
                  dev(xs["beta"]), o, ws, aux_stream=_aux())
    return recs, o, ws


def _bf16_round(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16).float().numpy()


def _one_interval(w, st0, xs, oc, kc, label):
    """One write-back interval (T <= 64 tokens, C = 64)."""
    T = xs["q"].shape[1]
    recs, o, ws = _gpu_prefill(kc, w, st0, xs, 64)
    Sg = ws_state32(ws, w)
    og = host(o).reshape(w.B, T, w.H, w.dv)
    # float64 recurrence from the same dequantised start, on the bf16 inputs
    X = step.dequantize(st0).astype(np.float64)
    q, k, v = (_bf16_round(xs[n]) for n in ("q", "k", "v"))
    ot = np.zeros_like(og, dtype=np.float64)
    m, e = step.ema_start(st0)
    fresh = (st0["ntok"] == 0)[..., None]
    for t in range(T):
        X, ot[:, t] = recurrence.truth_step_rowform(X, q[:, t], k[:, t], v[:, t], xs["s"][:, t],
                                                    xs["beta"][:, t], oc.erase)
        sr = np.broadcast_to(xs["s"][:, t], xs["s"][:, t].shape[:-1] + (w.dk,))
        bt = np.asarray(xs["beta"][:, t])[..., None]
        mi, ei = stats.ema_init(sr, k[:, t], bt, oc.erase)
        mu, eu = stats.ema_update(m, e, sr, k[:, t], bt, oc.span, oc.erase)
        m = np.where(fresh, mi, mu)
        e = np.where(fresh, ei, eu)
        fresh = np.zeros_like(fresh)
    es = np.max(np.abs(Sg - X), axis=(2, 3)) / np.max(np.abs(X), axis=(2, 3))
    eo = np.max(np.abs(og - ot), axis=(1, 3)) / np.max(np.abs(ot), axis=(1, 3))
    say(f"{label}: state err {es.max():.2e}, output err {eo.max():.2e} (bound {TOL:.2e})")
    assert np.all(np.isfinite(Sg)) and np.all(np.isfinite(og))
    assert es.max() <= TOL
    assert eo.max() <= TOL
    # the write-back of the GPU's own state, bit for bit
    exp, _ = step.write_back(Sg, m, e, st0["ntok"] + T, oc)
    got = bytes_to_state(host(recs), w.B, w.H, w.dk, w.dv, w.b_max)
    s_hat, r = stats.ema_rates(m, e)
    plain_check(Sg, stats.mode_gamma(s_hat, r), got, G=w.G, scope=kc.scope,
                mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max, label=label)
    for f in ("ntok", "widths", "z", "r16", "codes"):
        assert np.array_equal(got[f], exp[f]), f
    assert np.array_equal(got["scale"].view(np.uint16), exp["scale"].view(np.uint16))
    return got


@pytest.mark.parametrize("T", [64, 37, 1])
def test_chunk_d64_warm(T):
    w = W.sized(W.WORKLOADS["tiny"], bf16=True)
    kc, oc = _cfgs(w)
    warm = W.tokens(w, 0, 48)
    st0, _ = step.warm_state(warm["q"], warm["k"], warm["v"], warm["s"], warm["beta"], oc)
    _one_interval(w, st0, W.tokens(w, 48, 48 + T), oc, kc, f"chunk d=64 T={T}")


def test_chunk_d64_fresh_record():
    w = W.sized(W.WORKLOADS["tiny"], bf16=True)
    kc, oc = _cfgs(w)
    _one_interval(w, step.zero_state(w.B, w.H, oc), W.tokens(w, 0, 50), oc, kc, "chunk fresh")


def test_chunk_d128_prefill_shape():
    w = W.sized(W.WORKLOADS["prefill"], B=1, H=4)
    kc, oc = _cfgs(w)
    warm = W.tokens(w, 0, 16)
    st0, _ = step.warm_state(warm["q"], warm["k"], warm["v"], warm["s"], warm["beta"], oc)
    _one_interval(w, st0, W.tokens(w, 16, 16 + 64), oc, kc, "chunk d=128 prefill shape")


def test_chunk_large_decay_uses_exact_diagonal_blocks():
    """Decay rates of 6 per token: a 16-token block spans exponents of 96, past
    the split bound, so the diagonal blocks take the per-pair path; the
    off-diagonal factors underflow to zero, as the true ones nearly do."""
    w = W.sized(W.WORKLOADS["tiny"], bf16=True)
    kc, oc = _cfgs(w)
    warm = W.tokens(w, 0, 16)
    st0, _ = step.warm_state(warm["q"], warm["k"], warm["v"], warm["s"], warm["beta"], oc)
    xs = W.tokens(w, 16, 16 + 64)
    xs["s"] = xs["s"].copy()
    xs["s"][..., : w.dk // 2] = 6.0
    _one_interval(w, st0, xs, oc, kc, "chunk large decay")


def test_chunk_per_head_decay_head_scope():
    w = W.sized(W.WORKLOADS["gdn2"], B=1, H=4, dk=64, dv=64, G=64, T=40, bf16=True)
    kc, oc = _cfgs(w, scope=1)
    warm = W.tokens(w, 0, 24)
    st0, _ = step.warm_state(warm["q"], warm["k"], warm["v"], warm["s"], warm["beta"], oc)
    _one_interval(w, st0, W.tokens(w, 24, 24 + 40), oc, kc, "chunk per-head decay")


def test_chunk_d128_head_scope_two_groups_per_head():
    """d = 128 with groups of 64 rows (two per head) and the per-head budget:
    the apply blocks form both groups' weights and each requantisation block
    selects its own head's widths."""
    w = W.sized(W.WORKLOADS["prefill"], B=2, H=3, G=64)
    kc, oc = _cfgs(w, scope=1)
    warm = W.tokens(w, 0, 16)
    st0, _ = step.warm_state(warm["q"], warm["k"], warm["v"], warm["s"], warm["beta"], oc)
    _one_interval(w, st0, W.tokens(w, 16, 16 + 45), oc, kc, "chunk d=128 head scope G=64")


def test_chunk_no_erase_d128():
    w = W.sized(W.WORKLOADS["mamba2"], B=1, H=12, T=64, bf16=True)
    kc, oc = _cfgs(w, no_erase=True)
    warm = W.tokens(w, 0, 16)
    st0, _ = step.warm_state(warm["q"], warm["k"], warm["v"], warm["s"], warm["beta"], oc)
    _one_interval(w, st0, W.tokens(w, 16, 16 + 64), oc, kc, "chunk no erasure")


@pytest.mark.parametrize("n64", [18, 40])
def test_multi_chunk_call_equals_single_interval_calls(n64):
    """T = n64 intervals of 64 plus a ragged 5, in groups of chunks growing
    from one to 16 (later groups' records reuse earlier groups' space,
    prepared on the caller's second stream once those groups' intervals are
    done): one call against the single-interval calls, bit for bit; and the
    same call on one stream."""
    w = W.sized(W.WORKLOADS["tiny"], bf16=True)
    kc, oc = _cfgs(w)
    T = n64 * 64 + 5
    xs = W.tokens(w, 0, T)
    st0 = step.zero_state(w.B, w.H, oc)
    recs, o, _ = _gpu_prefill(kc, w, st0, xs, 64)
    whole = host(recs)
    o_whole = host(o).reshape(w.B, T, w.H, w.dv)
    r = dev(state_to_bytes(st0, w.dk, w.dv, w.b_max))
    ws = K.new_workspace(kc)
    parts = []
    for t0 in range(0, T, 64):
        t1 = min(T, t0 + 64)
        sub = {n: np.ascontiguousarray(xs[n][:, t0:t1]) for n in xs}
        o1 = torch.zeros(w.B * (t1 - t0) * w.H * w.dv, dtype=torch.float32, device="cuda")
        K.kda_prefill(kc, t1 - t0, 64, r, _bf16(sub["q"]), _bf16(sub["k"]), _bf16(sub["v"]),
                      dev(sub["s"]), dev(sub["beta"]), o1, ws)
        parts.append(host(o1).reshape(w.B, t1 - t0, w.H, w.dv))
    say(f"multi-chunk: {len(parts)} intervals")
    assert np.array_equal(host(r), whole)
    assert np.array_equal(np.concatenate(parts, axis=1).view(np.uint32), o_whole.view(np.uint32))
    r1 = dev(state_to_bytes(st0, w.dk, w.dv, w.b_max))
    o1 = torch.zeros(w.B * T * w.H * w.dv, dtype=torch.float32, device="cuda")
    K.kda_prefill(kc, T, 64, r1, _bf16(xs["q"]), _bf16(xs["k"]), _bf16(xs["v"]), dev(xs["s"]),
                  dev(xs["beta"]), o1, K.new_workspace(kc))
    assert np.array_equal(host(r1), whole)
    assert torch.equal(o1.view(torch.int32), o.view(torch.int32))


def test_chunked_rejects_long_interval_and_wide_heads():
    w = W.sized(W.WORKLOADS["tiny"], bf16=True)
    kc, oc = _cfgs(w)
    xs = W.tokens(w, 0, 8)
    with pytest.raises(K.KdaError):
        _gpu_prefill(kc, w, step.zero_state(w.B, w.H, oc), xs, 65)
    wide = K.Config(B=1, H=1, d_k=256, d_v=256, group_rows=256, chunked=1)
    assert K.record_bytes(wide) == 0
