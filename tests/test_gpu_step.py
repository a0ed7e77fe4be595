"""GPU parity of kda_step against the oracle.

* 32-bit mode: float32 contract of the recurrence, free-running.
* quantised decode, free-running from the zero state (tiny workload, all
  256 tokens): both sides run their own trajectories from identical inputs.
* oracle-forced single steps on the decode workload's shape (layer budget
  over 32 heads x 128 rows): the GPU starts from records the oracle produced
  and its output is compared with the oracle's next record.

Every quantised step is also checked against the plain definitions of the
widths, clip factors, scales and codes (oracle/plain.py) on the GPU's own
float32 state, independently of the float32 contract's evaluation order.
"""
import numpy as np
import pytest
import torch

import paper_2609_30950_amd as K
import workloads as W
from oracle import recurrence, step
from tests._gpu import (bytes_to_state, decode_gamma, decode_state_gpu, dev, host,
                        meaningful_equal, plain_check, say, state_to_bytes)

pytestmark = pytest.mark.gpu


def _cfgs(w, scope=0, span=64, state32=0):
    kc = K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.G, scope=scope,
                  mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max, ema_span=span,
                  decay_per_head=int(w.decay == "head"), state32=state32)
    oc = step.Cfg(dk=w.dk, dv=w.dv, G=w.G, scope="sequence" if scope == 0 else "head",
                  mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max, span=span)
    return kc, oc


def _s_arg(x, w):
    return x["s"] if w.decay != "head" else x["s"][..., 0]


def _compare(st_gpu, st_or, label):
    """Field-wise comparison; returns (code and rate-code mismatches, codes
    and rate codes compared)."""
    assert np.array_equal(st_gpu["ntok"], st_or["ntok"]), label
    dw = int(np.sum(st_gpu["widths"] != st_or["widths"]))
    ds = int(np.sum(st_gpu["scale"].view(np.uint16) != st_or["scale"].view(np.uint16)))
    dz = int(np.sum(st_gpu["z"] != st_or["z"]))
    dr = int(np.sum(st_gpu["r16"].view(np.uint16) != st_or["r16"].view(np.uint16)))
    same_w = st_gpu["widths"] == st_or["widths"]
    dc = int(np.sum((st_gpu["codes"] != st_or["codes"]) & same_w[..., None]))
    dc += int(np.sum(~same_w)) * st_gpu["codes"].shape[-1]
    say(f"{label}: widths {dw} scales {ds} zcodes {dz} r16 {dr} codes {dc}")
    assert dw == 0 and ds == 0 and dr == 0, label
    assert dz <= max(1, st_gpu["z"].size // 100000), label
    return dc + dz, st_gpu["codes"].size + st_gpu["z"].size


def _step_plain(kc, oc, recs, x, o, ws, st_old, label, gamma=None):
    """kda_step on device records, then the plain check of the new records
    on the GPU's own float32 state; returns the decoded new records."""
    before = recs.clone()
    K.kda_step(kc, recs, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(x["s"]), dev(x["beta"]), o,
               ws, gamma=None if gamma is None else dev(gamma))
    stg = bytes_to_state(host(recs), kc.B, kc.H, kc.d_k, kc.d_v, kc.b_max)
    S = decode_state_gpu(kc, before, ws)
    g = gamma if gamma is not None else decode_gamma(st_old, x, oc.span)
    plain_check(S, g, stg, G=kc.group_rows, scope=kc.scope, mean_bits=kc.mean_bits,
                b_min=kc.b_min, b_max=kc.b_max, label=label)
    return stg


@pytest.mark.parametrize("d", [64, 128])
def test_state32_step_matches_contract(d):
    w = W.sized(W.WORKLOADS["tiny"], B=2, H=3, dk=d, dv=d)
    kc, _ = _cfgs(w, state32=1)
    rng = np.random.default_rng(d)
    S = rng.standard_normal((w.B, w.H, d, d)).astype(np.float32)
    recs = dev(S.reshape(-1).view(np.uint8))
    o = torch.zeros(w.B * w.H * d, dtype=torch.float32, device="cuda")
    base = W.base_rates(w)
    X = S
    worst = 0
    for t in range(8):
        x = W.token(w, t, base=base)
        K.kda_step(kc, recs, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(x["s"]), dev(x["beta"]), o,
                   None)
        X, o_or = recurrence.mirror_step(X, x["q"], x["k"], x["v"], x["s"], x["beta"])
        Sg = host(recs).view(np.float32).reshape(X.shape)
        nbad = int(np.sum(Sg.view(np.uint32) != X.view(np.uint32)))
        worst = max(worst, nbad)
        assert nbad <= X.size // 10000, f"token {t}: {nbad} state values differ"
        og = host(o).reshape(o_or.shape)
        assert np.max(np.abs(og - o_or)) <= 1e-6 * np.max(np.abs(o_or))
        X = Sg            # continue from the GPU's own state (identical unless a rare exp ulp)
    say(f"state32 d={d}: worst mismatching state values per token {worst}")


def test_quantized_decode_free_running_tiny():
    """The tiny workload's whole run (T = 256 decode tokens from the zero
    state); the code-mismatch rate counts codes and rate codes."""
    w = W.WORKLOADS["tiny"]
    kc, oc = _cfgs(w)
    T = w.T
    recs = K.new_records(kc)
    ws = K.new_workspace(kc)
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    st = step.zero_state(w.B, w.H, oc)
    base = W.base_rates(w)
    bad = tot = 0
    worst_o = 0.0
    for t in range(T):
        x = W.token(w, t, base=base)
        stg = _step_plain(kc, oc, recs, x, o, ws, st, f"tiny t={t}")
        X = step.dequantize(st)
        st, o_or, _ = step.mirror_decode_step(st, x["q"], x["k"], x["v"], x["s"], x["beta"], oc)
        dc, n = _compare(stg, st, f"tiny t={t}")
        bad += dc
        tot += n
        og = host(o).reshape(o_or.shape)
        ot = step.truth_outputs(X, x["q"], x["k"], x["v"], x["s"], x["beta"])
        worst_o = max(worst_o, float(np.max(np.abs(og - ot)) / np.max(np.abs(ot))))
        if dc:
            st = stg      # continue each side from identical states only if needed
    say(f"free-running tiny, {T} tokens: code mismatch rate {bad / tot:.2e} ({bad} of {tot}), "
        f"worst o rel err {worst_o:.2e}")
    assert bad / tot <= 1e-5
    assert worst_o <= 1e-3


@pytest.mark.parametrize("scope", [0, 1])
def test_oracle_forced_steps_decode_shape(scope):
    w = W.sized(W.WORKLOADS["decode"], B=2)
    kc, oc = _cfgs(w, scope=scope)
    xs = W.tokens(w, 0, 24)
    st, _ = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    ws = K.new_workspace(kc)
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    base = W.base_rates(w)
    bad = tot = 0
    for t in range(24, 27):
        x = W.token(w, t, base=base)
        recs = dev(state_to_bytes(st, w.dk, w.dv, w.b_max))
        stg = _step_plain(kc, oc, recs, x, o, ws, st, f"decode-shape scope={scope} t={t}")
        X = step.dequantize(st)
        st, o_or, _ = step.mirror_decode_step(st, x["q"], x["k"], x["v"], x["s"], x["beta"], oc)
        dc, n = _compare(stg, st, f"decode-shape scope={scope} t={t}")
        bad += dc
        tot += n
        og = host(o).reshape(o_or.shape)
        ot = step.truth_outputs(X, x["q"], x["k"], x["v"], x["s"], x["beta"])
        err = float(np.max(np.abs(og - ot)) / np.max(np.abs(ot)))
        assert err <= 1e-3
        assert np.max(np.abs(og - o_or)) <= 1e-6 * np.max(np.abs(o_or))
    assert bad / tot <= 1e-5


@pytest.mark.parametrize("scope", [0, 1])
@pytest.mark.parametrize("d", [64, 128])
def test_forced_steps_narrow_widths(d, scope):
    # widths in [1, 3] at a 2-bit mean: the record's code words take less LDS
    # than the allocator's scratch, which the per-head budget places there
    w = W.sized(W.WORKLOADS["decode"], B=2, H=4, dk=d, dv=d, G=min(64, d), mean_bits=2.0,
                b_min=1, b_max=3)
    kc, oc = _cfgs(w, scope=scope)
    xs = W.tokens(w, 0, 16)
    st, _ = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    ws = K.new_workspace(kc)
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    base = W.base_rates(w)
    bad = tot = 0
    for t in range(16, 19):
        x = W.token(w, t, base=base)
        recs = dev(state_to_bytes(st, w.dk, w.dv, w.b_max))
        stg = _step_plain(kc, oc, recs, x, o, ws, st, f"narrow d={d} scope={scope} t={t}")
        st, o_or, _ = step.mirror_decode_step(st, x["q"], x["k"], x["v"], x["s"], x["beta"], oc)
        dc, n = _compare(stg, st, f"narrow d={d} scope={scope} t={t}")
        bad += dc
        tot += n
        og = host(o).reshape(o_or.shape)
        assert np.max(np.abs(og - o_or)) <= 1e-6 * np.max(np.abs(o_or))
    assert bad / tot <= 1e-5


def test_window_gamma_input_and_span1():
    w = W.WORKLOADS["tiny"]
    kc, oc = _cfgs(w, span=1)
    xs = W.tokens(w, 0, 8)
    st, _ = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    rng = np.random.default_rng(5)
    gamma = np.exp(rng.normal(0, 2, (w.B, w.H, w.dk)))
    x = W.token(w, 8)
    recs = dev(state_to_bytes(st, w.dk, w.dv, w.b_max))
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    stg = _step_plain(kc, oc, recs, x, o, K.new_workspace(kc), st, "gamma input", gamma=gamma)
    st2, _, _ = step.mirror_decode_step(st, x["q"], x["k"], x["v"], x["s"], x["beta"], oc, gamma=gamma)
    dc, n = _compare(stg, st2, "gamma input")
    assert dc == 0


def test_step_rejects_bad_config():
    w = W.WORKLOADS["tiny"]
    kc, _ = _cfgs(w)
    kc.mean_bits = 9.0
    with pytest.raises(K.KdaError):
        K.kda_step(kc, K.new_records(_cfgs(w)[0]), *[torch.zeros(1, device="cuda")] * 5,
                   torch.zeros(1, device="cuda"), K.new_workspace(_cfgs(w)[0]))


def test_split_phases_equal_step():
    """kda_step_outputs then kda_step_writeback (on another stream, after an
    event) leave the same records and outputs as kda_step."""
    w = W.sized(W.WORKLOADS["decode"], B=2)
    kc, oc = _cfgs(w)
    xs = W.tokens(w, 0, 12)
    st, _ = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    start = state_to_bytes(st, w.dk, w.dv, w.b_max)
    base = W.base_rates(w)
    recs_a, recs_b = dev(start), dev(start)
    ws_a, ws_b = K.new_workspace(kc), K.new_workspace(kc)
    o_a = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    o_b = torch.zeros_like(o_a)
    side = torch.cuda.Stream()
    for t in range(12, 15):
        x = {n: dev(a) for n, a in W.token(w, t, base=base).items()}
        K.kda_step(kc, recs_a, x["q"], x["k"], x["v"], x["s"], x["beta"], o_a, ws_a)
        K.kda_step_outputs(kc, recs_b, x["q"], x["k"], x["v"], x["s"], x["beta"], o_b, ws_b)
        ev = torch.cuda.Event()
        ev.record()
        side.wait_event(ev)
        with torch.cuda.stream(side):
            K.kda_step_writeback(kc, recs_b, ws_b)
        torch.cuda.current_stream().wait_stream(side)
        assert torch.equal(o_a, o_b)
    assert not meaningful_equal(host(recs_a), host(recs_b), w.B, w.H, w.dk, w.dv, w.b_max)
