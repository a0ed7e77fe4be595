"""GPU parity of the allocation-key variants (Sec. 5, Table ablate): decode
steps for every mode, prefill with the write-back factor h^(C) (which depends
on the write-back interval) on the token-sequential and the chunked path, and
head units with the modes that need no ranges.  Records are compared with the
oracle bit for bit (rate codes up to one last-bit transcendental difference)."""
import numpy as np
import pytest
import torch

import paper_2609_30950_amd as K
import workloads as W
from oracle import record, step
from tests._gpu import (bytes_to_state, decode_gamma, decode_state_gpu, dev, host, plain_check,
                        prefill_gamma, say, state_to_bytes, ws_state32)

pytestmark = pytest.mark.gpu

MODES = K.api.WEIGHT_MODES


def _cfgs(w, mode, **kw):
    kc = K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.G, mean_bits=w.mean_bits,
                  b_min=w.b_min, b_max=w.b_max, decay_per_head=int(w.decay == "head"),
                  weight_mode=MODES.index(mode), **kw)
    oc = step.Cfg(dk=w.dk, dv=w.dv, G=w.G, mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max,
                  weight=mode)
    return kc, oc


def _check(stg, st, label):
    same_w = stg["widths"] == st["widths"]
    dc = int(np.sum((stg["codes"] != st["codes"]) & same_w[..., None])) + \
        int(np.sum(~same_w)) * stg["codes"].shape[-1]
    say(f"{label}: widths {int(np.sum(~same_w))} codes {dc} of {stg['codes'].size}")
    assert np.array_equal(stg["ntok"], st["ntok"])
    assert np.array_equal(stg["widths"], st["widths"])
    assert np.array_equal(stg["scale"].view(np.uint16), st["scale"].view(np.uint16))
    assert int(np.sum(stg["z"] != st["z"])) <= 1
    assert dc / stg["codes"].size <= 1e-5


@pytest.mark.parametrize("mode", MODES)
def test_decode_steps_every_mode(mode):
    w = W.sized(W.WORKLOADS["tiny"], B=2, H=4, mean_bits=3.5)
    kc, oc = _cfgs(w, mode)
    xs = W.tokens(w, 0, 12)
    st, _ = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    ws = K.new_workspace(kc)
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    base = W.base_rates(w)
    for t in range(12, 14):
        x = W.token(w, t, base=base)
        recs = dev(state_to_bytes(st, w.dk, w.dv, w.b_max))
        before = recs.clone()
        K.kda_step(kc, recs, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(x["s"]), dev(x["beta"]),
                   o, ws)
        plain_check(decode_state_gpu(kc, before, ws), decode_gamma(st, x, oc.span, mode=mode),
                    bytes_to_state(host(recs), w.B, w.H, w.dk, w.dv, w.b_max), G=w.G, scope=0,
                    mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max, mode=mode,
                    label=f"{mode} t={t}")
        st, o_or, _ = step.mirror_decode_step(st, x["q"], x["k"], x["v"], x["s"], x["beta"], oc)
        _check(bytes_to_state(host(recs), w.B, w.H, w.dk, w.dv, w.b_max), st, f"{mode} t={t}")
    if mode == "uniform":
        assert np.all(np.ptp(st["widths"].reshape(w.B, -1), axis=1) <= 1)


def _bf(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(torch.bfloat16).cuda()


def test_prefill_write_back_factor():
    w = W.sized(W.WORKLOADS["tiny"], B=1, H=2, T=40, bf16=True, mean_bits=3.0)
    kc, oc = _cfgs(w, "writeback")
    xs = W.tokens(w, 0, 40)
    st0 = step.zero_state(w.B, w.H, oc)
    recs = dev(state_to_bytes(st0, w.dk, w.dv, w.b_max))
    o = torch.zeros(w.B * 40 * w.H * w.dv, dtype=torch.float32, device="cuda")
    ws = K.new_workspace(kc)
    K.kda_prefill(kc, 40, 16, recs, _bf(xs["q"]), _bf(xs["k"]), _bf(xs["v"]), dev(xs["s"]),
                  dev(xs["beta"]), o, ws)
    st, _, _ = step.mirror_prefill(st0, xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], 16, oc)
    plain_check(ws_state32(ws, w), prefill_gamma(st0, xs, 16, oc.span, mode="writeback"),
                bytes_to_state(host(recs), w.B, w.H, w.dk, w.dv, w.b_max), G=w.G, scope=0,
                mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max, mode="writeback",
                label="prefill h^(16)")
    _check(bytes_to_state(host(recs), w.B, w.H, w.dk, w.dv, w.b_max), st, "prefill h^(16)")


def test_chunked_prefill_write_back_factor():
    """One 48-token interval on the chunked path: its write-back is the
    oracle's quantiser on the GPU's own float32 state with h^(48)."""
    w = W.sized(W.WORKLOADS["tiny"], B=1, H=2, bf16=True, mean_bits=3.0)
    kc, oc = _cfgs(w, "writeback", chunked=1)
    warm = W.tokens(w, 0, 16)
    st0, _ = step.warm_state(warm["q"], warm["k"], warm["v"], warm["s"], warm["beta"], oc)
    xs = W.tokens(w, 16, 64)
    T = 48
    recs = dev(state_to_bytes(st0, w.dk, w.dv, w.b_max))
    o = torch.zeros(w.B * T * w.H * w.dv, dtype=torch.float32, device="cuda")
    ws = K.new_workspace(kc)
    K.kda_prefill(kc, T, 48, recs, _bf(xs["q"]), _bf(xs["k"]), _bf(xs["v"]), dev(xs["s"]),
                  dev(xs["beta"]), o, ws)
    rows = w.B * w.H * w.dk
    up = lambda x: (x + 255) // 256 * 256
    off = up(up(up(rows * 8) + rows * 4) + rows)
    Sg = host(ws)[off:off + rows * w.dv * 4].view(np.float32).reshape(w.B, w.H, w.dk, w.dv)
    m, e = step.ema_start(st0)
    for t in range(T):
        sr = xs["s"][:, t]
        bt = np.asarray(xs["beta"][:, t])[..., None]
        from oracle import stats
        m, e = stats.ema_update(m, e, sr, xs["k"][:, t], bt, oc.span)
    exp, _ = step.write_back(Sg, m, e, st0["ntok"] + T, oc, C=48)
    _check(bytes_to_state(host(recs), w.B, w.H, w.dk, w.dv, w.b_max), exp, "chunked h^(48)")


@pytest.mark.parametrize("mode", ["persist", "writeback", "no_erase_rate", "uniform", "decay"])
def test_head_units_modes(mode):
    w = W.sized(W.WORKLOADS["gdn2"], B=1, H=8, dk=64, dv=64, G=64, mean_bits=3.5, b_min=2)
    kc, oc = _cfgs(w, mode, head_units=1)
    oc.unit = "head"
    xs = W.tokens(w, 0, 6)
    st, _ = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    x = W.token(w, 6, base=W.base_rates(w))
    buf = np.concatenate([record.pack_heads(st["ntok"][0, h], st["width"][0, h], st["bscale"][0, h],
                                            st["z"][0, h], st["r16"][0, h], st["codes"][0, h],
                                            64, 64, w.b_max) for h in range(w.H)])
    recs = dev(buf)
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    K.kda_step(kc, recs, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(x["s"][..., 0]),
               dev(x["beta"]), o, K.new_workspace(kc))
    st, _, _ = step.mirror_decode_step(st, x["q"], x["k"], x["v"], x["s"], x["beta"], oc)
    slot = record.record_bytes_heads(64, 64, w.b_max)
    got = host(recs).reshape(w.H, slot)
    for h in range(w.H):
        f = record.unpack_heads(got[h], 64, 64, w.b_max)
        assert f["width"] == st["width"][0, h]
        assert np.array_equal(f["codes"], st["codes"][0, h])
        assert np.array_equal(f["bscale"].view(np.uint16), st["bscale"][0, h].view(np.uint16))
    say(f"heads {mode}: widths {st['width'].ravel().tolist()}")
