"""Helpers shared by the GPU parity tests: host<->device copies and oracle
records in the library's byte layout.  Uses the oracle only on the CPU side."""
import sys

import numpy as np
import torch

from oracle import record, stats


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def say(*msg):
    print(*msg, flush=True)
    sys.stdout.flush()


def state_to_bytes(st, dk, dv, bmax):
    B, H = st["ntok"].shape
    slot = record.record_bytes(dk, dv, bmax)
    out = np.zeros((B, H, slot), np.uint8)
    for b in range(B):
        for h in range(H):
            out[b, h] = record.pack(st["ntok"][b, h], st["widths"][b, h], st["scale"][b, h],
                                    st["z"][b, h], st["r16"][b, h], st["codes"][b, h], dk, dv, bmax)
    return out.reshape(-1)


def bytes_to_state(buf, B, H, dk, dv, bmax):
    slot = record.record_bytes(dk, dv, bmax)
    buf = np.asarray(buf, np.uint8).reshape(B, H, slot)
    fs = [[record.unpack(buf[b, h], dk, dv, bmax) for h in range(H)] for b in range(B)]
    st = {k: np.stack([np.stack([fs[b][h][k] for h in range(H)]) for b in range(B)])
          for k in ("widths", "scale", "z", "r16", "codes")}
    st["ntok"] = np.array([[fs[b][h]["ntok"] for h in range(H)] for b in range(B)], np.int64)
    return st


def meaningful_equal(a, b, B, H, dk, dv, bmax):
    slot = record.record_bytes(dk, dv, bmax)
    a = np.asarray(a, np.uint8).reshape(B * H, slot)
    b = np.asarray(b, np.uint8).reshape(B * H, slot)
    bad = []
    for i in range(B * H):
        ma = record.meaningful(a[i], dk, dv, bmax)
        mb = record.meaningful(b[i], dk, dv, bmax)
        if ma.size != mb.size or not np.array_equal(ma, mb):
            bad.append(i)
    return bad


def _up256(x):
    return (x + 255) // 256 * 256


def ws_state32(ws, w):
    """float32 state after the last write-back interval, read from the
    workspace (views in the order the library lays them out: EMA keys,
    rate codes, widths, then the float32 state)."""
    rows = w.B * w.H * w.dk
    zr = _up256(rows * 8)
    bits = _up256(zr + rows * 4)
    s32 = _up256(bits + rows)
    a = host(ws[s32:s32 + rows * w.dv * 4]).view(np.float32)
    return a.reshape(w.B, w.H, w.dk, w.dv)


# ------------------------------------------- plain validity checks (GPU) ---
# The discrete outputs of a GPU write-back are checked against the plain
# definitions of oracle/plain.py on the GPU's own float32 state (the state
# the write-back quantised), independently of the float32 contract's
# evaluation order.

def ws_offsets(B, H, dk, dv):
    """Byte offsets of the workspace views the library lays out (see
    kda_workspace_bytes): keys, rate codes, widths, float32 state, per-slice
    row maxima, Gamma, the decode token vectors."""
    rows = B * H * dk
    zr = _up256(rows * 8)
    bits = _up256(zr + rows * 4)
    s32 = _up256(bits + rows)
    rpart = _up256(s32 + rows * dv * 4)
    gam = _up256(rpart + rows * (dv // 64) * 4)
    hv = _up256(gam + rows * 8)
    return dict(zr=zr, bits=bits, s32=s32, rpart=rpart, gam=gam, hv=hv)


def decode_state_gpu(kc, recs_before, ws, sel=None):
    """float32 state a decode step's write-back quantised, from the GPU's
    own values: d_k <= 128 hands the token's vectors a, g, w to the
    write-back, which forms S = fma(g_i, w_j, fl32(a_i x^_ij)) from the
    record's dequantised state x^ (decoded here by kda_unpack_state on a copy
    of the records taken before the step); d_k = 256 leaves S itself.
    sel: the sequences to return (all if None)."""
    import paper_2609_30950_amd as K
    from oracle.fp import fma32
    B, H, dk, dv = kc.B, kc.H, kc.d_k, kc.d_v
    off = ws_offsets(B, H, dk, dv)
    sel = list(range(B)) if sel is None else list(sel)
    if dk > 128:
        a = ws[off["s32"]:off["s32"] + B * H * dk * dv * 4].view(torch.float32)
        return host(a.view(B, H, dk, dv)[sel]).copy()
    X = torch.empty(B * H * dk * dv, dtype=torch.float32, device="cuda")
    K.kda_unpack_state(kc, recs_before, X)
    X = host(X.view(B, H * dk * dv)[sel]).reshape(-1, dk, dv)
    hv = ws[off["hv"]:off["hv"] + B * H * (dv + 2 * dk) * 4].view(torch.float32)
    hv = host(hv.view(B, H * (dv + 2 * dk))[sel]).reshape(-1, dv + 2 * dk)
    wv, a, g = hv[:, :dv], hv[:, dv:dv + dk], hv[:, dv + dk:]
    S = fma32(g[:, :, None], wv[:, None, :], (a[:, :, None] * X).astype(np.float32))
    return S.reshape(len(sel), H, dk, dv)


def decode_gamma(st_old, x, span, erase=True, mode="ema", C=1):
    """Row factors at a decode step's write-back: the EMAs continued from the
    old record's codes (or initialised by the token on a fresh state)."""
    dk = st_old["z"].shape[-1]
    s = np.asarray(x["s"], np.float32)
    s = np.broadcast_to(s, s.shape[:-1] + (dk,)) if s.shape[-1] != dk else s
    bt = np.asarray(x["beta"])[..., None]
    m0, e0 = stats.ema_from_record(st_old["z"], st_old["r16"])
    mu, eu = stats.ema_update(m0, e0, s, x["k"], bt, span, erase)
    mi, ei = stats.ema_init(s, x["k"], bt, erase)
    fresh = (np.asarray(st_old["ntok"]) == 0)[..., None]
    s_hat, r = stats.ema_rates(np.where(fresh, mi, mu), np.where(fresh, ei, eu))
    return stats.mode_gamma(s_hat, r, mode, C)


def prefill_gamma(st0, xs, C, span, erase=True, mode="ema"):
    """Row factors at the last write-back of a prefill from records st0 over
    tokens xs ([B, T, H, .]): the token-sequential EMAs, re-coded at every
    write-back before the last."""
    B, T, H, dk = np.asarray(xs["k"]).shape
    s_all = np.asarray(xs["s"], np.float32)
    m, e = stats.ema_from_record(st0["z"], st0["r16"])
    fresh = (np.asarray(st0["ntok"]) == 0)[..., None]
    for t in range(T):
        s = s_all[:, t]
        s = np.broadcast_to(s, s.shape[:-1] + (dk,)) if s.shape[-1] != dk else s
        bt = np.asarray(xs["beta"][:, t])[..., None]
        mi, ei = stats.ema_init(s, xs["k"][:, t], bt, erase)
        mu, eu = stats.ema_update(m, e, s, xs["k"][:, t], bt, span, erase)
        m, e = np.where(fresh, mi, mu), np.where(fresh, ei, eu)
        fresh = np.zeros_like(fresh)
        if (t + 1) % C == 0 or t == T - 1:
            s_hat, r = stats.ema_rates(m, e)
            if t == T - 1:
                return stats.mode_gamma(s_hat, r, mode, C)
            m, e = stats.ema_from_record(stats.logq_encode(s_hat), stats.r_encode(r))
    raise ValueError("no tokens")


def plain_check(S, gamma, st, *, G, scope, mean_bits, b_min, b_max, mode="ema", label=""):
    """Widths, scales and codes of decoded records st ([B, H, ...]) against
    the plain definitions, on the float32 state S [B, H, dk, dv] they
    quantise and row factors gamma [B, H, dk].  Prints the exempt counts;
    fails on any invalid decision.  gamma None: the widths are not checked
    (given widths, as in kda_pack_state)."""
    from oracle import plain
    S = np.asarray(S, np.float32)
    B, H, dk, dv = S.shape
    wex = 0
    if gamma is not None:
        R = np.max(np.abs(S), axis=-1)
        if G <= dk:
            c = plain.keys(gamma, R, G, mode)
        else:
            c = plain.keys(np.asarray(gamma).reshape(B, H * dk), R.reshape(B, H * dk), G,
                           mode).reshape(B, H, dk)
        units = [(b, slice(None)) for b in range(B)] if scope == 0 else \
            [(b, h) for b in range(B) for h in range(H)]
        for b, h in units:
            res = plain.check_widths(c[b, h], st["widths"][b, h], mean_bits, b_min, b_max)
            assert res["ok"], f"{label}: widths of unit {(b, h)} are not optimal ({res})"
            wex += res["exempt"]
    fit = plain.check_fit(S.reshape(-1, dv), np.asarray(st["widths"]).reshape(-1),
                          np.asarray(st["scale"]).reshape(-1),
                          np.asarray(st["codes"]).reshape(-1, dv))
    say(plain.summary(f"plain {label}", fit) + f" exempt_width_rows={wex}")
    assert fit["bad_scale"] == 0 and fit["bad_fit"] == 0 and fit["bad_codes"] == 0, \
        f"{label}: invalid rows {fit['bad_rows'][:8]}"
    return fit, wex


def plain_check_heads(S, gamma, st, *, mean_bits, b_min, b_max, label=""):
    """Head units: one width per head from the mean Gamma of its rows
    (fsum / d_k), optimal over the H heads of each sequence; every scale
    group (32 rows of one column) fitted and coded as a row of 32."""
    import math
    from oracle import plain
    S = np.asarray(S, np.float32)
    B, H, dk, dv = S.shape
    gamma = np.asarray(gamma, np.float64)
    ch = np.array([[math.fsum(gamma[b, h]) / dk for h in range(H)] for b in range(B)])
    wex = 0
    for b in range(B):
        res = plain.check_widths(ch[b], st["width"][b], mean_bits, b_min, b_max)
        assert res["ok"], f"{label}: head widths of sequence {b} are not optimal ({res})"
        wex += res["exempt"]
    tot = None
    for b in range(B):
        for h in range(H):
            g = S[b, h].reshape(dk // 32, 32, dv).transpose(0, 2, 1).reshape(-1, 32)
            cg = np.asarray(st["codes"][b, h]).reshape(dk // 32, 32, dv).transpose(0, 2, 1)
            fit = plain.check_fit(g, np.full(g.shape[0], int(st["width"][b, h])),
                                  np.asarray(st["bscale"][b, h]).reshape(-1), cg.reshape(-1, 32))
            if tot is None:
                tot = fit
            else:
                for k_ in fit:
                    tot[k_] = tot[k_] + fit[k_]
    say(plain.summary(f"plain {label}", tot) + f" exempt_width_heads={wex}")
    assert tot["bad_scale"] == 0 and tot["bad_fit"] == 0 and tot["bad_codes"] == 0, label
    return tot, wex


def state32_step_gpu(kc, X, x):
    """float32 state after one decode token from the state X [B, H, dk, dv],
    by the library's 32-bit mode (the same float32 recurrence as every
    quantised path): how a head-unit step's own state is obtained, since that
    kernel quantises in registers."""
    import dataclasses
    import paper_2609_30950_amd as K
    c32 = dataclasses.replace(kc, state32=1, head_units=0, scope=0, weight_mode=0,
                              group_rows=kc.d_k)
    recs = dev(np.ascontiguousarray(X, np.float32).reshape(-1).view(np.uint8))
    o = torch.zeros(kc.B * kc.H * kc.d_v, dtype=torch.float32, device="cuda")
    s = x["s"][..., 0] if kc.decay_per_head else x["s"]
    K.kda_step(c32, recs, dev(x["q"]), dev(x["k"]), dev(x["v"]), dev(s), dev(x["beta"]), o, None)
    return host(recs).view(np.float32).reshape(np.shape(X)).copy()
