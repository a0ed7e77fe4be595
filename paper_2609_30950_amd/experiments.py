"""Synthetic experiments of the paper run on the library's entry points.

    python -m paper_2609_30950_amd.experiments erase [--heads 64] [--window 512]
    python -m paper_2609_30950_amd.experiments readout [--heads 64] [--tokens 2048]
    python -m paper_2609_30950_amd.experiments rounding [--heads 8] [--tokens 2048]
    python -m paper_2609_30950_amd.experiments ablate [--heads 64] [--tokens 2048]

``erase``: the diagonal erase approximation against the exact Gramian
(Sec. 2, Approximate erasure rate: with per-channel rates log-uniform in
[1e-3, 1], allocation distortion differs from the exact-Gramian allocation
by at most 3 % with diverse keys and 17-23 % with persistent keys).  For
every head, per-channel rates are drawn log-uniform in [1e-3, 1] and kept
over a window of W tokens; queries are random unit vectors; beta =
sigmoid(N(0, 1)); keys are either fresh random unit vectors every token
("diverse") or one fixed random unit vector per head ("persistent").
kda_weights (diagonal approximation) and kda_weights_exact (full
transition) give the row weights over the window with a write-back after
every token; kda_alloc_bits allocates each at the per-head scope with unit
ranges (only decay and erasure enter); the allocation distortion of widths b
is the proxy sum_i Gamma_i^exact 2^(-2 b_i) under the exact weights, and the
result is its excess over the exact allocation's, per head.

``readout``: the EMA weight estimate against exact-Gramian allocation
(Sec. 3, State bit allocation: with log-normal gates and widths in [1, 8],
the estimate increases readout error by at most 2.5 % over exact-Gramian
allocation across the tested C).  Per head: d_k = d_v = 64, per-channel
rates with log s ~ N(log 0.03, 1.5^2) (clamped to [1e-4, 4]) kept over the
sequence, random unit q and k, v ~ N(0, 1), beta = sigmoid(N(0, 1)), bf16
inputs.  Three prefills of the same tokens with a write-back every C tokens:
the unquantised 32-bit mode (reference outputs), the quantised path with its
EMA weights, and the quantised path with the exact-Gramian weights of the
whole sequence (kda_weights_exact with the same write-back positions: the
inputs are stationary, so one set of weights per head serves every
write-back).  Readout error = sum_t |o_t - o_ref,t|^2 / sum_t |o_ref,t|^2
over all heads; the result is the EMA run's error over the exact run's, and
a fourth run with uniform widths gives the ablation baseline.

``ablate``: the allocation keys of the paper's ablation (Sec. 5, Table
ablate, where only the key c_i varies and excess NLL is measured) with the
readout error of a synthetic layer in place of NLL.  Inputs as ``readout``,
with the values of each head scaled by exp(N(0, 1)) so that heads differ in
range, and one layer budget over all heads (normalisation groups of one
head).  Keys: the EMA weights (ours), range alone, raw range, relative
range, DAMP's persistence w^(1), the write-back factor h^(C), erase rate 0,
uniform widths (the library's weight modes), and shuffled decay: the
stationary exact-Gramian weights of every head permuted across its rows,
given as row weights, beside the same weights unpermuted.  With C = 64 and
two bits the run is repeated with natural and with equal row ranges (keys
scaled so that the rows' steady-state magnitudes agree), our reading of the
two settings of Fig. 1d.  Two errors: the
absolute one over all heads, and the mean over heads of each head's error
relative to its own output power (the paper's range normalisation assumes
per-head output normalisation, which divides by that power).

``rounding``: correlated rounding errors at C = 1 (Sec. 2, Correlated rounding
errors: with Kimi decays, rank-one writes and 2K tokens, lag-one error
correlations reach 0.23 for s <= 1e-3 at three to five bits, and the readout
error is 0.17-2.4 times that of independent noise of variance Delta^2/12).
Per head: d_k = d_v = 64, rates log-uniform in [1e-3, 1] per channel with
10 % of the channels in [1e-4, 1e-3), writes v_t = xi_t u with a fixed unit
u per head (rank one), random unit q, random unit k or one fixed unit k per
head (keys "fixed": the whole write k v^T keeps its direction), beta =
sigmoid(N(0, 1)); decode
steps on the GPU (kda_step, per-head budget, widths [1, 8]).  After every
step the dequantised state is read back (kda_unpack_state) and the step's
unquantised update is recomputed on the host in float64 from the previous
dequantised state, which gives the step's exact quantisation error.  Two
host trajectories run beside it: the unquantised recurrence (reference
outputs) and one that adds independent uniform noise of the GPU's per-row
step sizes after every token.  Reported: the lag-one correlation of the
quantisation errors of the slow rows, and the ratio of the quantised
outputs' error to the independent-noise outputs' error.

Inputs are drawn with numpy from a fixed seed; everything else runs on the
GPU through the C ABI.
"""
import argparse
import json

import numpy as np
import torch

from . import api


def _unit(x):
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def erase_inputs(heads, window, dk, keys, seed=0, beta_mode="sigmoid"):
    """q, s, beta, k of a window for `heads` heads as [1][W][H][.] arrays
    (beta = sigmoid(N(0, 1)), or 1/2 as in the paper's fixed-key example)."""
    rng = np.random.default_rng([seed, 7])
    s = np.exp(rng.uniform(np.log(1e-3), np.log(1.0), (1, 1, heads, dk)))
    s = np.broadcast_to(s, (1, window, heads, dk))
    q = _unit(rng.standard_normal((1, window, heads, dk)))
    beta = 1.0 / (1.0 + np.exp(-rng.standard_normal((1, window, heads))))
    if beta_mode == "half":
        beta = np.full_like(beta, 0.5)
    if keys == "persistent":
        k = np.broadcast_to(_unit(rng.standard_normal((1, 1, heads, dk))), (1, window, heads, dk))
    else:
        k = _unit(rng.standard_normal((1, window, heads, dk)))
    f = lambda a: np.ascontiguousarray(a, np.float32)
    return f(q), f(s), f(beta), f(k)


def erase_approximation(heads=64, window=512, dk=128, mean_bits=2.0, keys="diverse", seed=0,
                        beta_mode="sigmoid"):
    """Per-head excess allocation distortion of the diagonal erase
    approximation over the exact-Gramian allocation."""
    cfg = api.Config(B=1, H=heads, d_k=dk, d_v=dk, group_rows=dk, scope=1, mean_bits=mean_bits,
                     b_min=1, b_max=8)
    q, s, beta, k = (torch.from_numpy(a).cuda()
                     for a in erase_inputs(heads, window, dk, keys, seed, beta_mode))
    g_apx = torch.zeros(heads * dk, dtype=torch.float64, device="cuda")
    g_ex = torch.zeros_like(g_apx)
    api.kda_weights(cfg, window, 1, q, s, beta, k, g_apx)
    api.kda_weights_exact(cfg, window, 1, q, s, beta, k, g_ex)
    ones = torch.ones(heads * dk, dtype=torch.float32, device="cuda")
    ws = api.new_workspace(cfg)
    b_apx = torch.zeros(heads * dk, dtype=torch.uint8, device="cuda")
    b_ex = torch.zeros_like(b_apx)
    api.kda_alloc_bits(cfg, g_apx, ones, b_apx, ws)
    api.kda_alloc_bits(cfg, g_ex, ones, b_ex, ws)
    torch.cuda.synchronize()
    ge = g_ex.cpu().numpy().reshape(heads, dk)
    ba = b_apx.cpu().numpy().reshape(heads, dk).astype(np.float64)
    be = b_ex.cpu().numpy().reshape(heads, dk).astype(np.float64)
    d_apx = np.sum(ge * np.exp2(-2 * ba), axis=1)
    d_ex = np.sum(ge * np.exp2(-2 * be), axis=1)
    return d_apx / d_ex - 1.0


def readout_inputs(heads, tokens, dk, seed=0):
    rng = np.random.default_rng([seed, 11])
    ls = rng.normal(np.log(0.03), 1.5, (1, 1, heads, dk))
    s = np.broadcast_to(np.clip(np.exp(ls), 1e-4, 4.0), (1, tokens, heads, dk))
    q = _unit(rng.standard_normal((1, tokens, heads, dk)))
    k = _unit(rng.standard_normal((1, tokens, heads, dk)))
    v = rng.standard_normal((1, tokens, heads, dk))
    beta = 1.0 / (1.0 + np.exp(-rng.standard_normal((1, tokens, heads))))
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16)
    qb, kb, vb = bf(q), bf(k), bf(v)
    f = lambda a: np.ascontiguousarray(a, np.float32)
    return qb, kb, vb, f(s), f(beta)


def readout_error(heads=64, tokens=2048, C=16, mean_bits=3.0, dk=64, seed=0):
    """Readout errors with the EMA weights, the exact-Gramian weights and
    uniform widths (the ablation baseline, KDA_WEIGHT_UNIFORM)."""
    qb, kb, vb, s, beta = readout_inputs(heads, tokens, dk, seed)
    q, k, v = qb.cuda(), kb.cuda(), vb.cuda()
    sd, bd = torch.from_numpy(s).cuda(), torch.from_numpy(beta).cuda()
    base = dict(B=1, H=heads, d_k=dk, d_v=dk, group_rows=dk, scope=1, mean_bits=mean_bits,
                b_min=1, b_max=8)

    def run(cfg, gamma=None):
        recs = api.new_records(cfg)
        o = torch.zeros(tokens * heads * dk, dtype=torch.float32, device="cuda")
        ws = None if cfg.state32 else api.new_workspace(cfg)
        api.kda_prefill(cfg, tokens, C, recs, q, k, v, sd, bd, o, ws, gamma=gamma)
        return o

    o_ref = run(api.Config(state32=1, **base))
    cfg = api.Config(**base)
    o_ema = run(cfg)
    gam = torch.zeros(heads * dk, dtype=torch.float64, device="cuda")
    api.kda_weights_exact(cfg, tokens, C, qb.float().cuda(), sd, bd, kb.float().cuda(), gam)
    o_ex = run(cfg, gamma=gam)
    o_uni = run(api.Config(weight_mode=api.WEIGHT_MODES.index("uniform"), **base))
    ref2 = float(torch.sum(o_ref.double() ** 2))
    err = lambda o: float(torch.sum((o.double() - o_ref.double()) ** 2)) / ref2
    return err(o_ema), err(o_ex), err(o_uni)


def ablation(heads=64, tokens=2048, C=16, mean_bits=2.0, dk=64, seed=0, ranges="natural"):
    """Readout errors (against the 32-bit mode) of every allocation key of the
    ablation on one synthetic layer: {key: {"abs": e, "norm": e_head}}, plus
    "range_spread": the standard deviation of log row ranges within a head
    of the final unquantised state (median over heads).  ranges="equal"
    scales key channel i by sqrt(1 - exp(-2 s_i)), which evens out the rows'
    steady-state magnitudes 1/sqrt(1 - exp(-2 s_i)), so that decay is the
    only thing that tells rows apart."""
    qb, kb, vb, s, beta = readout_inputs(heads, tokens, dk, seed)
    if ranges == "equal":
        g = np.sqrt(-np.expm1(-2.0 * s[:, :1].astype(np.float64)))
        g = g / np.sqrt(np.mean(g * g, axis=-1, keepdims=True))
        kb = (kb.float() * torch.from_numpy(g.astype(np.float32))).to(torch.bfloat16)
    else:
        assert ranges == "natural", ranges
    rng = np.random.default_rng([seed, 13])
    scale = np.exp(rng.standard_normal(heads)).astype(np.float32)
    vb = (vb.float() * torch.from_numpy(scale)[None, None, :, None]).to(torch.bfloat16)
    q, k, v = qb.cuda(), kb.cuda(), vb.cuda()
    sd, bd = torch.from_numpy(s).cuda(), torch.from_numpy(beta).cuda()
    base = dict(B=1, H=heads, d_k=dk, d_v=dk, group_rows=dk, scope=0, mean_bits=mean_bits,
                b_min=1, b_max=8)

    state = {}

    def run(cfg, gamma=None):
        recs = api.new_records(cfg)
        o = torch.zeros(tokens * heads * dk, dtype=torch.float32, device="cuda")
        ws = None if cfg.state32 else api.new_workspace(cfg)
        api.kda_prefill(cfg, tokens, C, recs, q, k, v, sd, bd, o, ws, gamma=gamma)
        if cfg.state32:
            state["S"] = recs.view(torch.float32).view(heads, dk, dk).double()
        return o

    o_ref = run(api.Config(state32=1, **base))
    R = torch.amax(torch.abs(state["S"]), dim=2)
    spread = float(torch.median(torch.std(torch.log(R), dim=1)))
    ref2 = float(torch.sum(o_ref.double() ** 2))
    ref_h = torch.sum(o_ref.double().view(tokens, heads, dk) ** 2, dim=(0, 2))

    def err(o):
        d2 = (o.double() - o_ref.double()) ** 2
        # absolute readout error, and the mean over heads of each head's error
        # relative to its own output power (what a per-head output norm sees)
        return dict(abs=float(torch.sum(d2)) / ref2,
                    norm=float(torch.mean(torch.sum(d2.view(tokens, heads, dk), dim=(0, 2)) / ref_h)))

    out = {}
    for mode in api.WEIGHT_MODES:
        out[mode] = err(run(api.Config(weight_mode=api.WEIGHT_MODES.index(mode), **base)))
    cfg = api.Config(**base)
    gam = torch.zeros(heads * dk, dtype=torch.float64, device="cuda")
    api.kda_weights_exact(cfg, tokens, C, qb.float().cuda(), sd, bd, kb.float().cuda(), gam)
    out["exact"] = err(run(cfg, gamma=gam))
    perm = np.argsort(rng.random((heads, dk)), axis=1) + np.arange(heads)[:, None] * dk
    shuffled = gam[torch.from_numpy(perm.reshape(-1)).cuda()].contiguous()
    out["shuffled_exact"] = err(run(cfg, gamma=shuffled))
    out["range_spread"] = spread
    return out


def _host_step(S, q, k, v, s, beta):
    """eq. rule in float64 for a reference trajectory: S [H, dk, dv]; q, k, s
    [H, dk]; v [H, dv]; beta [H].  Returns (S, o)."""
    Sd = np.exp(-s)[:, :, None] * S
    u = np.einsum("hi,hij->hj", k, Sd)
    S = Sd + (beta[:, None] * k)[:, :, None] * (v - u)[:, None, :]
    return S, np.einsum("hi,hij->hj", q, S)


def correlated_rounding(bits=4, heads=8, tokens=2048, dk=64, seed=0, keys="random"):
    """Lag-one correlation of the quantisation errors of the slow rows (mean
    over their elements, and the largest row mean) and the ratio of the
    quantised outputs' error to the independent-noise outputs' error."""
    rng = np.random.default_rng([seed, 13])
    s = np.exp(rng.uniform(np.log(1e-3), 0.0, (heads, dk)))
    slow = rng.random((heads, dk)) < 0.1
    s[slow] = np.exp(rng.uniform(np.log(1e-4), np.log(1e-3), slow.sum()))
    s = s.astype(np.float32).astype(np.float64)
    u_dir = _unit(rng.standard_normal((heads, dk)))
    k_fix = _unit(rng.standard_normal((heads, dk))).astype(np.float32)
    cfg = api.Config(B=1, H=heads, d_k=dk, d_v=dk, group_rows=dk, scope=1, mean_bits=bits,
                     b_min=1, b_max=8)
    slot = api.record_bytes(cfg)
    sc_off = 16 + dk // 2                      # FP16 row scales of the record layout
    recs = api.new_records(cfg)
    ws = api.new_workspace(cfg)
    o = torch.zeros(heads * dk, dtype=torch.float32, device="cuda")
    Sg = torch.zeros(heads * dk * dk, dtype=torch.float32, device="cuda")
    bits_g = torch.zeros(heads * dk, dtype=torch.uint8, device="cuda")
    sd = torch.from_numpy(s.astype(np.float32)).cuda()
    S_hat = np.zeros((heads, dk, dk))          # the GPU's dequantised state
    S_ref = np.zeros((heads, dk, dk))          # unquantised reference
    S_ind = np.zeros((heads, dk, dk))          # independent-noise trajectory
    prev_e = None
    acc = np.zeros((5, heads, dk, dk))          # sums of e, e', e e', e^2, e'^2
    n_pairs = 0
    err_det = err_ind = ref2 = 0.0
    for t in range(tokens):
        q = _unit(rng.standard_normal((heads, dk))).astype(np.float32)
        k = _unit(rng.standard_normal((heads, dk))).astype(np.float32)
        if keys == "fixed":
            k = k_fix
        v = (rng.standard_normal((heads, 1)) * u_dir).astype(np.float32)
        beta = (1.0 / (1.0 + np.exp(-rng.standard_normal(heads)))).astype(np.float32)
        dq, dk_, dv, db = (torch.from_numpy(a).cuda() for a in (q, k, v, beta))
        api.kda_step(cfg, recs, dq, dk_, dv, sd, db, o, ws)
        api.kda_unpack_state(cfg, recs, Sg, bits_g)
        q64, k64, v64, b64 = (a.astype(np.float64) for a in (q, k, v, beta))
        S_pre, _ = _host_step(S_hat, q64, k64, v64, s, b64)
        S_hat = Sg.cpu().numpy().reshape(heads, dk, dk).astype(np.float64)
        e = S_hat - S_pre
        if prev_e is not None:
            acc += np.stack([e, prev_e, e * prev_e, e * e, prev_e * prev_e])
            n_pairs += 1
        prev_e = e
        S_ref, o_ref = _host_step(S_ref, q64, k64, v64, s, b64)
        rec = recs.cpu().numpy().reshape(heads, slot)
        wid = bits_g.cpu().numpy().reshape(heads, dk).astype(np.int64)
        sc = rec[:, sc_off:sc_off + 2 * dk].copy().view(np.float16).astype(np.float64)
        step = np.where(wid >= 2, sc, 2.0 * sc)          # one-bit rows: levels +-mu
        X_pre, o_ind = _host_step(S_ind, q64, k64, v64, s, b64)
        S_ind = X_pre + rng.uniform(-0.5, 0.5, X_pre.shape) * step[:, :, None]
        o_det = o.cpu().numpy().reshape(heads, dk).astype(np.float64)
        err_det += float(np.sum((o_det - o_ref) ** 2))
        err_ind += float(np.sum((o_ind - o_ref) ** 2))
        ref2 += float(np.sum(o_ref ** 2))
    m = acc / n_pairs
    cov = m[2] - m[0] * m[1]
    var = np.sqrt(np.maximum(m[3] - m[0] ** 2, 0) * np.maximum(m[4] - m[1] ** 2, 0))
    corr = np.where(var > 0, cov / np.where(var > 0, var, 1.0), 0.0)
    row_corr = corr.mean(axis=2)                      # [heads, dk]
    return dict(lag1_slow_mean=float(row_corr[slow].mean()),
                lag1_slow_max_row=float(row_corr[slow].max()),
                lag1_fast_mean=float(row_corr[~slow].mean()),
                readout_ratio=err_det / err_ind,
                readout_error_quantised=err_det / ref2, readout_error_independent=err_ind / ref2)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("experiment", choices=["erase", "readout", "rounding", "ablate"])
    ap.add_argument("--heads", type=int, default=64)
    ap.add_argument("--window", type=int, default=512)
    ap.add_argument("--tokens", type=int, default=2048)
    args = ap.parse_args()
    out = {}
    if args.experiment == "rounding":
        for keys in ("random", "fixed"):
            for bits in (3, 4, 5, 6):
                out[f"{keys} keys, {bits} bits"] = correlated_rounding(
                    bits, args.heads if args.heads != 64 else 8, args.tokens, keys=keys)
        print(json.dumps(out, indent=1))
        return
    if args.experiment == "ablate":
        for C, mean in ((1, 4.0), (16, 2.0), (64, 2.0)):
            out[f"C={C}, mean {mean:g} bits"] = ablation(args.heads, args.tokens, C, mean)
        for rg in ("natural", "equal"):   # the two settings of Fig. 1d: C = 64, two bits
            out[f"C=64, mean 2 bits, {rg} row ranges"] = ablation(args.heads, args.tokens, 64, 2.0,
                                                                  ranges=rg)
        print(json.dumps(out, indent=1))
        return
    if args.experiment == "readout":
        for C in (1, 16, 64):
            for mean in (2.0, 4.0):
                e_ema, e_ex, e_uni = readout_error(args.heads, args.tokens, C, mean)
                out[f"C={C}, mean {mean:g} bits"] = dict(ema=e_ema, exact=e_ex, uniform=e_uni,
                                                         excess=e_ema / e_ex - 1.0)
        print(json.dumps(out, indent=1))
        return
    for keys, bm in (("diverse", "sigmoid"), ("persistent", "sigmoid"), ("diverse", "half"),
                     ("persistent", "half")):
        for mean in (2.0, 4.0):
            ex = erase_approximation(args.heads, args.window, 128, mean, keys, 0, bm)
            out[f"{keys} keys, beta {bm}, mean {mean:g} bits"] = dict(
                mean_excess=float(np.mean(ex)), max_excess=float(np.max(ex)),
                median_excess=float(np.median(ex)))
    print(json.dumps(out, indent=1))


if __name__ == "__main__":
    main()
