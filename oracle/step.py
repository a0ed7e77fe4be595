"""Decode step and chunked prefill with quantised write-backs (Sec. 2-3, Protocol).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Protocol (Sec. 2, Accumulated readout error; Sec. 5, Protocol): the state is
float32 between write-backs; outputs are read from the unquantised state
(outputs precede quantisation); a write-back follows every C-th token (and the
last token of a prefill) and replaces the state by Deq(Q(S)) with no residual.
A decode step is C = 1.

At a write-back, per sequence:
  1. s_hat, r from the token-sequential EMAs; Gamma^ (eq. weight), or a given
     window Gramian;
  2. R_i = max_j |S_ij|; R~ within groups of G rows; c_i = Gamma_i R~_i^2;
  3. widths from the budget over the allocation scope (all H*dk rows of the
     sequence, or one head);
  4. per-row fitted quantiser; the rates are stored as a 16-bit log code and
     the erase rate as FP16; the EMAs continue from the decoded values.

Head units (Cfg.unit = "head", Sec. 3, Allocation units: Gated DeltaNet with
per-head decay and normalisation): R~ = 1, each head's key is the mean Gamma
of its rows, one width per head from the layer budget over the H heads, and
the block quantiser (scales per 32 rows of a column).

State is handled as a dict of decoded record fields with a leading [B, H]
(see ``record.py`` for the bytes).  ``mirror_*`` use the float32 contract of
``recurrence.mirror_step``; ``truth_outputs`` gives float64 outputs from the
same starting state for accuracy checks.
"""
from dataclasses import dataclass

import numpy as np

from . import alloc, quant, recurrence, stats

F32 = np.float32
F64 = np.float64


@dataclass
class Cfg:
    dk: int
    dv: int
    G: int = 64
    scope: str = "sequence"          # "sequence" (layer budget) or "head"
    mean_bits: float = 4.0
    b_min: int = 2
    b_max: int = 8
    span: int = 64
    erase: bool = True              # False: no erasure (Mamba-2)
    unit: str = "row"               # "row" (a width per row) or "head" (block scales)
    weight: str = "ema"             # allocation key variant (stats.WEIGHT_MODES)


def zero_state(B, H, cfg):
    if cfg.unit == "head":
        return dict(ntok=np.zeros((B, H), np.int64), width=np.zeros((B, H), np.int64),
                    bscale=np.zeros((B, H, cfg.dk // quant.BLOCK, cfg.dv), np.float16),
                    z=np.zeros((B, H, cfg.dk), np.uint16),
                    r16=np.zeros((B, H, cfg.dk), np.float16),
                    codes=np.zeros((B, H, cfg.dk, cfg.dv), np.int64))
    return dict(ntok=np.zeros((B, H), np.int64),
                widths=np.ones((B, H, cfg.dk), np.int64),
                scale=np.zeros((B, H, cfg.dk), np.float16),
                z=np.zeros((B, H, cfg.dk), np.uint16),
                r16=np.zeros((B, H, cfg.dk), np.float16),
                codes=np.zeros((B, H, cfg.dk, cfg.dv), np.int64))


def dequantize(state):
    if "bscale" in state:
        return quant.dequantize_blocks(state["codes"], state["bscale"])
    B, H, dk, dv = state["codes"].shape
    x = quant.dequantize_rows(state["codes"].reshape(-1, dv),
                              state["scale"].reshape(-1),
                              state["widths"].reshape(-1))
    return x.reshape(B, H, dk, dv)


def ema_start(state):
    return stats.ema_from_record(state["z"], state["r16"])


def _rows(s, dk):
    s = np.asarray(s, F32)
    return np.broadcast_to(s, s.shape[:-1] + (dk,)) if s.shape[-1] == 1 else s


def allocate_widths(c, cfg):
    B, H, dk = c.shape
    if cfg.scope == "sequence":
        return np.stack([alloc.allocate(c[b].reshape(-1), cfg.mean_bits, cfg.b_min,
                                        cfg.b_max).reshape(H, dk) for b in range(B)])
    out = np.empty((B, H, dk), np.int64)
    for b in range(B):
        for h in range(H):
            out[b, h] = alloc.allocate(c[b, h], cfg.mean_bits, cfg.b_min, cfg.b_max)
    return out


def write_back_heads(S, m, e, ntok, cfg, gamma=None, C=1):
    """Head units: one width per head from the mean Gamma of its rows, block
    scales.  Same arguments and results as write_back."""
    B, H, dk, dv = S.shape
    s_hat, r = stats.ema_rates(m, e)
    g = (stats.mode_gamma(s_hat, r, cfg.weight, C) if gamma is None
         else np.asarray(gamma, F64))
    ch = alloc.head_weights(g)
    width = np.stack([alloc.allocate(ch[b], cfg.mean_bits, cfg.b_min, cfg.b_max)
                      for b in range(B)])
    codes = np.zeros((B, H, dk, dv), np.int64)
    bscale = np.zeros((B, H, dk // quant.BLOCK, dv), np.float16)
    mstar = np.zeros((B, H, dk // quant.BLOCK, dv), np.int64)
    for b in range(B):
        for h in range(H):
            c, sc, ms = quant.quantize_blocks(S[b, h], int(width[b, h]))
            codes[b, h], bscale[b, h], mstar[b, h] = c, sc, ms
    state = dict(ntok=np.asarray(ntok, np.int64), width=width, bscale=bscale,
                 z=stats.logq_encode(s_hat), r16=stats.r_encode(r), codes=codes)
    diag = dict(S=S, c=ch, gamma=g, s_hat=s_hat, r=r, mstar=mstar)
    return state, diag


def write_back(S, m, e, ntok, cfg, gamma=None, C=1):
    """Quantise float32 S [B,H,dk,dv] with EMA states m, e -> (state, diag).
    C is the write-back interval (used by the "writeback" weight variant)."""
    if cfg.unit == "head":
        return write_back_heads(S, m, e, ntok, cfg, gamma, C)
    B, H, dk, dv = S.shape
    s_hat, r = stats.ema_rates(m, e)
    g = (stats.mode_gamma(s_hat, r, cfg.weight, C) if gamma is None
         else np.asarray(gamma, F64))
    R = np.max(np.abs(S), axis=-1).astype(F32)
    if cfg.G <= dk:
        Rt = alloc.normalized_ranges(R, cfg.G)
    else:
        # groups of G rows across consecutive heads of a sequence
        Rt = alloc.normalized_ranges(R.reshape(B, H * dk), cfg.G).reshape(B, H, dk)
    c = alloc.mode_weights(g, R, Rt, cfg.weight)
    widths = allocate_widths(c, cfg)
    codes, scale, mstar = quant.quantize_rows(S.reshape(-1, dv), widths.reshape(-1))
    state = dict(ntok=np.asarray(ntok, np.int64), widths=widths,
                 scale=scale.reshape(B, H, dk), z=stats.logq_encode(s_hat),
                 r16=stats.r_encode(r), codes=codes.reshape(B, H, dk, dv).astype(np.int64))
    diag = dict(S=S, R=R, c=c, gamma=g, s_hat=s_hat, r=r, mstar=mstar.reshape(B, H, dk))
    return state, diag


def mirror_decode_step(state, q, k, v, s, beta, cfg, gamma=None):
    """One token for B x H heads.  q, k: [B,H,dk]; v: [B,H,dv]; s: [B,H,dk]
    or [B,H,1]; beta: [B,H].  Returns (new state, o [B,H,dv], diag)."""
    X = dequantize(state)
    S, o = recurrence.mirror_step(X, q, k, v, s, beta, cfg.erase)
    sr = _rows(s, cfg.dk)
    m0, e0 = ema_start(state)
    mi, ei = stats.ema_init(sr, k, np.asarray(beta)[..., None], cfg.erase)
    mu, eu = stats.ema_update(m0, e0, sr, k, np.asarray(beta)[..., None], cfg.span, cfg.erase)
    fresh = (state["ntok"] == 0)[..., None]
    m = np.where(fresh, mi, mu)
    e = np.where(fresh, ei, eu)
    new, diag = write_back(S, m, e, state["ntok"] + 1, cfg, gamma)
    diag["X"] = X
    return new, o, diag


def mirror_prefill(state, q, k, v, s, beta, C, cfg, gamma=None):
    """T tokens.  q, k: [B,T,H,dk]; v: [B,T,H,dv]; s: [B,T,H,dk|1];
    beta: [B,T,H].  Write-back after every C-th token and after the last.
    Returns (state, o [B,T,H,dv], list of per-write-back diagnostics)."""
    B, T, H, _ = np.asarray(q).shape
    X = dequantize(state)
    m, e = ema_start(state)
    ntok = state["ntok"].copy()
    fresh = ntok == 0
    o_all = np.zeros((B, T, H, cfg.dv), F32)
    diags = []
    since = 0
    for t in range(T):
        X, o = recurrence.mirror_step(X, q[:, t], k[:, t], v[:, t], s[:, t], beta[:, t], cfg.erase)
        o_all[:, t] = o
        sr = _rows(s[:, t], cfg.dk)
        bt = np.asarray(beta[:, t])[..., None]
        mi, ei = stats.ema_init(sr, k[:, t], bt, cfg.erase)
        mu, eu = stats.ema_update(m, e, sr, k[:, t], bt, cfg.span, cfg.erase)
        m = np.where(fresh[..., None], mi, mu)
        e = np.where(fresh[..., None], ei, eu)
        fresh = np.zeros_like(fresh)
        since += 1
        if (t + 1) % C == 0 or t == T - 1:
            ntok = ntok + since
            since = 0
            state, diag = write_back(X, m, e, ntok, cfg, gamma, C)
            diags.append(diag)
            X = dequantize(state)
            m, e = ema_start(state)
    return state, o_all, diags


def truth_outputs(X, q, k, v, s, beta, erase=True):
    """float64 outputs of one token from the float32 state X (no quantisation)."""
    return recurrence.truth_step_rowform(X, q, k, v, s, beta, erase)[1]


def warm_state(q, k, v, s, beta, cfg):
    """Quantised record after an unquantised warm-up from the zero state.

    q, k: [B,T,H,dk]; v: [B,T,H,dv]; s: [B,T,H,dk|1]; beta: [B,T,H].  The
    float64 recurrence (eq. rule) and the token-sequential EMAs run over all
    T tokens; the state is then written back once (quantised with the
    allocation of that moment).  Returns (state, float64 state before the
    write-back).
    """
    B, T, H, _ = np.asarray(q).shape
    S = np.zeros((B, H, cfg.dk, cfg.dv), F64)
    m = e = None
    for t in range(T):
        S, _ = recurrence.truth_step_rowform(S, q[:, t], k[:, t], v[:, t], s[:, t], beta[:, t],
                                             cfg.erase)
        sr = _rows(s[:, t], cfg.dk)
        bt = np.asarray(beta[:, t])[..., None]
        if m is None:
            m, e = stats.ema_init(sr, k[:, t], bt, cfg.erase)
        else:
            m, e = stats.ema_update(m, e, sr, k[:, t], bt, cfg.span, cfg.erase)
    st, _ = write_back(S.astype(F32), m, e, np.full((B, H), T, np.int64), cfg)
    return st, S
