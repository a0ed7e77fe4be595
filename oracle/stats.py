"""Decay/erase statistics, Gramian weights and log-uniform rate codes.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

All arithmetic is float64; each function states its operation order so that
the kernels can follow it.  Transcendentals (exp, log, log2, exp2, expm1) come
from NumPy; the kernels call HIP's device functions, so values that pass
through one may differ in the last float64 bit.

* ``ema_init`` / ``ema_update``: the exponential moving averages of Sec. 3
  (State bit allocation): m_i tracks exp(2 g) = exp(-2 s) and e_i tracks
  beta (2 - beta) k_i^2 (0 without erasure: the erase term comes from the
  erase vector a = beta k), with alpha = 2 / (span + 1); the first token of a
  fresh state initialises both; updates are token-sequential, so any write-back
  interval C sees the same estimates.  s_hat = -log(m)/2, r = e/2.
* ``gamma_hat``: eq. weight, 1 / expm1(2 (s_hat + r)), with s_hat + r clamped
  below at 1e-12 (the paper requires s > 0).
* ``mode_gamma``: the row factor of the allocation key for the weight
  variants the paper ablates (Sec. 5, Table ablate): "ema" (ours, eq.
  weight), "gamma_raw" (the same factor, raw ranges), "range" and
  "rel_range" and "uniform" (factor 1), "persist" (DAMP's uncapped
  persistence w^(1) = 1/(1 - a^2) with a = exp(-s_hat), Related work),
  "writeback" (h^(C) = 1/(1 - exp(-2 C s_hat)), Choice of persistence
  factor), "no_erase_rate" (eq. weight with r = 0).  Rates are clamped below
  at 1e-12 as in gamma_hat.
* ``window_gamma``: eq. gram restricted to a window of W tokens with the
  diagonal erase approximation of Sec. 2 (Approximate erasure rate): per row,
  lambda_t = exp(-2 s_t - beta_t (2 - beta_t) k_t^2)  (no erase term
  without erasure),
  A_t = lambda_t (chi_{t-1} + A_{t-1}), Gamma = (1/W) sum_{t>=1} q_t^2 A_t,
  chi_tau = 1 when a write-back follows token tau.
* ``exact_window_gamma`` / ``stationary_gamma``: the full matrix Gramian of
  eq. gram (backward recursion over a window, or the Lyapunov fixed point
  O = F^T (Q + O) F for a constant transition); for pins only.
* ``logq_encode`` / ``logq_decode``: rates coded with levels uniform in
  log s (Sec. 3, Decay-gate quantization), 16 bits over [2^-20, 2^5].
* ``gate_quantize``: per-token gate quantisation with 2^b levels uniform in
  log s (or, for comparison, in g = -s) over the range of a head's channels
  at that token (Sec. 3, Decay-gate quantization).

Parity: pinned (P5 closed form, P6 worked example, P7 fixed-key series, P8
bound, P17 codes, P18 EMA) in ``tests/test_oracle_stats.py``.
"""
import numpy as np

F64 = np.float64
F32 = np.float32

LOGQ_LO = -20.0          # log2 of the smallest coded rate
LOGQ_HI = 5.0            # log2 of the largest coded rate
LOGQ_LEVELS = 65535
LOGQ_STEP = F64(LOGQ_HI - LOGQ_LO) / F64(LOGQ_LEVELS)     # fl64(25/65535)
LOGQ_INV_STEP = F64(LOGQ_LEVELS) / F64(LOGQ_HI - LOGQ_LO)  # fl64(65535/25)
GAMMA_FLOOR = 1e-12


def ema_alpha(span):
    return F64(2.0) / F64(span + 1)


def decay_sample(s):
    """z = exp(-2 s), s float32 promoted exactly."""
    return np.exp(F64(-2.0) * np.asarray(s, F32).astype(F64))


def erase_sample(k, beta, erase=True):
    """y = (beta (2 - beta)) (k k), float64, each product rounded once
    (0 without erasure)."""
    b = np.asarray(beta, F32).astype(F64)
    kk = np.asarray(k, F32).astype(F64)
    y = (b * (F64(2.0) - b)) * (kk * kk)
    return y if erase else np.zeros_like(y)


def ema_init(s, k, beta, erase=True):
    return decay_sample(s), erase_sample(k, beta, erase)


def ema_update(m, e, s, k, beta, span, erase=True):
    al = ema_alpha(span)
    om = F64(1.0) - al
    m = om * m + al * decay_sample(s)
    e = om * e + al * erase_sample(k, beta, erase)
    return m, e


def ema_rates(m, e):
    """(s_hat, r) from the EMA states."""
    with np.errstate(divide="ignore"):
        s_hat = F64(-0.5) * np.log(m)
    return s_hat, F64(0.5) * e


def gamma_hat(s_hat, r):
    t = np.maximum(np.asarray(s_hat, F64) + np.asarray(r, F64), GAMMA_FLOOR)
    return F64(1.0) / np.expm1(F64(2.0) * t)


WEIGHT_MODES = ("ema", "range", "gamma_raw", "rel_range", "persist", "writeback",
                "no_erase_rate", "uniform", "decay")


def mode_gamma(s_hat, r, mode="ema", C=1):
    s_hat = np.asarray(s_hat, F64)
    if mode in ("ema", "gamma_raw", "decay"):
        return gamma_hat(s_hat, r)
    if mode == "no_erase_rate":
        return gamma_hat(s_hat, np.zeros_like(s_hat))
    if mode == "persist":
        return F64(1.0) / -np.expm1(F64(-2.0) * np.maximum(s_hat, GAMMA_FLOOR))
    if mode == "writeback":
        return F64(1.0) / -np.expm1((F64(-2.0) * F64(C)) * np.maximum(s_hat, GAMMA_FLOOR))
    assert mode in ("range", "rel_range", "uniform"), mode
    return np.ones_like(s_hat)


def logq_encode(s_hat):
    s_hat = np.asarray(s_hat, F64)
    with np.errstate(divide="ignore", invalid="ignore"):
        u = (np.log2(s_hat) - F64(LOGQ_LO)) * LOGQ_INV_STEP
    u = np.where(s_hat > 0, u, 0.0)
    u = np.where(np.isnan(u), 0.0, u)
    return np.clip(np.rint(u), 0, LOGQ_LEVELS).astype(np.uint16)


def logq_decode(z):
    return np.exp2(np.asarray(z, np.uint16).astype(F64) * LOGQ_STEP + F64(LOGQ_LO))


def r_encode(r):
    """r stored as FP16 of its float32 rounding."""
    return np.asarray(r, F64).astype(F32).astype(np.float16)


def ema_from_record(z, r16):
    """EMA states a write-back leaves behind: m = exp(-2 s_dec), e = 2 r_dec."""
    s_dec = logq_decode(z)
    return np.exp(F64(-2.0) * s_dec), F64(2.0) * np.asarray(r16, np.float16).astype(F64)


def writeback_positions(W, C, offset=0):
    """chi_tau for tau = 0..W-1: 1 when token offset+tau+1 is a multiple of C."""
    t = np.arange(W) + offset + 1
    return (t % C == 0).astype(F64)


def window_gamma(q, s, k, beta, C, erase=True):
    """Windowed query-weighted decay sums, float64.

    q, s, k: [W, ..., dk]; beta: [W, ...].  Returns [..., dk].
    """
    q = np.asarray(q, F32).astype(F64)
    W = q.shape[0]
    y = erase_sample(k, np.asarray(beta, F32)[..., None], erase)
    lam = np.exp(F64(-2.0) * np.asarray(s, F32).astype(F64) - y)
    chi = writeback_positions(W, C)
    A = np.zeros(q.shape[1:], F64)
    acc = np.zeros(q.shape[1:], F64)
    for t in range(1, W):
        A = lam[t] * (chi[t - 1] + A)
        acc = acc + (q[t] * q[t]) * A
    return acc / F64(W)


def transition(k, s, beta, erase=True):
    """F = (I - beta k k^T) diag(exp(-s)), float64."""
    k = np.asarray(k, F64)
    dk = k.shape[0]
    D = np.diag(np.exp(-np.asarray(s, F64) * np.ones(dk)))
    E = np.eye(dk) - (beta * np.outer(k, k) if erase else 0.0)
    return E @ D


def exact_window_gamma(qs, Fs, C):
    """Matrix Gramian over a window: qs [W, dk], Fs [W, dk, dk] (F_t).

    M_tau = F_{tau+1}^T (q_{tau+1} q_{tau+1}^T + M_{tau+1}) F_{tau+1},
    Gamma_i = (1/W) sum_tau chi_tau (M_tau)_{ii}.
    """
    W, dk = qs.shape
    chi = writeback_positions(W, C)
    M = np.zeros((dk, dk))
    out = np.zeros(dk)
    for tau in range(W - 2, -1, -1):
        F = Fs[tau + 1]
        M = F.T @ (np.outer(qs[tau + 1], qs[tau + 1]) + M) @ F
        out += chi[tau] * np.diag(M)
    return out / W


def stationary_gamma(F, Q, C=1):
    """Gamma_i = O_ii / C with O = sum_{l>=1} (F^l)^T Q F^l (eq. gram)."""
    from scipy.linalg import solve_discrete_lyapunov
    O = solve_discrete_lyapunov(F.T, F.T @ Q @ F)
    return np.diag(O) / C


def gate_quantize(s, bits, mode="log"):
    """Per-token decay-gate quantisation (Sec. 3, Decay-gate quantization):
    s [..., dk] float32 rates of one token and head; levels uniform in log s
    (mode "log") or in g = -s (mode "linear") over the range of the head's
    channels at that token; 2^bits levels, nearest level (ties to even).
    float64 arithmetic; returns the dequantised rates as float32.

        x = log(s) (or s), lo = min x, hi = max x over the channels,
        n = 2^bits - 1, step = (hi - lo) / n,
        code = clamp(rne((x - lo) / step), 0, n)  (0 when step = 0),
        x^ = lo + code step, s^ = fl32(exp(x^)) (or fl32(x^)).
    """
    s = np.asarray(s, F32).astype(F64)
    x = np.log(s) if mode == "log" else s
    lo = np.min(x, axis=-1, keepdims=True)
    hi = np.max(x, axis=-1, keepdims=True)
    n = F64((1 << bits) - 1)
    step = (hi - lo) / n
    with np.errstate(divide="ignore", invalid="ignore"):
        code = np.where(step > 0, np.clip(np.rint((x - lo) / step), 0, n), 0.0)
    xh = lo + code * step
    return (np.exp(xh) if mode == "log" else xh).astype(F32)
