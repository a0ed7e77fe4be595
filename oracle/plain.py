"""Plain definitions of the write-back's discrete decisions, as validity checks.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The float32 contract (``quant``, ``alloc``, ``recurrence``) fixes one
evaluation order for every sum so that two implementations decide bit for
bit alike.  Several of those orders are not the paper's but a kernel's
choice: error sums in 64-column segments, group sums of squares in runs of
64 rows, row contractions in blocks of 32 rows.  This module checks the same
decisions against their plain mathematical definitions -- no blocking, sums
exact or correctly rounded in float64, quotients instead of reciprocals --
so that a decision that is right only under the contract's order is caught.
It takes the float32 state a write-back quantises (the GPU's own, in the
tests) and the row factors Gamma, and the record's decoded fields.

* Keys (Sec. 3, eq. weight; Sec. 2, Range normalization): R_i = max_j |S_ij|,
  RMS_g = sqrt(fsum(R_j^2) / G) over the G rows of the group (math.fsum:
  the correctly rounded sum of the exact squares), c_i = Gamma_i (R_i/RMS_g)^2.
* Widths (Sec. 3, eq. alloc, rounded, clipped and adjusted to the budget):
  b minimises sum_i c_i 2^(-2 b_i) subject to sum_i b_i = K and
  b_min <= b_i <= b_max.  The objective is separable and convex in each b_i,
  so b is optimal iff moving one bit between two rows never lowers it:
      min_{i: b_i > b_min} c_i 4^(-b_i)  >=  max_{j: b_j < b_max} c_j 4^(-b_j - 1).
* Clip factor and scale (Sec. 3, Levels and storage): for width b >= 2,
  n = 2^(b-1) - 1 and candidate m = 0..15 has f_m = (5 + m)/20 and the FP16
  scale fp16(f_m R / n) (f_m R / n formed in float64, rounded once to FP16,
  saturating at 65504).  A candidate's error is sum_j (x_j - Delta c_j)^2
  with c_j the nearest level clamp(round(x_j / Delta), -n, n), summed in
  float64 over exact residuals.  The stored scale must be a candidate's and
  its error the minimum over the 16.
* Codes: the nearest clamped level of the stored scale.  One-bit rows: code
  1 for x < 0 and scale fp16(mean_j |x_j|).

Where the float32 contract's rounding can legitimately differ from the plain
value, the case is counted as exempt rather than failed, with a bound:
* a scale whose exact value f R / n lies within a relative 2^-22 of an FP16
  rounding midpoint (the contract rounds R * fl32(f / n) to float32 first):
  either neighbour may be a candidate, so the chosen error must not exceed,
  for every candidate, the larger error of its two versions;
* a clip factor whose error exceeds the minimum by at most the float32
  summation bound 2 (L + 4) 2^-24 (L summed elements) relative;
* a code whose quotient x / Delta lies within a relative 2^-21 of a midpoint
  between levels (the contract multiplies by fl32(1 / Delta));
* rows whose width slot lies within a relative 1e-12 of the allocation
  threshold (keys agree with the contract's to about 1e-15).

Pinned in ``tests/test_oracle_plain.py``: brute force over all width vectors
on tiny rows, exhaustive rational-arithmetic fits, and planted mistakes
(a moved bit, another candidate's scale, a code off by one) that must fail.
"""
import math
from fractions import Fraction

import numpy as np

F64 = np.float64
F32 = np.float32
N_FIT = 16
FP16_MAX = 65504.0
WIDTH_RTOL = 1e-12
SCALE_RTOL = 2.0 ** -22
CODE_RTOL = 2.0 ** -21


# ----------------------------------------------------------------- keys ---

def group_rms(R, G):
    """R [..., N] float32 row maxima -> RMS per row's group, float64 [..., N]."""
    R = np.asarray(R, F32)
    flat = R.reshape(-1, R.shape[-1]).astype(F64)
    N = flat.shape[-1]
    assert N % G == 0
    out = np.empty_like(flat)
    for u in range(flat.shape[0]):
        for g0 in range(0, N, G):
            sq = [float(v) * float(v) for v in flat[u, g0:g0 + G]]   # exact in float64
            out[u, g0:g0 + G] = math.sqrt(math.fsum(sq) / G)
    return out.reshape(R.shape)


def keys(gamma, R, G, mode="ema"):
    """Allocation keys c [..., N] from row factors gamma and row maxima R
    (groups of G consecutive rows along the last axis)."""
    gamma = np.asarray(gamma, F64)
    Rr = np.asarray(R, F32).astype(F64)
    if mode == "uniform":
        return np.ones_like(gamma)
    if mode == "decay":
        return gamma.copy()
    if mode in ("range", "gamma_raw"):
        return gamma * (Rr * Rr)
    rms = group_rms(R, G)
    with np.errstate(divide="ignore", invalid="ignore"):
        Rt = np.where(rms > 0, Rr / rms, 0.0)
    return gamma * (Rt * Rt)


# --------------------------------------------------------------- widths ---

def check_widths(c, b, mean_bits, b_min, b_max, rtol=WIDTH_RTOL):
    """Optimality of widths b [N] for keys c [N] (one allocation scope).

    Returns dict(ok, exempt, margin): ok False on a budget or bound violation
    or a moved bit that lowers the objective by more than rtol; exempt = rows
    whose boundary slot lies within rtol of the threshold when the exchange
    condition holds only within rtol."""
    c = np.asarray(c, F64).ravel()
    b = np.asarray(b, np.int64).ravel()
    N = c.size
    K = int(math.floor(float(mean_bits) * N + 0.5))
    res = dict(ok=True, exempt=0, margin=math.inf)
    if int(b.sum()) != K or b.min() < b_min or b.max() > b_max:
        res["ok"] = False
        return res
    granted = b > b_min
    open_ = b < b_max
    if not granted.any() or not open_.any():
        return res
    last = np.ldexp(c, -2 * b)            # value of each row's last granted slot
    nxt = np.ldexp(c, -2 * (b + 1))       # value of each row's next slot
    g = float(np.min(last[granted]))
    n = float(np.max(nxt[open_]))
    if g >= n:
        res["margin"] = (g - n) / n if n > 0 else math.inf
        return res
    res["margin"] = (g - n) / n
    if g < n * (1.0 - rtol):
        res["ok"] = False
        return res
    band = (granted & (last < n)) | (open_ & (nxt > g))
    res["exempt"] = int(band.sum())
    return res


# ------------------------------------------------------------------ fit ---

def fp16_sat(v):
    """float64 -> FP16 value (round to nearest even), saturating at 65504."""
    v = np.asarray(v, F64)
    with np.errstate(over="ignore"):
        h = v.astype(np.float16)
    return np.where(np.isinf(h) & np.isfinite(v), np.copysign(FP16_MAX, v), h.astype(F64))


def _near_midpoint_alt(v, h, rtol):
    """For exact values v and their FP16 roundings h: the other FP16
    neighbour where v lies within rtol of the midpoint between them, else h."""
    v = np.asarray(v, F64)
    h16 = np.asarray(h, F64).astype(np.float16)
    with np.errstate(over="ignore", invalid="ignore"):
        up = np.nextafter(h16, np.float16(np.inf)).astype(F64)
        dn = np.nextafter(h16, np.float16(-np.inf)).astype(F64)
    other = np.where(v >= h, up, dn)
    mid = 0.5 * (np.asarray(h, F64) + other)
    near = np.isfinite(other) & (np.abs(v - mid) <= rtol * np.abs(v)) & (other <= FP16_MAX)
    return np.where(near, other, h)


def candidate_scales(R, b):
    """Plain FP16 scales of the 16 candidates: [rows, 16] float64."""
    n = F64((1 << (int(b) - 1)) - 1)
    R = np.asarray(R, F32).astype(F64)
    v = np.stack([(F64(5 + m) * R) / (F64(20.0) * n) for m in range(N_FIT)], axis=-1)
    return v, fp16_sat(v)


def nearest_codes(x, delta, n):
    """Nearest levels clamp(round(x / Delta), -n, n) (ties to even) with their
    quotients; Delta = 0 gives code 0.  x [rows, L], delta [rows]."""
    x = np.asarray(x, F32).astype(F64)
    d = np.asarray(delta, F64)[..., None]
    with np.errstate(divide="ignore", invalid="ignore"):
        y = np.where(d > 0, x / np.where(d > 0, d, 1.0), 0.0)
    return np.clip(np.rint(y), -n, n), y


def errors(x, delta, n):
    """Squared error of nearest-level quantisation with scale Delta, float64
    sums of exact residuals.  x [rows, L], delta [rows] -> [rows]."""
    c, _ = nearest_codes(x, delta, n)
    e = np.asarray(x, F32).astype(F64) - c * np.asarray(delta, F64)[..., None]
    return np.sum(e * e, axis=-1)


def check_fit(x, b, scale, codes):
    """Validity of scales and codes of rows (or scale groups) x [rows, L]
    float32 with widths b [rows], stored FP16 scales [rows] and codes
    [rows, L] (b >= 2: signed integers; b = 1: 1 for negative).

    Returns counts: rows, bad_scale, bad_fit, bad_codes (must be 0) and
    exempt_scale, exempt_fit, exempt_codes (near ties within the bounds of
    the module docstring)."""
    x = np.asarray(x, F32)
    b = np.asarray(b, np.int64).ravel()
    scale = np.asarray(scale, np.float16).ravel().astype(F64)
    codes = np.asarray(codes, np.int64)
    rows, L = x.shape
    ftol = 2.0 * (L + 4) * 2.0 ** -24
    out = dict(rows=rows, bad_scale=0, bad_fit=0, bad_codes=0, exempt_scale=0, exempt_fit=0,
               exempt_codes=0, bad_rows=[])
    for w in np.unique(b):
        idx = np.nonzero(b == w)[0]
        xs = x[idx]
        if w == 1:
            a = np.abs(xs.astype(F64))
            mean = np.array([math.fsum(r) for r in a]) / L
            mu = fp16_sat(mean)
            alt = _near_midpoint_alt(mean, mu, (L + 4) * 2.0 ** -24)
            ok_mu = (scale[idx] == mu)
            ex_mu = ~ok_mu & (scale[idx] == alt)
            out["exempt_scale"] += int(ex_mu.sum())
            bad = ~(ok_mu | ex_mu)
            out["bad_scale"] += int(bad.sum())
            out["bad_rows"] += [int(i) for i in idx[bad]]
            cb = (xs < 0).astype(np.int64)
            badc = np.any(codes[idx] != cb, axis=-1)
            out["bad_codes"] += int(np.sum(codes[idx] != cb))
            out["bad_rows"] += [int(i) for i in idx[badc]]
            continue
        n = (1 << (int(w) - 1)) - 1
        R = np.max(np.abs(xs), axis=-1)
        v, d = candidate_scales(R, w)                       # [k, 16]
        alt = _near_midpoint_alt(v, d, SCALE_RTOL)
        E = np.stack([errors(xs, d[:, m], n) for m in range(N_FIT)], axis=-1)
        Ea = np.stack([errors(xs, alt[:, m], n) for m in range(N_FIT)], axis=-1)
        Emin = np.min(E, axis=-1)
        # a float32-contract evaluation may have taken the other FP16
        # neighbour of any candidate whose value lies near a midpoint: its
        # choice cannot exceed the best of the worse versions
        Ebound = np.min(np.maximum(E, Ea), axis=-1)
        ds = scale[idx]
        in_plain = np.any(d == ds[:, None], axis=-1)
        in_alt = np.any(alt == ds[:, None], axis=-1) & ~in_plain
        bad_s = ~(in_plain | in_alt)
        out["bad_scale"] += int(bad_s.sum())
        Es = errors(xs, ds, n)
        exact = Es <= Emin * (1.0 + 1e-12)
        near = ~exact & (Es <= Emin * (1.0 + ftol))
        rounding = ~exact & ~near & (Es <= Ebound * (1.0 + ftol))
        out["exempt_fit"] += int((near & ~bad_s).sum())
        out["exempt_scale"] += int(((in_alt | rounding) & ~bad_s).sum())
        bad_f = ~exact & ~near & ~rounding
        out["bad_fit"] += int(bad_f.sum())
        cp, y = nearest_codes(xs, ds, n)
        fr = np.abs(y - np.floor(y) - 0.5)
        tie = (fr <= CODE_RTOL * np.maximum(np.abs(y), 1.0)) & (np.abs(y) <= n + 0.5)
        diff = codes[idx] != cp
        out["exempt_codes"] += int(np.sum(diff & tie))
        badc = diff & ~tie
        out["bad_codes"] += int(badc.sum())
        out["bad_rows"] += [int(i) for i in idx[bad_s | bad_f | np.any(badc, axis=-1)]]
    return out


def fp16_of_fraction(q):
    """Exact rational -> nearest FP16 value (ties to the even significand),
    saturating at 65504; q >= 0."""
    q = Fraction(q)
    if q >= Fraction(FP16_MAX):
        return FP16_MAX
    h = np.float16(float(q))
    cands = {float(h)}
    for d in (np.float16(np.inf), np.float16(-np.inf)):
        nb = float(np.nextafter(h, d))
        if math.isfinite(nb):
            cands.add(nb)
    best = None
    for c in sorted(cands):
        dist = abs(Fraction(c) - q)
        even = (int(np.float16(c).view(np.uint16)) & 1) == 0
        key = (dist, 0 if even else 1)
        if best is None or key < best[0]:
            best = (key, c)
    return best[1]


def fit_exact_rational(x, b):
    """Index m of the first strict minimum of the 16 candidates' errors in
    exact rational arithmetic (x one row of float32 values, b >= 2), each
    scale the exact FP16 rounding of f_m R / n: the definition check_fit
    evaluates in float64."""
    n = (1 << (b - 1)) - 1
    xs = [Fraction(float(v)) for v in np.asarray(x, F32)]
    R = max(abs(v) for v in xs)
    best = None
    for m in range(N_FIT):
        dlt = Fraction(fp16_of_fraction(Fraction(5 + m, 20 * n) * R))
        err = Fraction(0)
        for v in xs:
            c = 0 if dlt == 0 else max(-n, min(n, round(v / dlt)))
            err += (v - c * dlt) ** 2
        if best is None or err < best[0]:
            best = (err, m)
    return best[1]


def summary(label, res):
    keys_ = ("rows", "bad_scale", "bad_fit", "bad_codes", "exempt_scale", "exempt_fit",
             "exempt_codes")
    return f"{label}: " + " ".join(f"{k}={res[k]}" for k in keys_)
