"""Symmetric per-row quantiser with a fitted clip factor (Sec. 3, Levels and storage).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

For width b >= 2 the levels are {-n..n} * Delta with n = 2^(b-1) - 1 and
Delta = f R / n, R the row's absolute maximum; f is fitted over 16 values in
[1/4, 1] by squared error and the chosen Delta is stored as FP16.  One bit
stores the sign and the row's mean absolute value.  Float32 contract:

    f_m    = (5 + m) / 20, m = 0..15
    phi    = fl32((5 + m) / (20 n))                 (constant table)
    Delta  = fp16(fl32(R * phi)), saturating at 65504
    inv    = fl32(1 / Delta)   (0 when Delta = 0)
    c_j    = clamp(rne(fl32(x_j * inv)), -n, n)
    e_j    = fma32(-c_j, Delta, x_j)
    err    = segsum of e_j^2: per 64-column segment, sequential fma32(e, e, acc)
             from acc = 0; segments combined by strided halving
    m*     = smallest m with err_m equal to the minimum
    1 bit  : mu = fp16(fl32(segsum|x| * (1/d_v))) with float32 additions,
             bit = (x < 0), value = -mu if bit else mu

Dequantisation: x^ = fl32(c * Delta) (b >= 2), +-mu (b = 1).

Head units (Sec. 3, Allocation units: one width per head and scales per block
of 32 key channels): ``quantize_blocks`` applies the same levels and clip-factor
fit to every scale group of 32 consecutive rows of one column, R the group's
absolute maximum, the error summed over the group's rows in row order
(sequential fma32 from 0); widths are at least 2.

Parity: pinned (P13 single write-back MSE, P14 codec rules, P16 brute-force
argmin with rational arithmetic) in ``tests/test_oracle_quant.py``.
"""
import numpy as np

from .fp import fma32, fp16_sat, halving_tree, F32, F64

N_FIT = 16
SEG = 64
BLOCK = 32


def levels(b):
    return (1 << (b - 1)) - 1


def phi_table(b):
    n = levels(b)
    return np.array([F64(5 + m) / F64(20 * n) for m in range(N_FIT)]).astype(F32)


def clip_factor(m):
    return (5 + m) / 20.0


def seg_sumsq(e):
    """e: [rows, dv] float32 -> [rows] float32 (contract order)."""
    dv = e.shape[-1]
    parts = []
    for s0 in range(0, dv, SEG):
        acc = np.zeros(e.shape[:-1], F32)
        for j in range(s0, min(s0 + SEG, dv)):
            acc = fma32(e[..., j], e[..., j], acc)
        parts.append(acc)
    return halving_tree(parts).astype(F32)


def seg_sumabs(x):
    dv = x.shape[-1]
    parts = []
    for s0 in range(0, dv, SEG):
        acc = np.zeros(x.shape[:-1], F32)
        for j in range(s0, min(s0 + SEG, dv)):
            acc = (acc + np.abs(x[..., j])).astype(F32)
        parts.append(acc)
    return halving_tree(parts).astype(F32)


def candidate(x, R, b, m):
    """Codes, scale and error of candidate m for rows x [rows, dv] of width b."""
    n = levels(b)
    phi = phi_table(b)[m]
    delta = fp16_sat((R * phi).astype(F32)).astype(F32)
    with np.errstate(divide="ignore"):
        inv = np.where(delta > 0, (F32(1.0) / delta).astype(F32), F32(0.0)).astype(F32)
    c = np.clip(np.rint((x * inv[:, None]).astype(F32)), -n, n).astype(F32)
    e = fma32(-c, delta[:, None], x)
    return c, delta, seg_sumsq(e)


def quantize_rows(x, b):
    """x: [rows, dv] float32; b: [rows] widths in [1, 16].

    Returns codes int32 [rows, dv], scale float16 [rows], mstar int [rows]
    (-1 for one-bit rows).  One-bit rows return codes 0/1 (1 = negative).
    """
    x = np.asarray(x, F32)
    b = np.asarray(b)
    rows, dv = x.shape
    codes = np.zeros((rows, dv), np.int32)
    scale = np.zeros(rows, np.float16)
    mstar = np.full(rows, -1, np.int64)
    R = np.max(np.abs(x), axis=1).astype(F32)
    for w in np.unique(b):
        idx = np.nonzero(b == w)[0]
        xs = x[idx]
        if w == 1:
            mu = fp16_sat((seg_sumabs(xs) * F32(1.0 / dv)).astype(F32))
            scale[idx] = mu
            codes[idx] = (xs < 0).astype(np.int32)
            continue
        best_err = None
        for m in range(N_FIT):
            c, delta, err = candidate(xs, R[idx], int(w), m)
            if best_err is None:
                best_err, best_c, best_d, best_m = err, c, delta, np.zeros(len(idx), np.int64)
                continue
            better = err < best_err          # strict: keeps the smallest m on ties
            best_err = np.where(better, err, best_err)
            best_c = np.where(better[:, None], c, best_c)
            best_d = np.where(better, delta, best_d)
            best_m = np.where(better, m, best_m)
        codes[idx] = best_c.astype(np.int32)
        scale[idx] = best_d.astype(np.float16)
        mstar[idx] = best_m
    return codes, scale, mstar


def dequantize_rows(codes, scale, b):
    """codes [rows, dv] int, scale float16 [rows], b [rows] -> float32."""
    codes = np.asarray(codes)
    sc = np.asarray(scale, np.float16).astype(F32)
    b = np.asarray(b)
    out = (codes.astype(F32) * sc[:, None]).astype(F32)
    one = b == 1
    if one.any():
        mu = sc[one][:, None]
        out[one] = np.where(codes[one] != 0, -mu, mu)
    return out


def quantize_blocks(x, b):
    """x: [dk, dv] float32 (one head), b >= 2 the head's width.

    Returns codes int32 [dk, dv], scale float16 [dk/32, dv] and mstar
    [dk/32, dv]; scale group (k, j) is rows 32k .. 32k+31 of column j.
    """
    x = np.asarray(x, F32)
    dk, dv = x.shape
    assert b >= 2 and dk % BLOCK == 0
    g = x.reshape(dk // BLOCK, BLOCK, dv)
    R = np.max(np.abs(g), axis=1).astype(F32)
    n = levels(b)
    phi = phi_table(b)
    best_err = None
    for m in range(N_FIT):
        delta = fp16_sat((R * phi[m]).astype(F32)).astype(F32)
        with np.errstate(divide="ignore"):
            inv = np.where(delta > 0, (F32(1.0) / delta).astype(F32), F32(0.0)).astype(F32)
        c = np.clip(np.rint((g * inv[:, None, :]).astype(F32)), -n, n).astype(F32)
        e = fma32(-c, np.broadcast_to(delta[:, None, :], g.shape), g)
        err = np.zeros(R.shape, F32)
        for r in range(BLOCK):
            err = fma32(e[:, r, :], e[:, r, :], err)
        if best_err is None:
            best_err, best_c, best_d, best_m = err, c, delta, np.zeros(R.shape, np.int64)
            continue
        better = err < best_err          # strict: keeps the smallest m on ties
        best_err = np.where(better, err, best_err)
        best_c = np.where(better[:, None, :], c, best_c)
        best_d = np.where(better, delta, best_d)
        best_m = np.where(better, m, best_m)
    return best_c.reshape(dk, dv).astype(np.int32), best_d.astype(np.float16), best_m


def dequantize_blocks(codes, scale):
    """codes [..., dk, dv] int, scale float16 [..., dk/32, dv] -> float32."""
    codes = np.asarray(codes)
    sc = np.asarray(scale, np.float16).astype(F32)
    rep = np.repeat(sc, BLOCK, axis=-2)
    return (codes.astype(F32) * rep).astype(F32)
