"""Exact float helpers for the MIRROR (float32 contract) oracle.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

``fma32`` returns the correctly rounded float32 value of a*b+c.  NumPy has no
fused multiply-add, so it is emulated: a*b is exact in float64 (24+24 bit
significands), a*b+c is formed in float64 with its exact rounding error
(Knuth's TwoSum), and the only case in which rounding that float64 sum to
float32 differs from rounding the exact value (the float64 sum landing exactly
on a float32 midpoint) is resolved with the sign of the TwoSum error.
Pinned against rational arithmetic in ``tests/test_oracle_fp.py``.
"""
import numpy as np

F32 = np.float32
F64 = np.float64
FP16_MAX = 65504.0


def f32(x):
    return np.asarray(x, dtype=np.float32)


def fma32(a, b, c):
    """Correctly rounded float32 fused multiply-add, elementwise."""
    a, b, c = np.broadcast_arrays(np.asarray(a, F32), np.asarray(b, F32),
                                  np.asarray(c, F32))
    p = a.astype(F64) * b.astype(F64)           # exact
    cc = c.astype(F64)
    s = p + cc                                  # rounded float64 sum
    bb = s - p
    err = (p - (s - bb)) + (cc - bb)            # s + err == p + c exactly
    r = s.astype(F32)                           # round-to-nearest-even
    # neighbour of r on the side of s; is s exactly the float32 midpoint?
    with np.errstate(invalid="ignore", over="ignore"):
        toward = np.where(s > r.astype(F64), np.inf, -np.inf).astype(F32)
        rn = np.nextafter(r, toward)
        mid = (r.astype(F64) + rn.astype(F64)) * 0.5
        is_mid = (s == mid) & (s != r.astype(F64)) & (err != 0)
        # exact value lies on the rn side of the midpoint iff err points there
        goes_rn = np.sign(err) == np.sign(rn.astype(F64) - s)
        fix = is_mid & goes_rn
        r = np.where(fix, rn, r)
        # s rounded to r (the even neighbour) while the exact value is past
        # the midpoint away from rn: then the true neighbour is on r's far side
        # cannot happen (s is the midpoint between r and rn only).
    return r.astype(F32)


def fp16_sat(x):
    """float32 -> nearest FP16 (ties to even), saturating at +-65504."""
    with np.errstate(over="ignore"):
        h = np.asarray(x, F32).astype(np.float16)
    h = np.where(np.isinf(h) & np.isfinite(np.asarray(x, F32)),
                 np.copysign(np.float16(FP16_MAX), h), h)
    return h.astype(np.float16)


def halving_tree(parts):
    """Combine a list of equally shaped float arrays by strided halving.

    With L parts (a power of two): part[p] += part[p + L/2] for p < L/2, then
    L/2, ..., until one remains.  Each addition is rounded in the dtype of the
    parts.  This is the fixed combine order of partial sums used by the
    contract for row blocks and column segments.
    """
    parts = list(parts)
    L = len(parts)
    assert L & (L - 1) == 0, "number of parts must be a power of two"
    while L > 1:
        h = L // 2
        parts = [parts[p] + parts[p + h] for p in range(h)]
        L = h
    return parts[0]
