"""Gated delta-rule recurrence (Sec. 2, eq. rule), KDA instance (Sec. 1).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Per head, with unit-norm key k, per-row decay rates s > 0, D = diag(exp(-s)),
erase vector a = beta*k and write weights w = beta*1 (the KDA and Gated
DeltaNet choice stated after eq. rule):

    S_t = (I - k a^T) D S_{t-1} + k (w * v)^T,      o_t = S_t^T q.

With erase=False the erase vector is a = 0 (Mamba-2 has no erasure, stated
after eq. rule): S_t = D S_{t-1} + k (w * v)^T.

``truth_step`` evaluates that definition literally in float64 with explicit
d_k x d_k matrices.  ``truth_step_rowform`` is the algebraically equal
row form (I - b k k^T) D S = D S - b k (k^T D S), also float64.
``mirror_step`` is the float32 contract the kernels follow:

    a_i  = fl32(exp(-s_i))                     (exp evaluated in float64)
    S'   = fl32(a_i * S_ij)
    u_j  = blockdot(k, S'[:, j])
    g_i  = fl32(beta * k_i),   w_j = fl32(v_j - u_j)
    S_ij = fma32(g_i, w_j, S'_ij)
    o_j  = blockdot(q, S[:, j])

(without erasure: w_j = v_j, and u is not formed.)

blockdot: rows are cut into blocks of 32 consecutive rows; inside a block the
products are accumulated sequentially from the first row with float32 fused
multiply-adds starting from 0; block partials are combined by strided halving.

Parity: pinned (P1 dense form vs row form, P2 pure decay, P3 identity at
beta=0 s=0, P4 delta-rule recall) in ``tests/test_oracle_recurrence.py``.
"""
import numpy as np

from .fp import fma32, halving_tree, F32, F64

ROW_BLOCK = 32


def truth_step(S, q, k, v, s, beta, erase=True):
    """Literal eq. rule in float64 for one head.  S: [dk, dv]."""
    S = np.asarray(S, F64)
    dk = S.shape[0]
    k = np.asarray(k, F64)
    D = np.diag(np.exp(-np.asarray(s, F64) * np.ones(dk)))
    a = beta * k if erase else np.zeros(dk)
    w = beta * np.ones(S.shape[1])
    F = (np.eye(dk) - np.outer(k, a)) @ D
    S_new = F @ S + np.outer(k, w * np.asarray(v, F64))
    return S_new, S_new.T @ np.asarray(q, F64)


def truth_step_rowform(S, q, k, v, s, beta, erase=True):
    """Row form of the same update, float64, batched over leading axes.

    S: [..., dk, dv]; q, k, s: [..., dk] (s may be [..., 1]); v: [..., dv];
    beta: [...].
    """
    S = np.asarray(S, F64)
    k = np.asarray(k, F64)
    beta = np.asarray(beta, F64)[..., None]
    a = np.exp(-np.asarray(s, F64))
    Sd = a[..., :, None] * S
    u = np.einsum("...i,...ij->...j", k, Sd) if erase else 0.0
    S_new = Sd + (beta * k)[..., :, None] * (np.asarray(v, F64) - u)[..., None, :]
    o = np.einsum("...i,...ij->...j", np.asarray(q, F64), S_new)
    return S_new, o


def blockdot(x, M):
    """Contract's float32 dot over rows: x [..., dk], M [..., dk, dv] -> [..., dv]."""
    x = np.asarray(x, F32)
    M = np.asarray(M, F32)
    dk = M.shape[-2]
    assert dk % ROW_BLOCK == 0
    parts = []
    for b0 in range(0, dk, ROW_BLOCK):
        acc = np.zeros(M.shape[:-2] + M.shape[-1:], F32)
        for i in range(b0, b0 + ROW_BLOCK):
            acc = fma32(x[..., i:i + 1], M[..., i, :], acc)
        parts.append(acc)
    return halving_tree(parts).astype(F32)


def decay_factors(s):
    """a = fl32(exp(-s)) with exp taken in float64."""
    return np.exp(-np.asarray(s, F32).astype(F64)).astype(F32)


def mirror_step(S, q, k, v, s, beta, erase=True):
    """float32 contract form, batched: S [..., dk, dv] float32.

    s is [..., dk] (per-row decay) or [..., 1] (one rate per head).
    Returns (S_new float32, o float32).
    """
    S = np.asarray(S, F32)
    a = decay_factors(s)
    Sd = (a[..., :, None] * S).astype(F32)
    g = (np.asarray(beta, F32)[..., None] * np.asarray(k, F32)).astype(F32)
    if erase:
        w = (np.asarray(v, F32) - blockdot(k, Sd)).astype(F32)
    else:
        w = np.asarray(v, F32)
    S_new = fma32(g[..., :, None], w[..., None, :], Sd)
    o = blockdot(q, S_new)
    return S_new, o
