"""Seeded synthetic inputs shaped like the paper's hybrid-model layers.

Holds none of the method's arithmetic: only random draws, normalisation of
q/k to unit length and the bf16 rounding of prefill inputs.  Both the tests of
the oracle and the GPU tests and bench draw their inputs here, so the two sides
always see identical arrays.

Every token t of workload ``name`` with seed ``seed`` is drawn from
``numpy.random.default_rng([seed, 1, t])`` in the fixed order
q, k, v, beta, s (so any token range can be regenerated independently);
per-channel base rates come from ``default_rng([seed, 0])``.

Recipes (the paper's models and data are not available; these stand in):
  tiny      B=1  H=2  d=64   T=256   q,k ~ N(0,1) normalised; v ~ N(0,1);
            beta = sigmoid(N(0,1)); s = base + 0.05 N(0,1) clamped >= 1e-4,
            base = exp(U[log 1e-3, 0]) per (b, h, channel)
  decode    B=64 H=32 d=128  same draws as tiny; 512 warm-up tokens
  prefill   B=4  H=32 d=128  T=8192  bf16 q/k/v; s constant in time per
            (b, h, channel): 10% logU[1e-4, 1e-3), else logU[1e-3, 2]
  gdn       B=16 H=16 d=256  T=4096  one s per (b, h, token): logU[1e-4, 1]
  long      B=128 H=32 d=128 T=32768 v ~ Student-t(3); decay as tiny
  mamba2    B=16 H=24 d=128 T=4096  Mamba-2-style layer: one rate per (b, h,
            token) logU[1e-4, 1], no erasure, normalisation groups of 12 heads
            (1536 rows), mean 4 bits, widths [1,8]; draws as tiny otherwise
"""
from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    dk: int
    dv: int
    T: int
    C: int = 1
    mean_bits: float = 4.0
    b_min: int = 2
    b_max: int = 8
    G: int = 64
    decay: str = "jitter"        # jitter | static | head
    v_dist: str = "normal"       # normal | t3
    bf16: bool = False
    warmup: int = 0
    window: int = 0
    erase: bool = True           # False: no erasure (Mamba-2)


WORKLOADS = {
    "tiny": Workload("tiny", 1, 2, 64, 64, 256, C=1, mean_bits=4.0, b_min=2, b_max=8, G=64),
    "decode": Workload("decode", 64, 32, 128, 128, 1, C=1, mean_bits=4.0, b_min=2, b_max=8,
                       G=64, warmup=512),
    "prefill": Workload("prefill", 4, 32, 128, 128, 8192, C=64, mean_bits=4.0, b_min=1,
                        b_max=8, G=128, decay="static", bf16=True),
    "gdn2": Workload("gdn2", 16, 16, 256, 256, 4096, C=1, mean_bits=2.0, b_min=1, b_max=8,
                     G=256, decay="head"),
    "gdn6": Workload("gdn6", 16, 16, 256, 256, 4096, C=1, mean_bits=6.0, b_min=1, b_max=8,
                     G=256, decay="head"),
    "long": Workload("long", 128, 32, 128, 128, 32768, C=1, mean_bits=3.0, b_min=2, b_max=8,
                     G=64, v_dist="t3", window=1024),
    "mamba2": Workload("mamba2", 16, 24, 128, 128, 4096, C=1, mean_bits=4.0, b_min=1, b_max=8,
                       G=12 * 128, decay="head", erase=False),
}


def sized(w, **kw):
    """A copy of workload w with some fields replaced (smaller test shapes)."""
    d = dict(w.__dict__)
    d.update(kw)
    return Workload(**d)


def _unit(x):
    x = x / np.linalg.norm(x, axis=-1, keepdims=True)
    return x


def bf16_round(x):
    """Round float32 to bfloat16 (nearest even) and back to float32."""
    x = np.ascontiguousarray(x, np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32)


def base_rates(w, seed=0):
    rng = np.random.default_rng([seed, 0])
    if w.decay == "jitter":
        return np.exp(rng.uniform(np.log(1e-3), 0.0, (w.B, w.H, w.dk)))
    if w.decay == "static":
        slow = rng.random((w.B, w.H, w.dk)) < 0.1
        lo = np.exp(rng.uniform(np.log(1e-4), np.log(1e-3), (w.B, w.H, w.dk)))
        hi = np.exp(rng.uniform(np.log(1e-3), np.log(2.0), (w.B, w.H, w.dk)))
        return np.where(slow, lo, hi)
    return None


def tokens(w, t0, t1, seed=0, base=None):
    """Inputs for tokens [t0, t1): dict of float32 arrays
    q, k [B,T,H,dk]; v [B,T,H,dv]; beta [B,T,H]; s [B,T,H,dk] (or [B,T,H,1]
    for one rate per head)."""
    if base is None:
        base = base_rates(w, seed)
    out = {n: [] for n in ("q", "k", "v", "beta", "s")}
    for t in range(t0, t1):
        rng = np.random.default_rng([seed, 1, t])
        q = _unit(rng.standard_normal((w.B, w.H, w.dk)))
        k = _unit(rng.standard_normal((w.B, w.H, w.dk)))
        if w.v_dist == "t3":
            v = rng.standard_t(3, (w.B, w.H, w.dv))
        else:
            v = rng.standard_normal((w.B, w.H, w.dv))
        beta = 1.0 / (1.0 + np.exp(-rng.standard_normal((w.B, w.H))))
        if w.decay == "jitter":
            s = np.maximum(base + 0.05 * rng.standard_normal((w.B, w.H, w.dk)), 1e-4)
        elif w.decay == "static":
            s = base
        else:
            s = np.exp(rng.uniform(np.log(1e-4), 0.0, (w.B, w.H, 1)))
        for n, a in (("q", q), ("k", k), ("v", v), ("beta", beta), ("s", s)):
            out[n].append(np.asarray(a, np.float32))
    res = {n: np.stack(a, axis=1) for n, a in out.items()}
    if w.bf16:
        for n in ("q", "k", "v"):
            res[n] = bf16_round(res[n])
    return res


def token(w, t, seed=0, base=None):
    """Inputs of one token with the T axis removed: q, k [B,H,dk], ..."""
    return {n: a[:, 0] for n, a in tokens(w, t, t + 1, seed, base).items()}
