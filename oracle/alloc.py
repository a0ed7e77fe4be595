"""Range normalisation and high-rate bit allocation (Sec. 3, eq. weight, eq. alloc).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

* ``normalized_ranges``: R~_i = R_i / RMS of R over the output-normalisation
  group of row i (Sec. 2, Range normalization; Sec. 3 after eq. weight).
  Groups are G consecutive rows: within one head (KDA, Gated DeltaNet), or
  spanning consecutive heads (Mamba-2 normalises over 12 heads); the caller
  passes the rows of all heads of a group along the last axis.  Sum of squares is sequential in
  row order in float64 (each R_j^2 is exact); RMS = sqrt(sum / G); a group with
  RMS 0 gives R~ = 0.
* ``weights``: c_i = Gamma_i * (R~_i * R~_i)  (eq. weight).
* ``mode_weights``: the key for the ablated weight variants: R~^2 for the
  normalised modes, raw R^2 for "range" and "gamma_raw", 1 for "uniform"
  (the rows' factors from ``stats.mode_gamma``).
* ``allocate``: minimise the high-rate proxy sum_i c_i 2^(-2 b_i) over integer
  widths in [b_min, b_max] with sum b_i = K = round(mean_bits * N) (Sec. 3:
  round, clip and adjust to the layer budget).  Written as its greedy
  equivalent: every row owns slots l = b_min+1 .. b_max whose value is the
  proxy reduction c_i 2^(-2l) * 3 (monotone in c_i 4^(-l)); the K - N b_min
  slots with the largest c_i 4^(-l) are granted, ties to the lower row index
  (then the lower l).  Slot values of one row fall with l, so granted slots
  form a prefix and b_i = b_min + (slots granted to row i).  Keys are compared
  exactly as (exponent - 2l, mantissa) pairs.
* ``head_weights``: the key of a head unit (Sec. 3, Allocation units: one
  width per head, R~ = 1 so only decay sets widths).  Rows sharing one width
  b contribute (sum_i Gamma_i) 2^(-2b) to the proxy, so the head's key is the
  mean Gamma of its rows (sequential float64 sum in row order, / d_k); heads
  are then allocated like rows.
* ``allocate_bruteforce``: exhaustive search over all width vectors, tiny N.
* ``real_allocation`` / ``am_gm_gain``: eq. alloc and the AM/GM distortion
  ratio quoted after it.

Parity: pinned (P9 real-valued budget and AM/GM, P10 brute force, P11 scale
invariance, P12 normalisation) in ``tests/test_oracle_alloc.py``.
"""
import itertools
import numpy as np

F64 = np.float64


class BudgetError(ValueError):
    pass


def budget(mean_bits, n_rows):
    return int(np.floor(F64(mean_bits) * F64(n_rows) + 0.5))


# Rows per run of the group sum of squares (the paper fixes no summation
# order; runs let a group of many rows be summed in parallel).
RMS_RUN = 64


def normalized_ranges(R, G):
    """R: [..., dk] float32 row maxima -> R~ float64 [..., dk]."""
    R = np.asarray(R, np.float32).astype(F64)
    dk = R.shape[-1]
    assert dk % G == 0
    out = np.zeros_like(R)
    for g0 in range(0, dk, G):
        # sum of squares in runs of RMS_RUN consecutive rows, each run summed
        # in row order from zero and the run sums added in order
        acc = np.zeros(R.shape[:-1], F64)
        for c0 in range(g0, g0 + G, RMS_RUN):
            part = np.zeros(R.shape[:-1], F64)
            for j in range(c0, min(c0 + RMS_RUN, g0 + G)):
                part = part + R[..., j] * R[..., j]
            acc = acc + part
        rms = np.sqrt(acc / F64(G))
        with np.errstate(divide="ignore", invalid="ignore"):
            rt = R[..., g0:g0 + G] / rms[..., None]
        out[..., g0:g0 + G] = np.where(rms[..., None] > 0, rt, 0.0)
    return out


def weights(gamma, Rt):
    Rt = np.asarray(Rt, F64)
    return np.asarray(gamma, F64) * (Rt * Rt)


def mode_weights(gamma, R, Rt, mode="ema"):
    """gamma: row factors; R: float32 row maxima; Rt: normalised ranges."""
    gamma = np.asarray(gamma, F64)
    if mode == "uniform":
        return np.ones_like(gamma)
    if mode == "decay":
        return gamma.copy()   # ranges ignored (R~ taken as 1)
    if mode in ("range", "gamma_raw"):
        Rr = np.asarray(R, np.float32).astype(F64)
        return gamma * (Rr * Rr)
    return weights(gamma, Rt)


def allocate(c, mean_bits, b_min, b_max):
    """c: [N] float64 >= 0 -> widths [N] int, greedy top-K slots."""
    c = np.asarray(c, F64).ravel()
    N = c.size
    K = budget(mean_bits, N)
    need = K - N * b_min
    if need < 0 or K > N * b_max:
        raise BudgetError("budget outside [b_min, b_max]")
    mant, expo = np.frexp(c)                      # c = mant * 2^expo, mant in [0.5, 1)
    expo = expo.astype(np.int64)
    rows, levels, e_key, m_key = [], [], [], []
    for l in range(b_min + 1, b_max + 1):
        rows.append(np.arange(N))
        levels.append(np.full(N, l))
        e_key.append(np.where(c > 0, expo - 2 * l, np.iinfo(np.int64).min // 2))
        m_key.append(np.where(c > 0, mant, 0.0))
    rows = np.concatenate(rows)
    levels = np.concatenate(levels)
    e_key = np.concatenate(e_key).astype(np.int64)
    m_key = np.concatenate(m_key)
    # sort: larger key first, then lower row, then lower level
    order = np.lexsort((levels, rows, -m_key, -e_key))
    chosen = order[:need]
    b = np.full(N, b_min, np.int64)
    np.add.at(b, rows[chosen], 1)
    return b


def head_weights(gamma):
    """gamma: [..., dk] float64 -> [...] mean over the rows."""
    gamma = np.asarray(gamma, F64)
    dk = gamma.shape[-1]
    acc = np.zeros(gamma.shape[:-1], F64)
    for i in range(dk):
        acc = acc + gamma[..., i]
    return acc / F64(dk)


def proxy(c, b):
    return float(np.sum(np.asarray(c, F64) * np.exp2(-2.0 * np.asarray(b, F64))))


def allocate_bruteforce(c, mean_bits, b_min, b_max):
    """Minimum proxy value over all integer width vectors with the budget."""
    c = np.asarray(c, F64).ravel()
    N = c.size
    K = budget(mean_bits, N)
    best = None
    for b in itertools.product(range(b_min, b_max + 1), repeat=N):
        if sum(b) != K:
            continue
        v = proxy(c, b)
        if best is None or v < best[0]:
            best = (v, b)
    return best


def real_allocation(c, mean_bits):
    """eq. alloc: b_i = mean + 0.5 log2(c_i / GM(c))."""
    c = np.asarray(c, F64)
    lg = np.log2(c)
    return F64(mean_bits) + 0.5 * (lg - lg.mean())


def am_gm_gain(c):
    c = np.asarray(c, F64)
    return c.mean() / np.exp(np.log(c).mean())
