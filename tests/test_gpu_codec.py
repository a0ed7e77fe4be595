"""GPU parity of kda_pack_state / kda_unpack_state against the oracle (bit
exact), and the packed scales and codes against the plain definitions of the
fit (oracle/plain.py)."""
import numpy as np
import pytest
import torch

import paper_2609_30950_amd as K
from oracle import quant, record, stats
from tests._gpu import bytes_to_state, dev, host, meaningful_equal, plain_check, say

pytestmark = pytest.mark.gpu


def _oracle_pack(S, bits, s_hat, r, ntok, dk, dv, bmax):
    B, H = bits.shape[:2]
    out = []
    for b in range(B):
        for h in range(H):
            codes, scale, _ = quant.quantize_rows(S[b, h], bits[b, h])
            out.append(record.pack(ntok, bits[b, h], scale, stats.logq_encode(s_hat[b, h]),
                                   stats.r_encode(r[b, h]), codes, dk, dv, bmax))
    return np.concatenate(out)


CASES = [
    # B, H, d, bmin, bmax, distribution
    (2, 3, 64, 1, 8, "normal"),
    (1, 4, 128, 1, 8, "t3"),
    (2, 2, 128, 2, 16, "normal"),
    (1, 2, 64, 1, 16, "mixed"),
]


def _inputs(rng, B, H, d, bmin, bmax, dist):
    shape = (B, H, d, d)
    if dist == "t3":
        S = rng.standard_t(3, shape)
    elif dist == "mixed":
        S = rng.standard_normal(shape) * np.exp(rng.uniform(-30, 12, (B, H, d, 1)))
        S[0, 0, 3] = 0.0
        S[0, 0, 5, ::7] = -0.0
        S[0, 1, 9] = 1e7
    else:
        S = rng.standard_normal(shape)
    S = S.astype(np.float32)
    bits = rng.integers(bmin, bmax + 1, (B, H, d)).astype(np.uint8)
    s_hat = np.exp(rng.uniform(np.log(1e-6), np.log(30), (B, H, d)))
    r = rng.uniform(0, 0.5, (B, H, d))
    return S, bits, s_hat, r


@pytest.mark.parametrize("case", CASES)
def test_pack_matches_oracle_bit_exact(case):
    B, H, d, bmin, bmax, dist = case
    say("pack case", case)
    rng = np.random.default_rng(d + bmax)
    S, bits, s_hat, r = _inputs(rng, B, H, d, bmin, bmax, dist)
    cfg = K.Config(B=B, H=H, d_k=d, d_v=d, group_rows=d, b_min=bmin, b_max=bmax,
                   mean_bits=(bmin + bmax) / 2)
    recs = K.new_records(cfg)
    K.kda_pack_state(cfg, dev(S), dev(bits), dev(s_hat), dev(r), 5, recs)
    got = host(recs)
    want = _oracle_pack(S, bits, s_hat, r, 5, d, d, bmax)
    bad = meaningful_equal(got, want, B, H, d, d, bmax)
    assert not bad, f"records differ for slots {bad}"
    plain_check(S, None, bytes_to_state(got, B, H, d, d, bmax), G=d, scope=0,
                mean_bits=cfg.mean_bits, b_min=bmin, b_max=bmax, label=f"pack {case}")


@pytest.mark.parametrize("case", CASES)
def test_unpack_matches_oracle(case):
    B, H, d, bmin, bmax, dist = case
    say("unpack case", case)
    rng = np.random.default_rng(100 + d + bmax)
    S, bits, s_hat, r = _inputs(rng, B, H, d, bmin, bmax, dist)
    want_rec = _oracle_pack(S, bits, s_hat, r, 3, d, d, bmax)
    cfg = K.Config(B=B, H=H, d_k=d, d_v=d, group_rows=d, b_min=bmin, b_max=bmax,
                   mean_bits=(bmin + bmax) / 2)
    recs = dev(want_rec)
    Sg = torch.empty(B * H * d * d, dtype=torch.float32, device="cuda")
    bg = torch.empty(B * H * d, dtype=torch.uint8, device="cuda")
    sg = torch.empty(B * H * d, dtype=torch.float64, device="cuda")
    rg = torch.empty(B * H * d, dtype=torch.float64, device="cuda")
    K.kda_unpack_state(cfg, recs, Sg, bg, sg, rg)
    slot = record.record_bytes(d, d, bmax)
    X = np.zeros((B, H, d, d), np.float32)
    for b in range(B):
        for h in range(H):
            f = record.unpack(want_rec[(b * H + h) * slot:(b * H + h + 1) * slot], d, d, bmax)
            X[b, h] = quant.dequantize_rows(f["codes"], f["scale"], f["widths"])
    assert np.array_equal(host(Sg).reshape(B, H, d, d).view(np.uint32), X.view(np.uint32))
    assert np.array_equal(host(bg).reshape(B, H, d), bits)
    np.testing.assert_allclose(host(sg).reshape(B, H, d),
                               stats.logq_decode(stats.logq_encode(s_hat)), rtol=4e-16)
    assert np.array_equal(host(rg).reshape(B, H, d),
                          stats.r_encode(r).astype(np.float64))


def test_zero_records_unpack_to_zero_state():
    cfg = K.Config(B=2, H=2, d_k=128, d_v=128)
    recs = K.new_records(cfg)
    Sg = torch.full((2 * 2 * 128 * 128,), 7.0, dtype=torch.float32, device="cuda")
    K.kda_unpack_state(cfg, recs, Sg)
    assert torch.count_nonzero(Sg).item() == 0


def test_one_bit_rows_with_zero_mean_keep_signs():
    """A one-bit row whose mean |x| rounds to an FP16 zero decodes to +-0
    with the sign of each code (the oracle's -mu for negative codes)."""
    d = 64
    rng = np.random.default_rng(11)
    S = (np.where(rng.random((1, 1, d, d)) < 0.5, -1.0, 1.0) * 1e-30).astype(np.float32)
    bits = np.ones((1, 1, d), np.uint8)
    cfg = K.Config(B=1, H=1, d_k=d, d_v=d, group_rows=d, b_min=1, b_max=8, mean_bits=4)
    want = _oracle_pack(S, bits, np.full((1, 1, d), 0.01), np.zeros((1, 1, d)), 1, d, d, 8)
    f = record.unpack(want, d, d, 8)
    X = quant.dequantize_rows(f["codes"], f["scale"], f["widths"])
    assert np.all(X == 0) and np.any(np.signbit(X))
    Sg = torch.empty(d * d, dtype=torch.float32, device="cuda")
    K.kda_unpack_state(cfg, dev(want), Sg)
    assert np.array_equal(host(Sg).view(np.uint32), X.reshape(-1).view(np.uint32))


def _midpoint_ranges(b, m, count, rng):
    """float32 ranges R whose float32 product R*phi lands exactly on an FP16
    midpoint while the exact product does not (single vs double rounding
    disagree there)."""
    phi = quant.phi_table(b)[m]
    out = []
    while len(out) < count:
        R = np.float32(rng.uniform(0.05, 4.0))
        for _ in range(4000):
            p = np.float32(R * phi)
            h = np.float16(p)
            if float(p) != float(h):
                up = np.nextafter(h, np.float16(np.inf))
                dn = np.nextafter(h, np.float16(-np.inf))
                mids = ((float(h) + float(up)) / 2, (float(h) + float(dn)) / 2)
                exact = float(R) * float(phi)
                if float(p) in mids and exact != float(p):
                    out.append(R)
                    break
            R = np.nextafter(R, np.float32(np.inf))
    return np.array(out, np.float32)


def test_scale_rounding_on_fp16_midpoints():
    """Delta = fp16(fl32(R phi)): the float32 product is rounded first."""
    rng = np.random.default_rng(3)
    b, d = 5, 64
    R = _midpoint_ranges(b, 15, 16, rng)
    S = np.where(rng.random((1, 16, d, d)) < 0.5, -1.0, 1.0).astype(np.float32)
    S = S * R[None, :, None, None]        # rows of +-R: the fit picks f = 1
    bits = np.full((1, 16, d), b, np.uint8)
    s_hat = np.full((1, 16, d), 0.01)
    r = np.zeros((1, 16, d))
    cfg = K.Config(B=1, H=16, d_k=d, d_v=d, group_rows=d, b_min=1, b_max=8, mean_bits=4)
    recs = K.new_records(cfg)
    K.kda_pack_state(cfg, dev(S), dev(bits), dev(s_hat), dev(r), 1, recs)
    want = _oracle_pack(S, bits, s_hat, r, 1, d, d, 8)
    assert not meaningful_equal(host(recs), want, 1, 16, d, d, 8)
