"""Pins for head allocation units with block scales (Sec. 3, Allocation units:
Gated DeltaNet has one width per head and FP16 scales per block of 32 key
channels; R~ = 1, so only decay sets the widths; a two-bit mean reduces to
uniform block quantisation)."""
import itertools
from fractions import Fraction

import numpy as np
import pytest

import workloads as W
from oracle import alloc, quant, record, step


@pytest.mark.parametrize("b", [2, 3, 4, 6, 8])
def test_block_fit_is_argmin_of_exact_error(b):
    rng = np.random.default_rng(300 + b)
    x = rng.standard_t(3, (64, 3)).astype(np.float32)     # two blocks x three columns
    codes, scale, mstar = quant.quantize_blocks(x, b)
    n = 2 ** (b - 1) - 1
    phi = quant.phi_table(b)
    for kb in range(2):
        for j in range(3):
            g = x[32 * kb:32 * kb + 32, j]
            R = np.float32(np.max(np.abs(g)))
            exact = []
            for m in range(16):
                d = np.float32(np.float16(np.float32(R * phi[m])))
                inv = np.float32(1.0) / d if d > 0 else np.float32(0.0)
                c = np.clip(np.rint((g * inv).astype(np.float32)), -n, n)
                D = Fraction(float(d))
                exact.append(sum((Fraction(float(xx)) - int(cc) * D) ** 2 for xx, cc in zip(g, c)))
            lo = min(exact)
            assert exact[mstar[kb, j]] <= lo * (1 + Fraction(1, 2 ** 16))
            f = quant.clip_factor(mstar[kb, j])
            assert float(scale[kb, j]) == pytest.approx(f * float(R) / n, rel=2 ** -10)
            assert np.all(np.abs(codes[32 * kb:32 * kb + 32, j]) <= n)


def test_block_codes_are_nearest_clamped_levels():
    rng = np.random.default_rng(7)
    x = rng.uniform(-1, 1, (128, 64)).astype(np.float32)
    codes, scale, _ = quant.quantize_blocks(x, 5)
    d = np.repeat(scale.astype(np.float64), 32, axis=0)
    inside = np.abs(x) <= 15 * d
    # inside the clip range the code is the nearest level
    assert np.all(np.abs(x - codes * d)[inside] <= d[inside] / 2 * (1 + 1e-6))
    xh = quant.dequantize_blocks(codes, scale)
    # uniform-noise model Delta^2/12: the fit over only 32 elements per group
    # picks the best of 16 grids, which biases the error a little below it
    assert np.mean((x - xh) ** 2 / (d ** 2 / 12)) == pytest.approx(1.0, abs=0.1)


def _gdn(H=4, dk=64):
    w = W.sized(W.WORKLOADS["gdn2"], B=1, H=H, dk=dk, dv=dk, G=dk, T=24)
    xs = W.tokens(w, 0, 24)
    return w, xs


def test_two_bit_mean_reduces_to_uniform_block_quantization():
    w, xs = _gdn()
    oc = step.Cfg(dk=64, dv=64, G=64, mean_bits=2.0, b_min=2, b_max=8, unit="head")
    st, S = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    assert np.all(st["width"] == 2)
    for h in range(4):
        c, sc, _ = quant.quantize_blocks(S[0, h].astype(np.float32), 2)
        assert np.array_equal(st["codes"][0, h], c)
        assert np.array_equal(st["bscale"][0, h].view(np.uint16), sc.view(np.uint16))


def test_widths_depend_only_on_decay():
    """R~ = 1: scaling the state leaves the widths unchanged; slower decay
    (larger Gamma) never gets fewer bits."""
    w, xs = _gdn()
    oc = step.Cfg(dk=64, dv=64, G=64, mean_bits=4.0, b_min=2, b_max=8, unit="head")
    st, S = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    m, e = step.ema_start(st)
    a, da = step.write_back_heads(S.astype(np.float32), m, e, st["ntok"], oc)
    b, db = step.write_back_heads((10 * S).astype(np.float32), m, e, st["ntok"], oc)
    assert np.array_equal(a["width"], b["width"])
    order = np.argsort(da["c"][0])
    assert np.all(np.diff(a["width"][0][order]) >= 0)
    assert len(set(a["width"][0].tolist())) > 1


def test_head_key_minimises_the_row_proxy_by_brute_force():
    """With one width per head the proxy is sum_h sum_i Gamma_hi 2^(-2 b_h); the
    widths from the heads' mean Gamma reach its brute-force minimum."""
    rng = np.random.default_rng(11)
    for _ in range(20):
        g = np.exp(rng.uniform(-6, 3, (4, 64)))
        for mean in (2.5, 3.0, 4.25):
            wid = alloc.allocate(alloc.head_weights(g), mean, 2, 6)
            K = alloc.budget(mean, 4)
            best = min(sum(float(np.sum(g[h])) * 2.0 ** (-2 * bb[h]) for h in range(4))
                       for bb in itertools.product(range(2, 7), repeat=4) if sum(bb) == K)
            got = sum(float(np.sum(g[h])) * 2.0 ** (-2 * wid[h]) for h in range(4))
            assert got == pytest.approx(best, rel=1e-12)


def test_head_weights_mean_in_row_order():
    g = np.array([[1e16, 1.0, -1e16, 1.0]])
    assert alloc.head_weights(g)[0] == ((1e16 + 1.0) - 1e16 + 1.0) / 4


def test_head_record_round_trip_and_zero_state():
    rng = np.random.default_rng(5)
    for dk, b in ((64, 2), (128, 5), (256, 8)):
        x = rng.standard_normal((dk, 32)).astype(np.float32)
        c, sc, _ = quant.quantize_blocks(x, b)
        z = rng.integers(0, 65535, dk)
        r16 = rng.uniform(0, 1, dk).astype(np.float16)
        buf = record.pack_heads(7, b, sc, z, r16, c, dk, 32, 8)
        assert buf.size == record.record_bytes_heads(dk, 32, 8)
        f = record.unpack_heads(buf, dk, 32, 8)
        assert f["ntok"] == 7 and f["width"] == b
        assert np.array_equal(f["codes"], c) and np.array_equal(f["z"], z)
        assert np.array_equal(f["bscale"].view(np.uint16), sc.view(np.uint16))
        # row i of every column starts at bit i b
        words = buf[record.layout_heads(dk, 32, 8)["codes_off"]:].view(np.uint32)
        fld = (int(words[(3 * b) // 32 * 32]) >> ((3 * b) % 32)) & ((1 << b) - 1)
        if (3 * b) % 32 + b <= 32:
            assert fld == int(c[3, 0]) & ((1 << b) - 1)
    zero = record.unpack_heads(np.zeros(record.record_bytes_heads(64, 64, 8), np.uint8), 64, 64, 8)
    assert zero["width"] == 0 and not zero["codes"].any()
    oc = step.Cfg(dk=64, dv=64, unit="head")
    assert not step.dequantize(step.zero_state(1, 2, oc)).any()


def test_head_stored_bits():
    # payload + 0.5 (block scales) + rate code and erase rate per row + width
    assert record.stored_bits_heads(2.0, 256, 256) == 2.0 + 0.5 + 32 / 256 + 32 / 65536
    assert record.accounting(2.0, 256, block_scale=True) == 2.5
