"""Pins for the record layout and the paper's bit accounting (Sec. 3)."""
import json
import os

import numpy as np
import pytest

from oracle import quant, record

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))


@pytest.mark.parametrize("dk,dv,bmax", [(64, 64, 8), (128, 128, 8), (128, 128, 16), (256, 256, 8)])
def test_pack_unpack_roundtrip(dk, dv, bmax):
    rng = np.random.default_rng(dk + bmax)
    widths = rng.integers(1, bmax + 1, dk)
    codes = np.zeros((dk, dv), np.int64)
    for i, b in enumerate(widths):
        n = (1 << (b - 1)) - 1
        codes[i] = rng.integers(0, 2, dv) if b == 1 else rng.integers(-n, n + 1, dv)
    scale = rng.random(dk).astype(np.float16)
    z = rng.integers(0, 65536, dk).astype(np.uint16)
    r16 = rng.random(dk).astype(np.float16)
    buf = record.pack(7, widths, scale, z, r16, codes, dk, dv, bmax)
    assert buf.size == record.record_bytes(dk, dv, bmax) and buf.size % 256 == 0
    f = record.unpack(buf, dk, dv, bmax)
    assert f["ntok"] == 7
    assert np.array_equal(f["widths"], widths) and np.array_equal(f["codes"], codes)
    assert np.array_equal(f["scale"].view(np.uint16), scale.view(np.uint16))
    assert np.array_equal(f["z"], z) and np.array_equal(f["r16"].view(np.uint16), r16.view(np.uint16))
    # code bits: d_v * sum(b) / 8 bytes, prefix-sum offsets
    nw = record.used_words(widths)
    assert nw * 32 >= widths.sum() > (nw - 1) * 32
    L = record.layout(dk, dv, bmax)
    words = np.frombuffer(buf[L["codes_off"]:].tobytes(), np.uint32)[: L["wc"] * dv].reshape(L["wc"], dv)
    assert np.all(words[nw:] == 0)
    tail = int(widths.sum()) % 32
    if tail:
        assert np.all(words[nw - 1] >> tail == 0)


def test_row_offsets_are_prefix_sums():
    dk, dv = 64, 64
    widths = np.array([3, 5] * 32)
    codes = np.zeros((dk, dv), np.int64)
    codes[1, :] = -1                     # row 1: all ones in 5 bits at bit 3
    buf = record.pack(0, widths, np.zeros(dk, np.float16), np.zeros(dk, np.uint16),
                      np.zeros(dk, np.float16), codes, dk, dv, 8)
    L = record.layout(dk, dv, 8)
    w0 = np.frombuffer(buf[L["codes_off"]:L["codes_off"] + 4 * dv].tobytes(), np.uint32)
    assert np.all(w0 == 0b11111000)


def test_zero_record_is_zero_state():
    dk, dv = 128, 128
    f = record.unpack(np.zeros(record.record_bytes(dk, dv, 8), np.uint8), dk, dv, 8)
    x = quant.dequantize_rows(f["codes"], f["scale"], f["widths"])
    assert f["ntok"] == 0 and np.all(f["widths"] == 1) and np.all(x == 0)


def test_p15_bit_accounting_matches_paper():
    g = GOLD["metadata_bits"]
    dv = g["dv"]
    assert round(record.accounting(2, dv, 3), 3) == g["table3_ours_bits_kimi"]
    assert round(record.accounting(4, dv, 4), 3) == g["table2_ours_bits_kimi"]
    assert record.accounting(4, dv, block_scale=True) == g["table2_ours_bits_qwen"]
    assert record.accounting(2, dv, block_scale=True) == g["table3_ours_bits_qwen36"]
    assert (16 + 3) == g["scale_plus_3bit_width_per_dv"]
    assert record.stored_bits(4, 128) == pytest.approx(4 + 52 / 128)
