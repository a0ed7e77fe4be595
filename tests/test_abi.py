"""CPU-side checks of the C ABI: the library loads, exports every declared
symbol, sizes records like the oracle's layout and validates arguments
before launching anything (no GPU needed)."""
import ctypes
import os
import re

import pytest

import paper_2609_30950_amd as K
from oracle import record

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "kda.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(kda_[a-z0-9_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2609_30950_amd", "libkda.so"))
    names = _declared()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n


@pytest.mark.parametrize("d,bmax", [(64, 8), (128, 8), (128, 16), (256, 8), (256, 4)])
def test_record_bytes_match_layout(d, bmax):
    cfg = K.Config(B=1, H=1, d_k=d, d_v=d, group_rows=d, b_min=1, b_max=bmax, mean_bits=2)
    assert K.record_bytes(cfg) == record.record_bytes(d, d, bmax)
    cfg.state32 = 1
    assert K.record_bytes(cfg) == record.state32_bytes(d, d)


def test_invalid_configs_rejected():
    lib = K.load()
    bad = [
        dict(d_k=96, d_v=96),                  # unsupported width
        dict(d_k=64, d_v=128),
        dict(mean_bits=1.5),                   # budget below b_min
        dict(mean_bits=8.5),
        dict(b_min=0),
        dict(b_max=17),
        dict(group_rows=48),
        dict(scope=2),
        dict(ema_span=0),
        dict(H=64, d_k=128, d_v=128),          # > 4096 rows in one budget
        dict(H=17, d_k=256, d_v=256, group_rows=256),
        dict(d_k=256, d_v=256, group_rows=256, b_max=16),   # 256 rows: widths up to 8
    ]
    for kw in bad:
        base = dict(B=1, H=2, d_k=64, d_v=64, group_rows=64)
        base.update(kw)
        cfg = K.Config(**base)
        assert K.record_bytes(cfg) == 0, kw
        st = lib.kda_step(ctypes.byref(cfg.c()), None, None, None, None, None, None, None, None,
                          None, None)
        assert st != 0, kw


def test_null_pointers_rejected_before_launch():
    lib = K.load()
    cfg = K.Config(B=1, H=2, d_k=64, d_v=64)
    assert lib.kda_step(ctypes.byref(cfg.c()), None, None, None, None, None, None, None, None,
                        None, None) == 1
    assert lib.kda_pack_state(ctypes.byref(cfg.c()), None, None, None, None, 0, None, None) == 1
    assert lib.kda_unpack_state(ctypes.byref(cfg.c()), None, None, None, None, None, None) == 1
    assert lib.kda_weights(ctypes.byref(cfg.c()), 0, 1, None, None, None, None, None, None) == 1
    assert lib.kda_weights_exact(ctypes.byref(cfg.c()), 4, 1, None, None, None, None, None,
                                 None) == 1
    wide = K.Config(B=1, H=2, d_k=256, d_v=256, group_rows=256)
    one = ctypes.c_void_p(1)
    assert lib.kda_weights_exact(ctypes.byref(wide.c()), 4, 1, one, one, one, one, one,
                                 one) == 3   # rejected before any launch
    assert lib.kda_status_str(3).decode() == "unsupported configuration"


def test_head_unit_configs():
    base = dict(B=1, H=16, d_k=256, d_v=256, group_rows=256, b_min=2, b_max=8, mean_bits=2.0,
                decay_per_head=1, head_units=1)
    from oracle import record as rec
    assert K.record_bytes(K.Config(**base)) == rec.record_bytes_heads(256, 256, 8)
    for kw in (dict(b_min=1), dict(b_max=9), dict(group_rows=64), dict(scope=1),
               dict(mean_bits=1.5), dict(head_units=2)):
        cfg = dict(base)
        cfg.update(kw)
        assert K.record_bytes(K.Config(**cfg)) == 0, kw
    lib = K.load()
    cfg = K.Config(**base)
    one = ctypes.c_void_p(16)
    assert lib.kda_pack_state(ctypes.byref(cfg.c()), one, one, one, one, 0, one, None) == 3
    assert lib.kda_unpack_state(ctypes.byref(cfg.c()), one, one, None, None, None, None) == 3
    assert lib.kda_alloc_bits(ctypes.byref(cfg.c()), one, one, one, one, None) == 3
    for mode, ok in ((1, False), (2, False), (3, False), (4, True), (7, True), (8, True), (9, False)):
        c = K.Config(**base)
        c.weight_mode = mode
        assert (K.record_bytes(c) > 0) == ok, mode
    bad = K.Config(B=1, H=2, d_k=64, d_v=64, weight_mode=9)
    assert K.record_bytes(bad) == 0


def test_empty_requests_rejected_before_launch():
    """Zero sequences, heads, tokens, window or interval: an error status, and
    nothing launched (the calls return on a machine without a GPU)."""
    lib = K.load()
    one = ctypes.c_void_p(256)
    for kw in (dict(B=0), dict(H=0), dict(B=-1)):
        base = dict(B=1, H=2, d_k=64, d_v=64, group_rows=64)
        base.update(kw)
        cfg = K.Config(**base)
        assert K.record_bytes(cfg) == 0 and K.workspace_bytes(cfg) == 0
        assert lib.kda_step(ctypes.byref(cfg.c()), one, one, one, one, one, one, None, one, one,
                            None) == 2
        assert lib.kda_prefill(ctypes.byref(cfg.c()), 8, 4, one, one, one, one, one, one, None,
                               one, one, None) == 2
    cfg = K.Config(B=1, H=2, d_k=64, d_v=64, group_rows=64)
    c = ctypes.byref(cfg.c())
    for T, C in ((0, 4), (8, 0), (-3, 4)):
        assert lib.kda_prefill(c, T, C, one, one, one, one, one, one, None, one, one, None) == 1
    for W, C in ((0, 1), (16, 0)):
        assert lib.kda_weights(c, W, C, one, one, one, one, one, None) == 1
        assert lib.kda_weights_exact(c, W, C, one, one, one, one, one, None) == 1
    assert lib.kda_gate_quant(c, 0, 4, 0, one, one, None) == 1
    ch = K.Config(B=1, H=2, d_k=64, d_v=64, group_rows=64, chunked=1)
    assert lib.kda_prefill(ctypes.byref(ch.c()), 128, 65, one, one, one, one, one, one, None, one,
                           one, None) == 1   # chunked intervals hold at most 64 tokens
