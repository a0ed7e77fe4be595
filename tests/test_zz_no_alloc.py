"""kda_step_noalloc (the allocation-free decode step on the library's own
device scratch) against kda_step with a caller workspace, through the C ABI:
records and outputs bit for bit on two calls in a row, the second with a
smaller input (fewer sequences and heads, narrower heads), each starting
from records the library wrote."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2609_30950_amd as K
import workloads as W
from tests._gpu import dev, say

pytestmark = pytest.mark.gpu


def _cfg(w):
    return K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.G, mean_bits=w.mean_bits,
                    b_min=w.b_min, b_max=w.b_max)


def _compare_once(w, warm, label):
    kc = _cfg(w)
    base = W.base_rates(w)
    recs = K.new_records(kc)
    ws = K.new_workspace(kc)
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    for t in range(warm):   # records written by the library
        x = {n: dev(a) for n, a in W.token(w, t, base=base).items()}
        K.kda_step(kc, recs, x["q"], x["k"], x["v"], x["s"], x["beta"], o, ws)
    x = {n: dev(a) for n, a in W.token(w, warm, base=base).items()}
    ra, rb = recs.clone(), recs.clone()
    oa = torch.full_like(o, 7.0)
    ob = torch.full_like(o, -7.0)
    K.kda_step(kc, ra, x["q"], x["k"], x["v"], x["s"], x["beta"], oa, ws)
    K.api.kda_step_noalloc(kc, rb, x["q"], x["k"], x["v"], x["s"], x["beta"], ob)
    torch.cuda.synchronize()
    same_r = torch.equal(ra, rb)
    same_o = torch.equal(oa.view(torch.int32), ob.view(torch.int32))
    say(f"{label}: records equal {same_r}, outputs equal {same_o}")
    assert same_r and same_o


def test_noalloc_step_equals_workspace_step_then_smaller():
    lib = K.load()
    assert lib.kda_step_noalloc_max_bytes() == 16 << 20
    _compare_once(W.WORKLOADS["decode"], 6, "decode B=64 H=32 d=128")
    _compare_once(W.sized(W.WORKLOADS["tiny"], B=3, H=4, mean_bits=3.0), 9, "B=3 H=4 d=64")


def test_noalloc_rejects_oversized_scratch_before_launch():
    w = W.sized(W.WORKLOADS["decode"], B=128)
    kc = _cfg(w)
    st = K.load().kda_step_noalloc(ctypes.byref(kc.c()), None, None, None, None, None, None, None,
                                   None, None)
    assert st == 4   # KDA_ERR_WORKSPACE
