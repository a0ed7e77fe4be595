"""GPU parity of per-token decay-gate quantisation (kda_gate_quant) against
the oracle's codec: levels uniform in log s and in g = -s, 2 and 4 bits,
d_k = 64, 128 and 256, in place.  float64 log/exp on both sides may differ in
the last bit, which can move a value across a level boundary only at exact
ties: at most one element in 10^5 may differ, by one level."""
import numpy as np
import pytest
import torch

import paper_2609_30950_amd as K
from oracle import stats
from tests._gpu import dev, host, say

pytestmark = pytest.mark.gpu


def _gates(rng, shape):
    s = np.exp(rng.uniform(np.log(1e-3), np.log(2.0), shape))
    slow = rng.random(shape) < 0.1
    s[slow] = np.exp(rng.uniform(np.log(1e-4), np.log(1e-3), slow.sum()))
    return s.astype(np.float32)


@pytest.mark.parametrize("dk", [64, 128, 256])
@pytest.mark.parametrize("bits,mode", [(2, "log"), (4, "log"), (2, "linear"), (4, "linear")])
def test_gate_codec_matches_oracle(dk, bits, mode):
    B, T, H = 2, 24, 4
    s = _gates(np.random.default_rng(dk + bits), (B, T, H, dk))
    cfg = K.Config(B=B, H=H, d_k=dk, d_v=dk, group_rows=dk)
    g = dev(s)
    K.kda_gate_quant(cfg, T, bits, g, g, mode)          # in place
    got = host(g)
    want = stats.gate_quantize(s, bits, mode)
    diff = got.view(np.uint32) != want.view(np.uint32)
    say(f"gates d={dk} bits={bits} {mode}: {int(diff.sum())} of {diff.size} differ")
    assert diff.sum() <= max(1, diff.size // 100000)
    assert np.allclose(got, want, rtol=1e-6) or diff.sum() <= 1
    assert max(len(np.unique(r)) for r in got.reshape(-1, dk)) <= 2 ** bits


def test_gate_codec_rejects_per_head_decay():
    cfg = K.Config(B=1, H=2, d_k=64, d_v=64, group_rows=64, decay_per_head=1)
    g = torch.ones(1 * 4 * 2, dtype=torch.float32, device="cuda")
    with pytest.raises(K.KdaError):
        K.kda_gate_quant(cfg, 4, 2, g, g)
