"""The entry points are asynchronous on the caller's stream, allocate nothing
and synchronise nothing, so they can be captured in a HIP graph (through
torch.cuda.CUDAGraph).  A captured decode step is replayed token after token
with eager input updates between the replays, and a captured chunked prefill
is replayed from reset records; every replay must equal the eager call bit
for bit."""
import numpy as np
import pytest
import torch

import paper_2609_30950_amd as K
import workloads as W
from oracle import step
from tests._gpu import dev, host, say, state_to_bytes

pytestmark = pytest.mark.gpu


def test_captured_decode_step_replays_equal_eager_steps():
    w = W.sized(W.WORKLOADS["tiny"], B=2, H=4)
    kc = K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.G, mean_bits=w.mean_bits,
                  b_min=w.b_min, b_max=w.b_max)
    oc = step.Cfg(dk=w.dk, dv=w.dv, G=w.G, mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max)
    xs = W.tokens(w, 0, 8)
    st, _ = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    start = dev(state_to_bytes(st, w.dk, w.dv, w.b_max))
    rec_e, rec_g = start.clone(), start.clone()
    ws_e, ws_g = K.new_workspace(kc), K.new_workspace(kc)
    o_e = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    o_g = torch.zeros_like(o_e)
    base = W.base_rates(w)
    x0 = W.token(w, 8, base=base)
    inp = {n: dev(a) for n, a in x0.items()}           # static inputs of the graph
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):                         # warm-up off the default stream
        scratch = start.clone()
        K.kda_step(kc, scratch, inp["q"], inp["k"], inp["v"], inp["s"], inp["beta"], o_g, ws_g)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        K.kda_step(kc, rec_g, inp["q"], inp["k"], inp["v"], inp["s"], inp["beta"], o_g, ws_g)
    torch.cuda.synchronize()
    assert torch.equal(rec_g, start)                      # capture ran nothing
    for t in range(8, 14):
        x = W.token(w, t, base=base)
        for n in inp:
            inp[n].copy_(torch.from_numpy(x[n]))          # eager work between replays
        K.kda_step(kc, rec_e, inp["q"], inp["k"], inp["v"], inp["s"], inp["beta"], o_e, ws_e)
        g.replay()
        torch.cuda.synchronize()
        same_r = torch.equal(rec_e, rec_g)
        same_o = torch.equal(o_e.view(torch.int32), o_g.view(torch.int32))
        say(f"decode replay t={t}: records equal {same_r}, outputs equal {same_o}")
        assert same_r and same_o


@pytest.mark.parametrize("T", [150, 40 * 64 + 5])
def test_captured_chunked_prefill_replays_equal_eager(T):
    """T = 150 and T = 2565 (groups of chunks growing from one to 16): the
    preparation of later groups runs on the caller's second stream, forked
    from and joined back into the captured stream (branches of the graph)."""
    w = W.sized(W.WORKLOADS["tiny"], B=1, H=2, bf16=True)
    kc = K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.G, mean_bits=w.mean_bits,
                  b_min=w.b_min, b_max=w.b_max, chunked=1)
    xs = W.tokens(w, 0, T)
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(torch.bfloat16).cuda()
    q, k, v = bf(xs["q"]), bf(xs["k"]), bf(xs["v"])
    s, beta = dev(xs["s"]), dev(xs["beta"])
    zero = K.new_records(kc)
    rec_e, rec_g = zero.clone(), zero.clone()
    ws_e, ws_g = K.new_workspace(kc), K.new_workspace(kc)
    o_e = torch.zeros(w.B * T * w.H * w.dv, dtype=torch.float32, device="cuda")
    o_g = torch.zeros_like(o_e)
    aux = torch.cuda.Stream()
    K.kda_prefill(kc, T, 64, rec_e, q, k, v, s, beta, o_e, ws_e, aux_stream=aux)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        K.kda_prefill(kc, T, 64, zero.clone(), q, k, v, s, beta, o_g, ws_g, aux_stream=aux)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        K.kda_prefill(kc, T, 64, rec_g, q, k, v, s, beta, o_g, ws_g, aux_stream=aux)
    for rep in range(3):
        rec_g.copy_(zero)                                  # eager reset between replays
        o_g.zero_()
        g.replay()
        torch.cuda.synchronize()
        same = torch.equal(rec_e, rec_g) and torch.equal(o_e.view(torch.int32), o_g.view(torch.int32))
        say(f"prefill replay {rep}: equal {same}")
        assert same
