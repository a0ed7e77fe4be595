"""Helpers shared by the GPU parity tests: host<->device copies and oracle
records in the library's byte layout.  Uses the oracle only on the CPU side."""
import sys

import numpy as np
import torch

from oracle import record, stats


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def say(*msg):
    print(*msg, flush=True)
    sys.stdout.flush()


def state_to_bytes(st, dk, dv, bmax):
    B, H = st["ntok"].shape
    slot = record.record_bytes(dk, dv, bmax)
    out = np.zeros((B, H, slot), np.uint8)
    for b in range(B):
        for h in range(H):
            out[b, h] = record.pack(st["ntok"][b, h], st["widths"][b, h], st["scale"][b, h],
                                    st["z"][b, h], st["r16"][b, h], st["codes"][b, h], dk, dv, bmax)
    return out.reshape(-1)


def bytes_to_state(buf, B, H, dk, dv, bmax):
    slot = record.record_bytes(dk, dv, bmax)
    buf = np.asarray(buf, np.uint8).reshape(B, H, slot)
    fs = [[record.unpack(buf[b, h], dk, dv, bmax) for h in range(H)] for b in range(B)]
    st = {k: np.stack([np.stack([fs[b][h][k] for h in range(H)]) for b in range(B)])
          for k in ("widths", "scale", "z", "r16", "codes")}
    st["ntok"] = np.array([[fs[b][h]["ntok"] for h in range(H)] for b in range(B)], np.int64)
    return st


def meaningful_equal(a, b, B, H, dk, dv, bmax):
    slot = record.record_bytes(dk, dv, bmax)
    a = np.asarray(a, np.uint8).reshape(B * H, slot)
    b = np.asarray(b, np.uint8).reshape(B * H, slot)
    bad = []
    for i in range(B * H):
        ma = record.meaningful(a[i], dk, dv, bmax)
        mb = record.meaningful(b[i], dk, dv, bmax)
        if ma.size != mb.size or not np.array_equal(ma, mb):
            bad.append(i)
    return bad


def _up256(x):
    return (x + 255) // 256 * 256


def ws_state32(ws, w):
    """float32 state after the last write-back interval, read from the
    workspace (views in the order the library lays them out: EMA keys,
    rate codes, widths, then the float32 state)."""
    rows = w.B * w.H * w.dk
    zr = _up256(rows * 8)
    bits = _up256(zr + rows * 4)
    s32 = _up256(bits + rows)
    a = host(ws[s32:s32 + rows * w.dv * 4]).view(np.float32)
    return a.reshape(w.B, w.H, w.dk, w.dv)
