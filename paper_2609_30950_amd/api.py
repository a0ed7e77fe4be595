"""Python binding of libkda with the C ABI's names (argument marshalling only).

Tensors are torch tensors on the current HIP device; calls are enqueued on
torch's current stream.  Every computation runs in the HIP library.
"""
import ctypes
from dataclasses import dataclass

import torch

from ._lib import KdaError, kda_config, load


@dataclass
class Config:
    B: int
    H: int
    d_k: int
    d_v: int
    group_rows: int = 64
    scope: int = 0             # 0: sequence (layer budget), 1: head
    mean_bits: float = 4.0
    b_min: int = 2
    b_max: int = 8
    ema_span: int = 64
    decay_per_head: int = 0
    state32: int = 0
    no_erase: int = 0          # 1: Mamba-2 style recurrence without erasure
    chunked: int = 0           # 1: chunked (WY/UT) prefill on MFMA
    head_units: int = 0        # 1: one width per head, block scales (Gated DeltaNet)
    weight_mode: int = 0       # allocation key variant (WEIGHT_MODES)

    def c(self):
        return kda_config(self.B, self.H, self.d_k, self.d_v, self.group_rows, self.scope,
                          float(self.mean_bits), self.b_min, self.b_max, self.ema_span,
                          self.decay_per_head, self.state32, self.no_erase,
                          self.chunked, self.head_units, self.weight_mode)


def _ptr(t, dtype=None, numel=None, name="tensor"):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise KdaError(f"{name}: expected a device tensor")
    if not t.is_contiguous():
        raise KdaError(f"{name}: expected a contiguous tensor")
    dtypes = dtype if isinstance(dtype, tuple) else (dtype,)
    if dtype is not None and t.dtype not in dtypes:
        raise KdaError(f"{name}: expected {dtype}, got {t.dtype}")
    if numel is not None and t.numel() != numel:
        raise KdaError(f"{name}: expected {numel} elements, got {t.numel()}")
    return ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _check(status):
    if status != 0:
        msg = load().kda_status_str(status).decode()
        raise KdaError(f"libkda status {status}: {msg}")


def record_bytes(cfg):
    return int(load().kda_record_bytes(ctypes.byref(cfg.c())))


def workspace_bytes(cfg):
    return int(load().kda_workspace_bytes(ctypes.byref(cfg.c())))


def new_records(cfg, device="cuda"):
    n = record_bytes(cfg)
    if n == 0:
        raise KdaError("invalid config")
    return torch.zeros(cfg.B * cfg.H * n, dtype=torch.uint8, device=device)


def new_workspace(cfg, device="cuda"):
    n = workspace_bytes(cfg)
    if n == 0:
        raise KdaError("invalid config")
    return torch.zeros(n, dtype=torch.uint8, device=device)


def _rows(cfg):
    return cfg.B * cfg.H * cfg.d_k


def kda_weights(cfg, W, C, q, s, beta, k, gamma):
    n_s = cfg.B * W * cfg.H * (1 if cfg.decay_per_head else cfg.d_k)
    _check(load().kda_weights(
        ctypes.byref(cfg.c()), W, C,
        _ptr(q, torch.float32, cfg.B * W * cfg.H * cfg.d_k, "q"), _ptr(s, torch.float32, n_s, "s"),
        _ptr(beta, torch.float32, cfg.B * W * cfg.H, "beta"),
        _ptr(k, torch.float32, cfg.B * W * cfg.H * cfg.d_k, "k"),
        _ptr(gamma, torch.float64, _rows(cfg), "gamma"), _stream()))


def kda_weights_exact(cfg, W, C, q, s, beta, k, gamma):
    n_s = cfg.B * W * cfg.H * (1 if cfg.decay_per_head else cfg.d_k)
    _check(load().kda_weights_exact(
        ctypes.byref(cfg.c()), W, C,
        _ptr(q, torch.float32, cfg.B * W * cfg.H * cfg.d_k, "q"), _ptr(s, torch.float32, n_s, "s"),
        _ptr(beta, torch.float32, cfg.B * W * cfg.H, "beta"),
        _ptr(k, torch.float32, cfg.B * W * cfg.H * cfg.d_k, "k"),
        _ptr(gamma, torch.float64, _rows(cfg), "gamma"), _stream()))


def kda_alloc_bits(cfg, gamma, R, bits, ws):
    _check(load().kda_alloc_bits(
        ctypes.byref(cfg.c()), _ptr(gamma, torch.float64, _rows(cfg), "gamma"),
        _ptr(R, torch.float32, _rows(cfg), "R"), _ptr(bits, torch.uint8, _rows(cfg), "bits"),
        _ptr(ws, torch.uint8, None, "ws"), _stream()))


def kda_pack_state(cfg, S, bits, s_hat, r, tokens_seen, records):
    _check(load().kda_pack_state(
        ctypes.byref(cfg.c()), _ptr(S, torch.float32, _rows(cfg) * cfg.d_v, "S"),
        _ptr(bits, torch.uint8, _rows(cfg), "bits"), _ptr(s_hat, torch.float64, _rows(cfg), "s_hat"),
        _ptr(r, torch.float64, _rows(cfg), "r"), int(tokens_seen),
        _ptr(records, torch.uint8, cfg.B * cfg.H * record_bytes(cfg), "records"), _stream()))


def kda_unpack_state(cfg, records, S=None, bits=None, s_hat=None, r=None):
    _check(load().kda_unpack_state(
        ctypes.byref(cfg.c()), _ptr(records, torch.uint8, cfg.B * cfg.H * record_bytes(cfg), "records"),
        _ptr(S, torch.float32, _rows(cfg) * cfg.d_v, "S"), _ptr(bits, torch.uint8, _rows(cfg), "bits"),
        _ptr(s_hat, torch.float64, _rows(cfg), "s_hat"), _ptr(r, torch.float64, _rows(cfg), "r"),
        _stream()))


def kda_step(cfg, records, q, k, v, s, beta, o, ws, gamma=None):
    n_s = cfg.B * cfg.H * (1 if cfg.decay_per_head else cfg.d_k)
    _check(load().kda_step(
        ctypes.byref(cfg.c()), _ptr(records, torch.uint8, cfg.B * cfg.H * record_bytes(cfg), "records"),
        _ptr(q, torch.float32, _rows(cfg), "q"), _ptr(k, torch.float32, _rows(cfg), "k"),
        _ptr(v, torch.float32, cfg.B * cfg.H * cfg.d_v, "v"), _ptr(s, torch.float32, n_s, "s"),
        _ptr(beta, torch.float32, cfg.B * cfg.H, "beta"),
        _ptr(gamma, torch.float64, _rows(cfg), "gamma"),
        _ptr(o, torch.float32, cfg.B * cfg.H * cfg.d_v, "o"), _ptr(ws, torch.uint8, None, "ws"),
        _stream()))


def kda_step_noalloc(cfg, records, q, k, v, s, beta, o, gamma=None):
    """kda_step on the library's own device scratch (no workspace argument,
    no device allocation)."""
    n_s = cfg.B * cfg.H * (1 if cfg.decay_per_head else cfg.d_k)
    _check(load().kda_step_noalloc(
        ctypes.byref(cfg.c()), _ptr(records, torch.uint8, cfg.B * cfg.H * record_bytes(cfg), "records"),
        _ptr(q, torch.float32, _rows(cfg), "q"), _ptr(k, torch.float32, _rows(cfg), "k"),
        _ptr(v, torch.float32, cfg.B * cfg.H * cfg.d_v, "v"), _ptr(s, torch.float32, n_s, "s"),
        _ptr(beta, torch.float32, cfg.B * cfg.H, "beta"),
        _ptr(gamma, torch.float64, _rows(cfg), "gamma"),
        _ptr(o, torch.float32, cfg.B * cfg.H * cfg.d_v, "o"), _stream()))


def kda_step_outputs(cfg, records, q, k, v, s, beta, o, ws, gamma=None):
    n_s = cfg.B * cfg.H * (1 if cfg.decay_per_head else cfg.d_k)
    _check(load().kda_step_outputs(
        ctypes.byref(cfg.c()), _ptr(records, torch.uint8, cfg.B * cfg.H * record_bytes(cfg), "records"),
        _ptr(q, torch.float32, _rows(cfg), "q"), _ptr(k, torch.float32, _rows(cfg), "k"),
        _ptr(v, torch.float32, cfg.B * cfg.H * cfg.d_v, "v"), _ptr(s, torch.float32, n_s, "s"),
        _ptr(beta, torch.float32, cfg.B * cfg.H, "beta"),
        _ptr(gamma, torch.float64, _rows(cfg), "gamma"),
        _ptr(o, torch.float32, cfg.B * cfg.H * cfg.d_v, "o"), _ptr(ws, torch.uint8, None, "ws"),
        _stream()))


def kda_step_writeback(cfg, records, ws):
    _check(load().kda_step_writeback(
        ctypes.byref(cfg.c()), _ptr(records, torch.uint8, cfg.B * cfg.H * record_bytes(cfg), "records"),
        _ptr(ws, torch.uint8, None, "ws"), _stream()))


_BF16 = (torch.bfloat16, torch.int16)   # bf16 values or their raw bit patterns


def kda_prefill(cfg, T, C, records, q, k, v, s, beta, o, ws, gamma=None, aux_stream=None):
    """aux_stream: a torch.cuda.Stream for the chunked form's preparation of
    later chunks (kda_prefill_aux), or None for one stream."""
    n_s = cfg.B * T * cfg.H * (1 if cfg.decay_per_head else cfg.d_k)
    n_qk = cfg.B * T * cfg.H * cfg.d_k
    args = [ctypes.byref(cfg.c()), int(T), int(C),
            _ptr(records, torch.uint8, cfg.B * cfg.H * record_bytes(cfg), "records"),
            _ptr(q, _BF16, n_qk, "q"), _ptr(k, _BF16, n_qk, "k"),
            _ptr(v, _BF16, cfg.B * T * cfg.H * cfg.d_v, "v"), _ptr(s, torch.float32, n_s, "s"),
            _ptr(beta, torch.float32, cfg.B * T * cfg.H, "beta"),
            _ptr(gamma, torch.float64, _rows(cfg), "gamma"),
            _ptr(o, torch.float32, cfg.B * T * cfg.H * cfg.d_v, "o"),
            _ptr(ws, torch.uint8, None, "ws"), _stream()]
    if aux_stream is None:
        _check(load().kda_prefill(*args))
    else:
        _check(load().kda_prefill_aux(*args, ctypes.c_void_p(aux_stream.cuda_stream)))


# kda_weight_mode values, in the order of the oracle's stats.WEIGHT_MODES
WEIGHT_MODES = ("ema", "range", "gamma_raw", "rel_range", "persist", "writeback",
                "no_erase_rate", "uniform", "decay")

def kda_gate_quant(cfg, T, bits, s, s_out, mode="log"):
    """Per-token decay-gate quantisation; mode "log" or "linear"."""
    n = cfg.B * T * cfg.H * cfg.d_k
    _check(load().kda_gate_quant(
        ctypes.byref(cfg.c()), int(T), int(bits), 0 if mode == "log" else 1,
        _ptr(s, torch.float32, n, "s"), _ptr(s_out, torch.float32, n, "s_out"), _stream()))


PROFILE_EVENTS = 1
PROFILE_COUNTERS = 2


def kda_profile_enable(flags=PROFILE_EVENTS):
    """flags: PROFILE_EVENTS | PROFILE_COUNTERS, or 0 to disable."""
    _check(load().kda_profile_enable(int(flags)))


def kda_profile_read(max_kinds=16):
    """{kind: (total_ms, launches)} since the previous read (synchronises)."""
    kinds = (ctypes.c_char_p * max_kinds)()
    ms = (ctypes.c_double * max_kinds)()
    cnt = (ctypes.c_int * max_kinds)()
    n = ctypes.c_int(0)
    _check(load().kda_profile_read(max_kinds, kinds, ms, cnt, ctypes.byref(n)))
    return {kinds[i].decode(): (ms[i], cnt[i]) for i in range(min(n.value, max_kinds))}


def kda_profile_counters():
    """Clip-factor evaluations (row segment x candidate) counted while
    profiling was enabled since the previous call (synchronises)."""
    n = ctypes.c_ulonglong(0)
    _check(load().kda_profile_counters(ctypes.byref(n)))
    return int(n.value)
