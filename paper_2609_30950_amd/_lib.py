"""ctypes loader of the in-tree libkda.so (built by ``build.py``).

The product path has no fallback: if the library is missing or cannot be
loaded, every call raises.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libkda.so")


class kda_config(ctypes.Structure):
    _fields_ = [
        ("B", ctypes.c_int32), ("H", ctypes.c_int32), ("d_k", ctypes.c_int32),
        ("d_v", ctypes.c_int32), ("group_rows", ctypes.c_int32), ("scope", ctypes.c_int32),
        ("mean_bits", ctypes.c_double), ("b_min", ctypes.c_int32), ("b_max", ctypes.c_int32),
        ("ema_span", ctypes.c_int32), ("decay_per_head", ctypes.c_int32),
        ("state32", ctypes.c_int32), ("no_erase", ctypes.c_int32),
        ("chunked", ctypes.c_int32), ("head_units", ctypes.c_int32),
        ("weight_mode", ctypes.c_int32),
    ]


_P = ctypes.c_void_p
_CFG = ctypes.POINTER(kda_config)
_I32 = ctypes.c_int32
SIGNATURES = {
    "kda_record_bytes": (ctypes.c_size_t, [_CFG]),
    "kda_workspace_bytes": (ctypes.c_size_t, [_CFG]),
    "kda_status_str": (ctypes.c_char_p, [ctypes.c_int]),
    "kda_weights": (ctypes.c_int, [_CFG, _I32, _I32, _P, _P, _P, _P, _P, _P]),
    "kda_weights_exact": (ctypes.c_int, [_CFG, _I32, _I32, _P, _P, _P, _P, _P, _P]),
    "kda_alloc_bits": (ctypes.c_int, [_CFG, _P, _P, _P, _P, _P]),
    "kda_pack_state": (ctypes.c_int, [_CFG, _P, _P, _P, _P, ctypes.c_uint32, _P, _P]),
    "kda_unpack_state": (ctypes.c_int, [_CFG, _P, _P, _P, _P, _P, _P]),
    "kda_step": (ctypes.c_int, [_CFG, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "kda_step_noalloc": (ctypes.c_int, [_CFG, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "kda_step_noalloc_max_bytes": (ctypes.c_size_t, []),
    "kda_step_outputs": (ctypes.c_int, [_CFG, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "kda_step_writeback": (ctypes.c_int, [_CFG, _P, _P, _P]),
    "kda_prefill": (ctypes.c_int, [_CFG, _I32, _I32, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "kda_prefill_aux": (ctypes.c_int, [_CFG, _I32, _I32, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                       _P]),
    "kda_gate_quant": (ctypes.c_int, [_CFG, _I32, _I32, _I32, _P, _P, _P]),
    "kda_profile_enable": (ctypes.c_int, [ctypes.c_int]),
    "kda_profile_counters": (ctypes.c_int, [ctypes.POINTER(ctypes.c_ulonglong)]),
    "kda_profile_read": (ctypes.c_int, [ctypes.c_int, ctypes.POINTER(ctypes.c_char_p),
                                         ctypes.POINTER(ctypes.c_double),
                                         ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_int)]),
}

_lib = None


class KdaError(RuntimeError):
    pass


def load():
    """Load libkda.so once; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise KdaError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_30950_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib
