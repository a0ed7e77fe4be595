"""MI355X-native KDA recurrence with a decay-aware mixed-precision state.

Python binding of libkda (HIP, gfx950).  See include/kda.h for the C ABI.
"""
from ._lib import KdaError, load  # noqa: F401
from .api import (Config, kda_alloc_bits, kda_gate_quant, kda_pack_state, kda_prefill, kda_profile_enable,  # noqa: F401,E501
                  kda_profile_counters, kda_profile_read, kda_step, kda_step_noalloc, kda_step_outputs,
                  kda_step_writeback,
                  kda_unpack_state, kda_weights, kda_weights_exact, new_records, new_workspace, record_bytes,
                  workspace_bytes)
