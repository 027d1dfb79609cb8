"""Preference-packing hot path for AMD MI355X (gfx950).

The computation lives in libppattn.so (HIP kernels + host planner, C ABI in
include/pp_attn.h); `binding` marshals torch tensors into it, `workload` draws
seeded synthetic packed batches.
"""
from .binding import (PPError, pp_attn_bwd, pp_attn_fwd, pp_dpo_loss, pp_pack_export,  # noqa: F401
                      pp_seq_logprob, pp_timing_enable, pp_timing_get, pp_timing_reset,
                      pp_workspace_size)
from .workload import BY_NAME, CONFIGS, Pack, config_pack, make_pack  # noqa: F401

__version__ = "0.1.0"
