"""Split-KV single-query decode attention for MI355X (gfx950).

The computation lives in the HIP library libdecode_attn.so (C-ABI declared
in include/decode_attn.h); this package is its Python binding.
"""

from ._binding import (DA_OK, EXPORTS, POLICY_EVOLVED, POLICY_MI355X, POLICY_PAPER, POLICY_STREAMED, POLICY_TABLE,
                       POLICY_TABLE_STREAMED, DaPlan, DaSchedule,
                       DecodeAttnError, da_choose_splits, da_combine_splits, da_decode_attn, da_decode_attn_noalloc, da_decode_attn_paged,
                       da_decode_attn_paged_planned, da_decode_attn_planned, da_decode_attn_scheduled,
                       da_device_info, da_last_error, da_make_plan, da_model_time, da_make_schedule, da_schedule_max_bytes, da_schedule_workspace_bytes, da_split_bounds, da_split_partials,
                       da_strerror, da_workspace_bytes, load)

__all__ = [
    "DA_OK", "EXPORTS", "POLICY_EVOLVED", "POLICY_MI355X", "POLICY_PAPER", "POLICY_STREAMED", "POLICY_TABLE",
    "POLICY_TABLE_STREAMED", "DaPlan", "DaSchedule",
    "DecodeAttnError", "da_choose_splits", "da_combine_splits", "da_decode_attn", "da_decode_attn_noalloc",
    "da_decode_attn_paged",
    "da_decode_attn_paged_planned", "da_decode_attn_planned", "da_decode_attn_scheduled", "da_device_info", "da_last_error", "da_make_plan", "da_make_schedule", "da_model_time",
    "da_schedule_max_bytes", "da_schedule_workspace_bytes", "da_split_bounds", "da_split_partials", "da_strerror",
    "da_workspace_bytes", "load",
]
