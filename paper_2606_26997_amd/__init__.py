"""MI355X (gfx950) group decode attention over a paged, group-shared KV cache.

The computation lives in ``librp.so`` (HIP kernels behind a C ABI declared in
``include/rp.h``): the decode attention, the KV append, the shared-prefix
prefill, the decode step's q/k preparation and the GRPO group advantages, plus
a host-side simulation of the paper's rollout/training schedulers. This package is its Python binding. Calls raise if the library has not been built.
"""
from ._binding import (EXPORTED, LIB_PATH, RP_ERR_HIP, RP_ERR_INVALID_ARG, RP_ERR_LAYOUT,
                       RP_ERR_UNSUPPORTED, RP_ERR_WORKSPACE, RP_KV_BF16, RP_KV_FP8_E4M3, RP_NOALLOC_SCRATCH_BYTES, RP_OK,
                       RP_SELFTEST_SHAPES, RP_STREAM_READ_SINK_WORDS,
                       RpError, RpGroupLayout, RpPagedKV, RpPrefillLayout, combine_parts,
                       decode_qk_prep, decode_qk_prep_plan, grpo_advantage, group_decode_attn, group_decode_attn_noalloc,
                       group_decode_attn_workspace_size, group_layout,
                       kv_append, last_error, load, lse_combine, paged_kv, plan, attn_parts,
                       prefill, prefill_attn, prefill_kv_write, prefill_layout, status_string,
                       sched_simulate, selftest_mfma, stream_read, validate_layout)
from .batch import DeviceBatch, PrefillBatch

__all__ = ["EXPORTED", "LIB_PATH", "RP_OK", "RP_ERR_INVALID_ARG", "RP_ERR_UNSUPPORTED",
           "RP_ERR_WORKSPACE", "RP_ERR_HIP", "RP_NOALLOC_SCRATCH_BYTES", "RP_ERR_LAYOUT", "RP_KV_BF16", "RP_KV_FP8_E4M3",
           "RpError", "RpPagedKV", "RpGroupLayout", "load", "status_string", "last_error",
           "paged_kv", "group_layout", "kv_append", "group_decode_attn_workspace_size",
           "group_decode_attn", "group_decode_attn_noalloc", "lse_combine", "plan", "attn_parts", "combine_parts",
           "validate_layout", "DeviceBatch", "RpPrefillLayout", "prefill_layout", "prefill_kv_write", "prefill",
           "prefill_attn", "PrefillBatch", "decode_qk_prep", "decode_qk_prep_plan", "sched_simulate", "grpo_advantage",
           "RP_SELFTEST_SHAPES", "selftest_mfma", "RP_STREAM_READ_SINK_WORDS", "stream_read"]
