"""Composed prefill from per-context-unit KV states on MI355X (gfx950).

The hot path lives in libtsr.so (hand-written HIP kernels behind the C ABI
of include/tsr.h); this package is its thin Python binding plus device-buffer
plumbing.  Loading the binding fails loudly if the library was not built.
"""
from ._binding import (DTYPE_CODES, EXPORTS, TSR_ATTN_AFTER_COMPOSE, TSR_ATTN_ALL,
                       TSR_ATTN_BEFORE_COMPOSE, TSR_E4M3, TSR_BF16, TSR_ENTRY_ABSENT,
                       TSR_ENTRY_PENDING, TSR_ENTRY_READY, TSR_ERR_DEVICE,
                       TSR_ERR_INVALID_ARG, TSR_ERR_NO_SPACE, TSR_ERR_OUT_OF_RANGE,
                       TSR_ERR_STATE, TSR_ERR_UNSUPPORTED, UnitCache, tsr_copy_blocks,
                       TSR_F32, TSR_HIT, TSR_MISS, TSR_OK, TSR_SCOPE_GLOBAL, TSR_SCOPE_LOCAL,
                       Plan, RequestBatch, TsrError, lib, make_model,
                       tsr_abi_version, tsr_append_kv, tsr_assemble_kv, tsr_attn, tsr_attn_part, tsr_compose_kv, tsr_last_error,
                       tsr_peak_copy, tsr_peak_mfma, tsr_peak_mfma_flops,
                       tsr_plan_create, tsr_plan_workspace_size, tsr_prefill_attn,
                       tsr_retain_kv, tsr_rope_table_bytes, tsr_rope_table_init)

__all__ = [
    "DTYPE_CODES", "EXPORTS", "TSR_ATTN_AFTER_COMPOSE", "TSR_ATTN_ALL", "TSR_ATTN_BEFORE_COMPOSE", "TSR_E4M3", "TSR_BF16", "TSR_ENTRY_ABSENT",
    "TSR_ENTRY_PENDING", "TSR_ENTRY_READY", "TSR_ERR_DEVICE", "TSR_ERR_INVALID_ARG",
    "TSR_ERR_NO_SPACE", "TSR_ERR_OUT_OF_RANGE", "TSR_ERR_STATE", "TSR_ERR_UNSUPPORTED",
    "UnitCache", "tsr_copy_blocks", "TSR_F32", "TSR_HIT", "TSR_MISS", "TSR_OK",
    "TSR_SCOPE_GLOBAL", "TSR_SCOPE_LOCAL", "Plan", "RequestBatch", "TsrError", "lib",
    "make_model", "tsr_abi_version", "tsr_append_kv", "tsr_assemble_kv", "tsr_attn", "tsr_attn_part", "tsr_compose_kv",
    "tsr_last_error", "tsr_peak_copy", "tsr_peak_mfma", "tsr_peak_mfma_flops",
    "tsr_plan_create", "tsr_plan_workspace_size", "tsr_prefill_attn",
    "tsr_retain_kv", "tsr_rope_table_bytes", "tsr_rope_table_init",
]
