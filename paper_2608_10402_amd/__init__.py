"""Paged-KV resume attention for AMD MI355X (gfx950): the hot path of TideRL's
Continuous Task Batching (arXiv 2608.10402) -- KV-append, extend attention over a
retained paged prefix, split-K decode attention (also over prompt prefixes shared by a
GRPO group, and with the decoded token's append fused in), full re-prefill for
comparison, and the task-batching scheduler that drives them (ctb).

The compute lives in libtide.so (hand-written HIP kernels behind the C ABI of
include/tide.h).  This package is its ctypes binding plus a small pool helper.
"""
from ._lib import (TIDE_ERR_CAPACITY, TIDE_ERR_HIP, TIDE_ERR_INVALID_ARG, TIDE_ERR_PAGE_RANGE,
                   TIDE_ERR_UNSUPPORTED, TIDE_OK, TIDE_OP_DECODE, TIDE_OP_EXTEND,
                   TIDE_OP_FULL_PREFILL, TIDE_OP_KV_APPEND, TideError, alloc_workspace, load,
                   make_dims, status_string, tide_decode_append_attn, tide_decode_attn,
                   tide_decode_attn_noalloc, NOALLOC_SCRATCH_BYTES, tide_extend_append_attn,
                   tide_decode_attn_shared, tide_dims,
                   tide_extend_attn, tide_full_prefill_attn, tide_kv_append, tide_shutdown,
                   tide_plan_info_get, tide_workspace_size, tide_workspace_size_shared)
from .kvcache import PagedKV

__all__ = ["TIDE_ERR_CAPACITY", "TIDE_ERR_HIP", "TIDE_ERR_INVALID_ARG", "TIDE_ERR_PAGE_RANGE",
           "TIDE_ERR_UNSUPPORTED", "TIDE_OK", "TIDE_OP_DECODE", "TIDE_OP_EXTEND",
           "TIDE_OP_FULL_PREFILL", "TIDE_OP_KV_APPEND", "TideError", "alloc_workspace", "load",
           "make_dims", "status_string", "tide_decode_attn", "tide_dims", "tide_extend_attn",
           "tide_full_prefill_attn", "tide_kv_append", "tide_shutdown", "tide_workspace_size",
           "tide_decode_attn_shared", "tide_workspace_size_shared", "tide_decode_append_attn",
           "tide_decode_attn_noalloc", "NOALLOC_SCRATCH_BYTES", "tide_extend_append_attn",
           "tide_plan_info_get", "PagedKV"]
