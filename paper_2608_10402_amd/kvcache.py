"""A paged KV pool on one device with the four entry points bound to it.

Convenience layer over the C ABI: owns the K/V page pools, the block table and a
grow-only workspace, and forwards each call to libtide.so.  No arithmetic happens here.
"""
from __future__ import annotations

import math

import numpy as np
import torch

from . import _lib

CANARY_BITS = 0x7FC0  # bf16 quiet NaN; unused pool slots hold it so leaks are visible


class PagedKV:
    def __init__(self, num_pages: int, num_q_heads: int, num_kv_heads: int, head_dim: int,
                 block_table, sm_scale: float | None = None, device="cuda",
                 fill_canary: bool = True):
        self.device = torch.device(device)
        self.dims = _lib.make_dims(num_q_heads, num_kv_heads, head_dim,
                                   sm_scale if sm_scale is not None else 1.0 / math.sqrt(head_dim))
        shape_k = shape_v = (num_pages, num_kv_heads, 16, head_dim)
        if fill_canary:
            self.k_pool = torch.full(shape_k, CANARY_BITS, dtype=torch.int16,
                                     device=self.device).view(torch.bfloat16)
            self.v_pool = torch.full(shape_v, CANARY_BITS, dtype=torch.int16,
                                     device=self.device).view(torch.bfloat16)
        else:
            self.k_pool = torch.empty(shape_k, dtype=torch.bfloat16, device=self.device)
            self.v_pool = torch.empty(shape_v, dtype=torch.bfloat16, device=self.device)
        self.set_block_table(block_table)
        self._ws = None

    @property
    def num_q_heads(self):
        return self.dims.num_q_heads

    @property
    def head_dim(self):
        return self.dims.head_dim

    def set_block_table(self, block_table):
        bt = torch.as_tensor(np.ascontiguousarray(block_table, dtype=np.int32))
        self.block_table = bt.to(self.device).contiguous()

    def workspace(self, nbytes: int) -> torch.Tensor:
        if self._ws is None or self._ws.numel() < nbytes:
            self._ws = _lib.alloc_workspace(max(nbytes, 1 << 16), self.device)
        return self._ws

    def append(self, k_new, v_new, prefix_lens, extend_lens, stream=None):
        ws = self.workspace(_lib.tide_workspace_size(_lib.TIDE_OP_KV_APPEND, prefix_lens,
                                                     extend_lens, self.dims))
        _lib.tide_kv_append(k_new, v_new, self.k_pool, self.v_pool, self.block_table,
                            prefix_lens, extend_lens, self.dims, ws, stream)

    def extend(self, q, prefix_lens, extend_lens, out=None, lse=None, stream=None):
        out = torch.empty_like(q) if out is None else out
        ws = self.workspace(_lib.tide_workspace_size(_lib.TIDE_OP_EXTEND, prefix_lens,
                                                     extend_lens, self.dims))
        _lib.tide_extend_attn(q, self.k_pool, self.v_pool, self.block_table, prefix_lens,
                              extend_lens, self.dims, out, lse, ws, stream)
        return out

    def extend_append(self, q, k_new, v_new, prefix_lens, extend_lens, out=None, lse=None,
                      stream=None):
        """Append the new tokens' K/V and run extend attention, fused in one call."""
        out = torch.empty_like(q) if out is None else out
        ws = self.workspace(_lib.tide_workspace_size(_lib.TIDE_OP_EXTEND, prefix_lens,
                                                     extend_lens, self.dims))
        _lib.tide_extend_append_attn(q, k_new, v_new, self.k_pool, self.v_pool, self.block_table,
                                     prefix_lens, extend_lens, self.dims, out, lse, ws, stream)
        return out

    def decode(self, q, kv_lens, num_splits: int = 0, out=None, lse=None, stream=None):
        out = torch.empty_like(q) if out is None else out
        ws = self.workspace(_lib.tide_workspace_size(_lib.TIDE_OP_DECODE, kv_lens, None,
                                                     self.dims, num_splits))
        _lib.tide_decode_attn(q, self.k_pool, self.v_pool, self.block_table, kv_lens, self.dims,
                              out, lse, num_splits, ws, stream)
        return out

    def decode_append(self, q, k_new, v_new, kv_lens, num_splits: int = 0, out=None, lse=None,
                      stream=None):
        """Append each task's newest token (position kv_lens - 1) and decode, fused."""
        out = torch.empty_like(q) if out is None else out
        ws = self.workspace(_lib.tide_workspace_size(_lib.TIDE_OP_DECODE, kv_lens, None,
                                                     self.dims, num_splits))
        _lib.tide_decode_append_attn(q, k_new, v_new, self.k_pool, self.v_pool, self.block_table,
                                     kv_lens, self.dims, out, lse, num_splits, ws, stream)
        return out

    def decode_noalloc(self, q, kv_lens, num_splits: int = 0, out=None, lse=None, stream=None):
        """Decode in the library's static device scratch: no workspace is allocated."""
        out = torch.empty_like(q) if out is None else out
        _lib.tide_decode_attn_noalloc(q, self.k_pool, self.v_pool, self.block_table, kv_lens,
                                      self.dims, out, lse, num_splits, stream)
        return out

    def decode_shared(self, q, kv_lens, group_start, shared_lens, num_splits: int = 0, out=None,
                      lse=None, stream=None):
        out = torch.empty_like(q) if out is None else out
        ws = self.workspace(_lib.tide_workspace_size_shared(kv_lens, group_start, shared_lens,
                                                            self.dims, num_splits))
        _lib.tide_decode_attn_shared(q, self.k_pool, self.v_pool, self.block_table, kv_lens,
                                     group_start, shared_lens, self.dims, out, lse, num_splits,
                                     ws, stream)
        return out

    def prefill(self, q, seq_lens, out=None, lse=None, stream=None):
        out = torch.empty_like(q) if out is None else out
        ws = self.workspace(_lib.tide_workspace_size(_lib.TIDE_OP_FULL_PREFILL, seq_lens, None,
                                                     self.dims))
        _lib.tide_full_prefill_attn(q, self.k_pool, self.v_pool, self.block_table, seq_lens,
                                    self.dims, out, lse, ws, stream)
        return out
