"""Convenience callers of the C ABI for device-resident inputs.

They allocate the output and the workspace once (PyTorch allocations) and
forward every call to libtts; no arithmetic happens here. Inputs are any
object with the fields ``q, k_cache, v_cache, k_scale, v_scale,
block_tables, seq_lens`` (device tensors) plus a ``shape`` carrying
``num_q_heads, num_kv_heads, head_dim, block_size, q_dtype, kv_dtype``.
"""

from __future__ import annotations

from typing import Optional

import numpy as np
import torch

from . import tts as _t


def desc_for(shape, scale: float = 0.0) -> _t.tts_attn_desc:
    return _t.make_desc(shape.num_q_heads, shape.num_kv_heads, shape.head_dim, shape.block_size, shape.q_dtype,
                        shape.kv_dtype, "f32", scale)


class PagedAttention:
    """``tts_paged_decode_attn`` on fixed device inputs."""

    def __init__(self, inputs, max_seq_len: int, num_blocks: int, scale: float = 0.0):
        self.x = inputs
        self.desc = desc_for(inputs.shape, scale)
        self.max_seq_len = int(max_seq_len)
        self.num_blocks = int(num_blocks)
        s = int(inputs.seq_lens.shape[0])
        dev = inputs.q.device
        self.out = torch.empty((s, inputs.shape.num_q_heads, inputs.shape.head_dim), dtype=torch.float32, device=dev)
        self.ws_bytes = _t.tts_paged_decode_workspace_size(self.desc, s, self.max_seq_len)
        self.ws = torch.zeros(max(self.ws_bytes, 1), dtype=torch.uint8, device=dev)  # partial softmax states

    def __call__(self, k_cache=None, v_cache=None, k_scale=None, v_scale=None, out=None, stream=None):
        x = self.x
        o = self.out if out is None else out
        _t.tts_paged_decode_attn(
            self.desc, int(x.seq_lens.shape[0]), x.q, x.k_cache if k_cache is None else k_cache,
            x.v_cache if v_cache is None else v_cache, x.k_scale if k_scale is None else k_scale,
            x.v_scale if v_scale is None else v_scale, x.block_tables, int(x.block_tables.shape[1]), x.seq_lens,
            self.max_seq_len, self.num_blocks, o, self.ws, self.ws_bytes, stream)
        return o


class PrefixAttention:
    """``tts_build_prefix_meta`` once, then ``tts_prefix_decode_attn`` per call."""

    def __init__(self, inputs, req_seq_offsets, block_tables_host, seq_lens_host, num_blocks: int,
                 scale: float = 0.0, stream=None):
        self.x = inputs
        self.desc = desc_for(inputs.shape, scale)
        self.num_blocks = int(num_blocks)
        self.meta = _t.tts_build_prefix_meta(np.asarray(req_seq_offsets), np.asarray(block_tables_host),
                                             np.asarray(seq_lens_host), inputs.shape.block_size, self.num_blocks,
                                             desc=self.desc, stream=stream)
        s = int(inputs.seq_lens.shape[0])
        dev = inputs.q.device
        self.out = torch.empty((s, inputs.shape.num_q_heads, inputs.shape.head_dim), dtype=torch.float32, device=dev)
        self.ws_bytes = _t.tts_prefix_decode_workspace_size(self.desc, self.meta)
        self.ws = torch.zeros(max(self.ws_bytes, 1), dtype=torch.uint8, device=dev)  # partial softmax states

    def __call__(self, k_cache=None, v_cache=None, k_scale=None, v_scale=None, out=None,
                 seq_lens: Optional[torch.Tensor] = None, stream=None):
        x = self.x
        o = self.out if out is None else out
        _t.tts_prefix_decode_attn(
            self.desc, self.meta, x.q, x.k_cache if k_cache is None else k_cache,
            x.v_cache if v_cache is None else v_cache, x.k_scale if k_scale is None else k_scale,
            x.v_scale if v_scale is None else v_scale, x.block_tables, int(x.block_tables.shape[1]),
            x.seq_lens if seq_lens is None else seq_lens, self.num_blocks, o, self.ws, self.ws_bytes, stream)
        return o
