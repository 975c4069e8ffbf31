"""Oracle decode attention over a paged KV cache (fp32, plain definition).

What is computed (single-token decode of every beam, Sec. 3.1 "Generation"
over the paged KV cache of the serving substrate, Sec. 2.3): for beam ``b``
with ``L = seq_lens[b]`` cached tokens and query head ``h`` of a GQA model
with ``g = Hq / Hkv`` query heads per KV head,

    kvh     = h // g
    K_b[t]  = k_cache[block_tables[b][t // bs], kvh, t % bs, :]        t < L
    V_b[t]  = v_cache[block_tables[b][t // bs], kvh, :, t % bs]
    s_t     = scale * <q[b, h], K_b[t]>,  scale = 1/sqrt(D) unless given
    out     = sum_t softmax(s)_t V_b[t]   (max-subtracted softmax)
    L == 0  -> out = 0

Sharing KV blocks between beams changes which bytes a kernel reads, not this
result, so the oracle simply materialises each beam's full sequence (no
tries, no tiling, no online softmax). Storage decoding: bf16 bits are
widened to fp32 exactly; fp8 codes are decoded with the E4M3FN table and
multiplied by their block's fp32 scale; fp32 is used as is.

Layouts: ``q`` [S, Hq, D]; ``k_cache`` [NB, Hkv, bs, D]; ``v_cache``
[NB, Hkv, D, bs]; ``block_tables`` [S, max_blocks] (entries past
``ceil(L / bs)`` are ignored); ``out`` [S, Hq, D] fp32.
"""

from __future__ import annotations

import math
from typing import Optional

import numpy as np

from .fp8 import e4m3_table

_E4M3 = None


def decode_bf16(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float32, exactly (bf16 is fp32's top half)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _decode(store: np.ndarray, dtype: str) -> np.ndarray:
    global _E4M3
    if dtype == "f32":
        return np.asarray(store, dtype=np.float32)
    if dtype == "bf16":
        return decode_bf16(store)
    if dtype == "fp8":
        if _E4M3 is None:
            _E4M3 = e4m3_table()
        return _E4M3[np.asarray(store, dtype=np.uint8)]
    raise ValueError(f"unknown dtype {dtype}")


def _beam_kv(k_cache, v_cache, k_scale, v_scale, ids, length, kv_dtype):
    """Materialise one beam's K and V as fp32 [Hkv, L, D]."""
    kb = _decode(k_cache[ids], kv_dtype)  # [n, Hkv, bs, D]
    vb = _decode(v_cache[ids], kv_dtype)  # [n, Hkv, D, bs]
    if kv_dtype == "fp8":
        kb = kb * k_scale[ids].astype(np.float32)[:, None, None, None]
        vb = vb * v_scale[ids].astype(np.float32)[:, None, None, None]
    n, hkv, bs, d = kb.shape
    k_seq = kb.transpose(1, 0, 2, 3).reshape(hkv, n * bs, d)[:, :length]
    v_seq = vb.transpose(1, 0, 3, 2).reshape(hkv, n * bs, d)[:, :length]
    return k_seq, v_seq


def oracle_attn_row(
    q: np.ndarray,
    k_cache: np.ndarray,
    v_cache: np.ndarray,
    k_scale: Optional[np.ndarray],
    v_scale: Optional[np.ndarray],
    block_tables: np.ndarray,
    seq_lens: np.ndarray,
    b: int,
    *,
    num_q_heads: int,
    num_kv_heads: int,
    block_size: int,
    q_dtype: str,
    kv_dtype: str,
    scale: Optional[float] = None,
) -> np.ndarray:
    """Attention output of one beam, all query heads: float32 [Hq, D]."""
    d = q.shape[-1]
    g = num_q_heads // num_kv_heads
    sc = np.float32(1.0 / math.sqrt(d) if scale is None or scale <= 0 else scale)
    out = np.zeros((num_q_heads, d), dtype=np.float32)
    length = int(seq_lens[b])
    if length == 0:
        return out
    nblk = -(-length // block_size)
    ids = np.asarray(block_tables[b, :nblk], dtype=np.int64)
    k_seq, v_seq = _beam_kv(k_cache, v_cache, k_scale, v_scale, ids, length, kv_dtype)
    qb = _decode(q[b], q_dtype)
    for h in range(num_q_heads):
        kvh = h // g
        s = (k_seq[kvh] @ qb[h]).astype(np.float32) * sc
        m = s.max()
        p = np.exp(s - m)
        l = p.sum(dtype=np.float32)
        out[h] = (p @ v_seq[kvh]) / l
    return out


def oracle_attn(
    q: np.ndarray,
    k_cache: np.ndarray,
    v_cache: np.ndarray,
    k_scale: Optional[np.ndarray],
    v_scale: Optional[np.ndarray],
    block_tables: np.ndarray,
    seq_lens: np.ndarray,
    *,
    num_q_heads: int,
    num_kv_heads: int,
    block_size: int,
    q_dtype: str,
    kv_dtype: str,
    scale: Optional[float] = None,
    beams=None,
) -> np.ndarray:
    """Attention output for every beam (or the listed ``beams``): float32 [S, Hq, D]."""
    s_all = seq_lens.shape[0]
    rows = range(s_all) if beams is None else beams
    out = np.zeros((s_all, num_q_heads, q.shape[-1]), dtype=np.float32)
    for b in rows:
        out[b] = oracle_attn_row(
            q, k_cache, v_cache, k_scale, v_scale, block_tables, seq_lens, b,
            num_q_heads=num_q_heads, num_kv_heads=num_kv_heads, block_size=block_size,
            q_dtype=q_dtype, kv_dtype=kv_dtype, scale=scale,
        )
    return out


def oracle_attn_workload(wl, scale=None, beams=None) -> np.ndarray:
    """Convenience wrapper taking a ``tts_synth.Workload``."""
    sh = wl.shape
    return oracle_attn(
        wl.q, wl.k_cache, wl.v_cache, wl.k_scale, wl.v_scale, wl.block_tables, wl.seq_lens,
        num_q_heads=sh.num_q_heads, num_kv_heads=sh.num_kv_heads, block_size=sh.block_size,
        q_dtype=sh.q_dtype, kv_dtype=sh.kv_dtype, scale=scale, beams=beams,
    )


def oracle_verify_attn(
    q: np.ndarray,
    k_cache: np.ndarray,
    v_cache: np.ndarray,
    k_scale: Optional[np.ndarray],
    v_scale: Optional[np.ndarray],
    block_tables: np.ndarray,
    seq_lens: np.ndarray,
    q_len: int,
    *,
    num_q_heads: int,
    num_kv_heads: int,
    block_size: int,
    q_dtype: str,
    kv_dtype: str,
    scale: Optional[float] = None,
    beams=None,
) -> np.ndarray:
    """Verification attention (LookAhead Verification, Sec. 4.1: a verifier pass over a path's
    current and speculative steps at once): each beam's last ``q_len`` cached tokens are
    queries, query i at position p_i = L - q_len + i attending causally to tokens 0 .. p_i.

    q: [S, q_len, Hq, D]; returns float32 [S, q_len, Hq, D]."""
    s_all = seq_lens.shape[0]
    d = q.shape[-1]
    g = num_q_heads // num_kv_heads
    sc = np.float32(1.0 / math.sqrt(d) if scale is None or scale <= 0 else scale)
    out = np.zeros((s_all, q_len, num_q_heads, d), dtype=np.float32)
    for b in (range(s_all) if beams is None else beams):
        length = int(seq_lens[b])
        assert length >= q_len
        nblk = -(-length // block_size)
        ids = np.asarray(block_tables[b, :nblk], dtype=np.int64)
        k_seq, v_seq = _beam_kv(k_cache, v_cache, k_scale, v_scale, ids, length, kv_dtype)
        qb = _decode(q[b], q_dtype)  # [q_len, Hq, D]
        for i in range(q_len):
            visible = length - q_len + i + 1  # tokens 0 .. p_i
            for h in range(num_q_heads):
                kvh = h // g
                s = (k_seq[kvh, :visible] @ qb[i, h]).astype(np.float32) * sc
                p = np.exp(s - s.max())
                out[b, i, h] = (p @ v_seq[kvh, :visible]) / p.sum(dtype=np.float32)
    return out
