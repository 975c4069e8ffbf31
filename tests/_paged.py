"""Test helpers: scatter dense per-beam K/V sequences into a paged cache.

The scatter is written from the storage layout alone (K token-major and V
dim-major inside a block), independently of the oracle's gather, so that
comparing the oracle on the paged cache with a dense float64 reference pins
the oracle's indexing as well as its arithmetic.
"""

from __future__ import annotations

import numpy as np
import torch


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (RNE) and return the value as float64."""
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).double().numpy()


def bf16_bits(x: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def scatter_paged(ks, vs, block_size, rng, *, pool_extra=3, fill=np.nan, dtype="f32", table_fill=-1):
    """Place dense sequences ``ks[b]``/``vs[b]`` ([Hkv, L_b, D] float) into a paged cache.

    Returns (k_cache, v_cache, block_tables, seq_lens) with fresh, randomly
    permuted physical blocks per beam; unused slots hold ``fill``.
    """
    s = len(ks)
    hkv, _, d = ks[0].shape
    lens = np.array([k.shape[1] for k in ks], dtype=np.int32)
    nblk = [-(-int(L) // block_size) for L in lens]
    total = sum(nblk)
    pool = total + pool_extra
    ids = rng.permutation(pool)
    k_cache = np.full((pool, hkv, block_size, d), fill, dtype=np.float32)
    v_cache = np.full((pool, hkv, d, block_size), fill, dtype=np.float32)
    tables = np.full((s, max(nblk + [1]) + 1), table_fill, dtype=np.int32)
    nxt = 0
    for b in range(s):
        for j in range(nblk[b]):
            p = int(ids[nxt])
            nxt += 1
            tables[b, j] = p
            for t in range(j * block_size, min(int(lens[b]), (j + 1) * block_size)):
                slot = t - j * block_size
                k_cache[p, :, slot, :] = ks[b][:, t, :]
                v_cache[p, :, :, slot] = vs[b][:, t, :]
    if dtype == "bf16":
        k_cache, v_cache = bf16_bits(k_cache), bf16_bits(v_cache)
    return k_cache, v_cache, tables, lens


def dense_reference(q, ks, vs, scale=None):
    """float64 attention of each beam on its dense sequence via torch SDPA.

    ``q``: [S, Hq, D]; ``ks[b]``/``vs[b]``: [Hkv, L_b, D]. GQA by repeating
    each KV head over its ``Hq / Hkv`` consecutive query heads.
    """
    s, hq, d = q.shape
    out = np.zeros((s, hq, d), dtype=np.float64)
    for b in range(s):
        L = ks[b].shape[1]
        if L == 0:
            continue
        g = hq // ks[b].shape[0]
        k = torch.from_numpy(np.asarray(ks[b], dtype=np.float64)).repeat_interleave(g, dim=0)
        v = torch.from_numpy(np.asarray(vs[b], dtype=np.float64)).repeat_interleave(g, dim=0)
        qq = torch.from_numpy(np.asarray(q[b], dtype=np.float64))[:, None, :]
        o = torch.nn.functional.scaled_dot_product_attention(qq[None], k[None], v[None], scale=scale)
        out[b] = o[0, :, 0, :].numpy()
    return out
