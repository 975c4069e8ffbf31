"""Oracle of the KV-cache maintenance steps around decode (test infrastructure).

A decode step writes each beam's new token into the paged cache before
attention reads it, and the search's duplication step (DuplicateThenTruncate,
Sec. 3.1 and Alg. 1: surviving beams are duplicated, and the duplicates'
speculative tokens are truncated, Sec. 4.1) gives each child its parent's
full blocks and a private copy of the partially filled block it keeps
(copy-on-write). Plain NumPy, written from those definitions:

* ``e4m3_encode``: the OCP E4M3FN code nearest to each value, ties to the
  code with an even mantissa, saturating at +-448 -- found by searching the
  table of code values (``fp8.e4m3_table``), not by bit manipulation.
* ``append_kv``: each beam's token at position seq_len - 1 into its block;
  for fp8, the block-scale policy (set at the token that opens a block,
  raised with re-encoding of the block's earlier codes when a token exceeds
  it), every step in fp32 as the definition orders it.
* ``copy_blocks`` and ``fork_tables``: whole-block copies, and the
  children's tables (shared full blocks, one copied partial block each).
* ``truncated_lengths``: how many tokens each child keeps (Sec. 4.1,
  Alg. 1): an original keeps all of its parent's; a duplicate of a parent
  that speculated keeps the fraction clip(R + sigma z, 0, 1) of the parent's
  speculative tokens, drawn from a normal distribution with mean R (the
  truncation ratio), rounded half up. The paper gives no spread and no
  rounding: sigma (0.1 in the tests) and the rounding are readings of that
  silence; the standard-normal draws z are inputs.

The paper fixes none of the numeric policy: the fp8 scale rule is a
reading (one fp32 scale per block and tensor, as the workload generator
draws them).
"""

from __future__ import annotations

import numpy as np

from .fp8 import e4m3_table

_POS = None  # values of codes 0 .. 126 (non-negative finite, increasing)


def _pos_values() -> np.ndarray:
    global _POS
    if _POS is None:
        _POS = e4m3_table()[:127].astype(np.float64)
    return _POS


def e4m3_encode(x) -> np.ndarray:
    """uint8 codes of float32 values: nearest E4M3FN value, ties to even, +-448 saturation, NaN -> 0x7F."""
    x = np.asarray(x, dtype=np.float32)
    vals = _pos_values()
    a = np.abs(x.astype(np.float64))
    out = np.zeros(x.shape, dtype=np.uint8)
    flat_a = a.ravel()
    flat = out.ravel()
    for i, v in enumerate(flat_a):
        if np.isnan(v):
            flat[i] = 0x7F
            continue
        if v >= 448.0:
            code = 0x7E
        else:
            hi = int(np.searchsorted(vals, v, side="left"))  # first value >= v
            if hi == 0:
                code = 0
            elif vals[hi] == v:
                code = hi
            else:
                lo = hi - 1
                dl, dh = v - vals[lo], vals[hi] - v
                if dl < dh:
                    code = lo
                elif dh < dl:
                    code = hi
                else:
                    code = lo if lo % 2 == 0 else hi
        flat[i] = code
    sign = np.signbit(x).ravel() & ~np.isnan(x).ravel()
    flat[sign] |= 0x80
    return flat.reshape(x.shape)


def _bf16(bits) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _append_fp8_tensor(vals: np.ndarray, codes_prev: np.ndarray, scale: np.float32, slot: int):
    """One tensor of one token into an fp8 block.

    vals: float32 [Hkv, D] (the token); codes_prev: uint8 [Hkv, slot, D] (the
    block's earlier tokens). Returns (new token codes, earlier codes, scale)."""
    table = e4m3_table()
    f448 = np.float32(448.0)
    a = np.float32(np.max(np.abs(vals))) if vals.size else np.float32(0.0)
    s = np.float32(scale)
    if slot == 0:
        s = np.float32(a / f448) if a > 0 else np.float32(1.0)
    elif a > np.float32(f448 * np.float32(scale)):
        s = np.float32(a / f448)
        dec = table[codes_prev].astype(np.float32)
        codes_prev = e4m3_encode((dec * np.float32(scale)) / s)
    new = e4m3_encode(vals.astype(np.float32) / s)
    return new, codes_prev, s


def append_kv(kv_dtype: str, k_cache, v_cache, k_scale, v_scale, block_tables, seq_lens, k_new, v_new,
              num_blocks=None) -> None:
    """In place: every beam's token at position seq_len - 1 into its block.

    Caches: k [NB][Hkv][bs][D], v [NB][Hkv][D][bs] in storage form (float32,
    uint16 bf16 bits or uint8 codes); k_new/v_new [S][Hkv][D] (float32 for
    f32 caches, bf16 bits otherwise). Beams with seq_len 0, a block index past
    the table row or a block id outside the pool are skipped."""
    nb = k_cache.shape[0] if num_blocks is None else num_blocks
    bs = k_cache.shape[2]
    maxb = block_tables.shape[1]
    for b in range(len(seq_lens)):
        L = int(seq_lens[b])
        if L <= 0:
            continue
        t = L - 1
        lb, slot = t // bs, t % bs
        if lb >= maxb:
            continue
        p = int(block_tables[b, lb])
        if p < 0 or p >= nb:
            continue
        if kv_dtype in ("f32", "bf16"):
            k_cache[p, :, slot, :] = k_new[b]
            v_cache[p, :, :, slot] = v_new[b]
            continue
        kv = _bf16(k_new[b])
        codes, prev, s = _append_fp8_tensor(kv, k_cache[p, :, :slot, :].copy(), k_scale[p], slot)
        k_cache[p, :, :slot, :] = prev
        k_cache[p, :, slot, :] = codes
        k_scale[p] = s
        vv = _bf16(v_new[b])
        prev_v = np.transpose(v_cache[p, :, :, :slot], (0, 2, 1)).copy()  # [Hkv, slot, D]
        codes, prev_v, s = _append_fp8_tensor(vv, prev_v, v_scale[p], slot)
        v_cache[p, :, :, :slot] = np.transpose(prev_v, (0, 2, 1))
        v_cache[p, :, :, slot] = codes
        v_scale[p] = s


def copy_blocks(k_cache, v_cache, k_scale, v_scale, pairs, num_blocks=None) -> None:
    """In place: block dst := block src (K, V and fp8 scales) for each (src, dst)."""
    nb = k_cache.shape[0] if num_blocks is None else num_blocks
    for src, dst in np.asarray(pairs, dtype=np.int64).reshape(-1, 2):
        if src < 0 or src >= nb or dst < 0 or dst >= nb or src == dst:
            continue
        k_cache[dst] = k_cache[src]
        v_cache[dst] = v_cache[src]
        if k_scale is not None:
            k_scale[dst] = k_scale[src]
            v_scale[dst] = v_scale[src]


def fork_tables(parent_tables, parent_lens, block_size, child_parent, child_lens, free_ids):
    """Children's tables, the (source, destination) copies and the number of free ids used.

    Child c keeps the first child_lens[c] tokens of beam child_parent[c]: its
    full blocks are the parent's; a partial last block is a fresh id from
    free_ids (taken in order) holding a copy of the parent's block."""
    parent_tables = np.asarray(parent_tables, dtype=np.int32)
    maxb = parent_tables.shape[1]
    tables = np.full((len(child_parent), maxb), -1, dtype=np.int32)
    copies = []
    used = 0
    for c, (par, cl) in enumerate(zip(child_parent, child_lens)):
        assert 0 <= cl <= parent_lens[par]
        full = cl // block_size
        tables[c, :full] = parent_tables[par, :full]
        if cl % block_size:
            dst = int(free_ids[used])
            used += 1
            tables[c, full] = dst
            copies.append((int(parent_tables[par, full]), dst))
    return tables, np.asarray(copies, dtype=np.int32).reshape(-1, 2), used


def truncated_lengths(child_parent, parent_lens, parent_spec, ratio, sigma, z):
    """Tokens kept by each child: the first child of a parent (its original) keeps the parent's
    length; every later one keeps the non-speculative prefix plus
    floor(clip(ratio + sigma * z[c], 0, 1) * spec + 1/2) of the parent's spec speculative tokens
    (Python floats: each product and sum rounded to double in that order)."""
    out = []
    seen = set()
    for c, par in enumerate(child_parent):
        par = int(par)
        length, spec = int(parent_lens[par]), int(parent_spec[par])
        assert 0 <= spec <= length
        if par not in seen:
            seen.add(par)
            out.append(length)
            continue
        f = float(ratio) + float(sigma) * float(z[c])
        f = min(max(f, 0.0), 1.0)
        kept = min(spec, int(np.floor(f * float(spec) + 0.5)))
        out.append(length - spec + kept)
    return np.asarray(out, dtype=np.int32)
