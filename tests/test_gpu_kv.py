"""GPU parity of the KV-maintenance calls against the oracle (bit-exact).

Append (bf16, fp32, fp8 with the block-scale policy, including blocks whose
scale grows), block copies, and a replay of a small beam search (appends,
duplication with truncation, copy-on-write copies, attention after every
step) checked against the oracle's caches and attention.
"""

from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle.attention import oracle_attn
from oracle.kv_ops import append_kv, copy_blocks, fork_tables, truncated_lengths
from paper_2509_00195_amd import (
    make_desc,
    tts_append_kv,
    tts_build_prefix_meta,
    tts_copy_blocks,
    tts_fork_prefix_meta,
    tts_fork_tables,
    tts_prefix_decode_attn,
    tts_prefix_decode_workspace_size,
    tts_truncated_lengths,
)

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
BS = 16
TOL = {"f32": 1e-4, "bf16": 1e-2, "fp8": 2e-2}


def _bf16_bits(x: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _store_dtype(kv):
    return {"f32": np.float32, "bf16": np.uint16, "fp8": np.uint8}[kv]


def _to_dev(a: np.ndarray) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(DEV)
    return torch.from_numpy(a).to(DEV)


def _to_host(t: torch.Tensor, dtype) -> np.ndarray:
    a = t.cpu().numpy()
    return a.view(np.uint16) if dtype == np.uint16 else a


def _random_cache(kv, nb, hkv, d, rng):
    if kv == "f32":
        k = rng.normal(0, 1, (nb, hkv, BS, d)).astype(np.float32)
        v = rng.normal(0, 1, (nb, hkv, d, BS)).astype(np.float32)
        return k, v, None, None
    if kv == "bf16":
        return (_bf16_bits(rng.normal(0, 1, (nb, hkv, BS, d))), _bf16_bits(rng.normal(0, 1, (nb, hkv, d, BS))),
                None, None)
    k = rng.integers(0, 256, (nb, hkv, BS, d), dtype=np.uint8)
    v = rng.integers(0, 256, (nb, hkv, d, BS), dtype=np.uint8)
    k[(k & 0x7F) == 0x7F] = 0  # no NaN codes in the starting cache
    v[(v & 0x7F) == 0x7F] = 0
    return k, v, rng.uniform(0.001, 0.01, nb).astype(np.float32), rng.uniform(0.001, 0.01, nb).astype(np.float32)


def _new_tokens(kv, s, hkv, d, rng, boost):
    x = rng.normal(0, 1, (s, hkv, d)).astype(np.float32) * boost[:, None, None]
    y = rng.normal(0, 1, (s, hkv, d)).astype(np.float32) * boost[:, None, None]
    if kv == "f32":
        return x, y
    return _bf16_bits(x), _bf16_bits(y)


@pytest.mark.parametrize("kv", ["bf16", "f32", "fp8"])
def test_append_bit_exact(kv):
    rng = np.random.default_rng({"bf16": 0, "f32": 1, "fp8": 2}[kv])
    hkv, d, nb, s, maxb = 2, 128, 64, 12, 4
    k, v, ks, vs = _random_cache(kv, nb, hkv, d, rng)
    if ks is not None:  # scales that fit the stored codes' range: 448 * 0.005 ~ 2.2
        ks[:] = vs[:] = 0.005
    ids = rng.permutation(nb).astype(np.int32)
    tables = ids[: s * maxb].reshape(s, maxb).copy()
    # slot 0 of a new block, mid-block slots, the last slot, an empty beam, a bad id, a bad block index
    lens = np.array([1, 17, 33, 5, 16, 64, 0, 9, 20, 45, 2, 65], np.int32)
    tables[7, 0] = nb + 5
    boost = np.ones(s, np.float32)
    boost[[3, 8, 9]] = 40.0  # tokens far above their block's scale: re-encoding (fp8)
    kn, vn = _new_tokens(kv, s, hkv, d, rng, boost)
    desc = make_desc(2 * hkv, hkv, d, q_dtype="f32" if kv == "f32" else "bf16", kv_dtype=kv)
    dk, dv = _to_dev(k), _to_dev(v)
    dks = _to_dev(ks) if ks is not None else None
    dvs = _to_dev(vs) if vs is not None else None
    print(f"append {kv}", flush=True)
    tts_append_kv(desc, s, _to_dev(kn), _to_dev(vn), _to_dev(tables), maxb, _to_dev(lens), nb, dk, dv, dks, dvs)
    torch.cuda.synchronize()
    append_kv(kv, k, v, ks, vs, tables, lens, kn, vn)
    dt = _store_dtype(kv)
    gk, gv = _to_host(dk, dt), _to_host(dv, dt)
    if kv == "f32":
        assert np.array_equal(gk.view(np.uint32), k.view(np.uint32)) and np.array_equal(gv.view(np.uint32),
                                                                                      v.view(np.uint32))
    else:
        assert np.array_equal(gk, k) and np.array_equal(gv, v)
    if ks is not None:
        assert np.array_equal(dks.cpu().numpy().view(np.uint32), ks.view(np.uint32))
        assert np.array_equal(dvs.cpu().numpy().view(np.uint32), vs.view(np.uint32))
        # the boosted mid-block tokens did raise their block's scale
        for b in (3, 8, 9):
            assert ks[tables[b, (lens[b] - 1) // BS]] > 0.005


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
def test_copy_blocks_bit_exact(kv):
    rng = np.random.default_rng(5)
    hkv, d, nb = 4, 128, 30
    k, v, ks, vs = _random_cache(kv, nb, hkv, d, rng)
    pairs = np.array([[3, 10], [4, 11], [3, 12], [29, 0], [5, 5], [40, 1]], np.int32)
    desc = make_desc(4 * hkv, hkv, d, kv_dtype=kv)
    dk, dv = _to_dev(k), _to_dev(v)
    dks = _to_dev(ks) if ks is not None else None
    dvs = _to_dev(vs) if vs is not None else None
    tts_copy_blocks(desc, len(pairs), _to_dev(pairs), nb, dk, dv, dks, dvs)
    torch.cuda.synchronize()
    copy_blocks(k, v, ks, vs, pairs)
    dt = _store_dtype(kv)
    assert np.array_equal(_to_host(dk, dt), k) and np.array_equal(_to_host(dv, dt), v)
    if ks is not None:
        assert np.array_equal(dks.cpu().numpy(), ks) and np.array_equal(dvs.cpu().numpy(), vs)


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
def test_beam_search_replay(kv):
    """A small search on both sides: every step appends one token per beam (a block is
    allocated when a beam crosses into a new one), every 12 steps half the beams survive and
    are duplicated: the last 0-5 tokens of each survivor count as speculative, its original
    keeps them and its duplicate keeps a share drawn around R = 0.85 (tts_truncated_lengths
    against the oracle's truncated_lengths, same draws), with copy-on-write of the kept
    partial block. After every step: caches bit-exact; every 8 steps the prefix-shared
    attention within tolerance of the oracle's, with the metadata both rebuilt in full and
    re-planned warm from the previous step's (tts_fork_prefix_meta; same trie and order)."""
    rng = np.random.default_rng(7)
    hq, hkv, d, nb, maxb, s = 8, 2, 128, 160, 8, 8
    desc = make_desc(hq, hkv, d, kv_dtype=kv)
    k, v, ks, vs = _random_cache(kv, nb, hkv, d, rng)
    free = list(range(nb))
    # a shared 40-token prompt: blocks 0..2, the third partial -> each beam its own copy
    prompt = [free.pop(0) for _ in range(3)]
    tables = np.full((s, maxb), -1, np.int32)
    lens = np.zeros(s, np.int32)
    # the prompt itself, written token by token into beam 0 (fp8 scales follow the policy)
    ptab = np.full((1, maxb), -1, np.int32)
    ptab[0, :3] = prompt
    dk, dv = _to_dev(k), _to_dev(v)
    dks = _to_dev(ks) if ks is not None else None
    dvs = _to_dev(vs) if vs is not None else None
    for t in range(40):
        kn, vn = _new_tokens(kv, 1, hkv, d, rng, np.ones(1, np.float32))
        ln = np.array([t + 1], np.int32)
        tts_append_kv(desc, 1, _to_dev(kn), _to_dev(vn), _to_dev(ptab), maxb, _to_dev(ln), nb, dk, dv, dks, dvs)
        append_kv(kv, k, v, ks, vs, ptab, ln, kn, vn)
    tables, copies, used = fork_tables(ptab, np.array([40], np.int32), BS, np.zeros(s, np.int32),
                                       np.full(s, 40, np.int32), np.array(free, np.int32))
    free = free[used:]
    lens[:] = 40
    dcp = _to_dev(copies)
    tts_copy_blocks(desc, len(copies), dcp, nb, dk, dv, dks, dvs)
    copy_blocks(k, v, ks, vs, copies)
    dt = _store_dtype(kv)
    ks0 = ks.copy() if ks is not None else None
    prev_meta = None
    for step in range(40):
        # allocate the block a beam is about to enter
        for b in range(s):
            if lens[b] % BS == 0:
                tables[b, lens[b] // BS] = free.pop(0)
        lens += 1
        # N(0,1) tokens (fp8 blocks still re-encode whenever a token's amax beats the block's
        # first; the boosted-token case is the append test's), so 1e-2 / 2e-2 apply as in parity
        kn, vn = _new_tokens(kv, s, hkv, d, rng, np.ones(s, np.float32))
        tts_append_kv(desc, s, _to_dev(kn), _to_dev(vn), _to_dev(tables), maxb, _to_dev(lens), nb, dk, dv, dks, dvs)
        append_kv(kv, k, v, ks, vs, tables, lens, kn, vn)
        if step % 12 == 11:
            surv = np.sort(rng.choice(s, s // 2, replace=False))
            cp = np.repeat(surv, 2).astype(np.int32)
            spec = np.minimum(rng.integers(0, 6, s), lens).astype(np.int32)
            z = rng.standard_normal(len(cp))
            cl = tts_truncated_lengths(cp, lens, spec, 0.85, 0.1, z)
            assert np.array_equal(cl, truncated_lengths(cp, lens, spec, 0.85, 0.1, z))
            new_t, copies, used = tts_fork_tables(tables, lens, BS, cp, cl, np.array(free, np.int32))
            ot, oc, ou = fork_tables(tables, lens, BS, cp, cl, np.array(free, np.int32))
            assert np.array_equal(new_t, ot) and np.array_equal(copies, oc) and used == ou
            free = free[used:]
            # blocks no longer referenced go back to the pool
            live = set(new_t[new_t >= 0].tolist())
            free += sorted(set(tables[tables >= 0].tolist()) - live)
            tts_copy_blocks(desc, len(copies), _to_dev(copies), nb, dk, dv, dks, dvs)
            copy_blocks(k, v, ks, vs, copies)
            tables, lens = new_t, cl
        torch.cuda.synchronize()
        assert np.array_equal(_to_host(dk, dt), k) and np.array_equal(_to_host(dv, dt), v), step
        if ks is not None:
            assert np.array_equal(dks.cpu().numpy(), ks) and np.array_equal(dvs.cpu().numpy(), vs), step
        if step % 8 == 7:
            q = _bf16_bits(rng.normal(0, 1, (s, hq, d)))
            offs = np.array([0, s], np.int32)
            metas = [tts_build_prefix_meta(offs, tables, lens, BS, nb, desc=desc)]
            if prev_meta is not None:
                metas.append(tts_fork_prefix_meta(prev_meta, offs, tables, lens, BS, nb))
                full, warm = metas[0].export(), metas[1].export()
                for key in ("perm", "seg_beam_begin", "seg_beam_end", "seg_nblocks", "tail_lblock"):
                    assert np.array_equal(full[key], warm[key]), key
            ref = oracle_attn(q, k, v, ks, vs, tables, lens, num_q_heads=hq, num_kv_heads=hkv, block_size=BS,
                              q_dtype="bf16", kv_dtype=kv)
            for meta in metas:
                ws_bytes = tts_prefix_decode_workspace_size(desc, meta)
                ws = torch.zeros(max(ws_bytes, 1), dtype=torch.uint8, device=DEV)
                out = torch.zeros((s, hq, d), dtype=torch.float32, device=DEV)
                tts_prefix_decode_attn(desc, meta, _to_dev(q), dk, dv, dks, dvs, _to_dev(tables), maxb,
                                       _to_dev(lens), nb, out, ws, ws_bytes)
                err = float(np.max(np.abs(out.cpu().numpy() - ref)))
                regrow = int(np.sum(ks != ks0)) if ks is not None else 0
                print(f"replay {kv} step {step} ({'warm' if meta is not metas[0] else 'full'} plan): err "
                      f"{err:.2e}, fp8 scales changed since the prompt: {regrow}", flush=True)
                assert err <= TOL[kv]
            prev_meta = metas[0]


@pytest.mark.parametrize("name", ["7b64", "7b_straggler", "7b64_balanced", "1p5b16"])
def test_fork_prefix_meta_at_config_scale(name):
    """The metadata of the next search iteration re-planned warm from the current one's
    (tts_fork_prefix_meta: seed 1's tree after seed 0's, same shape): the same trie, segments and
    beam order as a full build, and attention within tolerance of the oracle. (The balanced tree's plan has
    128-row wide units and the 1.5B tree's 42-row narrow units, caps a warm re-plan keeps.)"""
    from oracle.attention import oracle_attn_workload
    from paper_2509_00195_amd.runner import PrefixAttention
    from tts_synth import make_workload
    from tts_synth.device import to_device

    prev_wl = make_workload(name, 0)
    prev = PrefixAttention(to_device(prev_wl), prev_wl.req_seq_offsets, prev_wl.block_tables, prev_wl.seq_lens,
                           prev_wl.num_blocks)
    wl = make_workload(name, 1)
    x = to_device(wl)
    full = PrefixAttention(x, wl.req_seq_offsets, wl.block_tables, wl.seq_lens, wl.num_blocks)
    warm = tts_fork_prefix_meta(prev.meta, wl.req_seq_offsets, wl.block_tables, wl.seq_lens, BS, wl.num_blocks)
    ef, ew = full.meta.export(), warm.export()
    for key in ("perm", "seg_req", "seg_parent", "seg_lblock_begin", "seg_nblocks", "seg_beam_begin", "seg_beam_end",
                "tail_lblock"):
        assert np.array_equal(ef[key], ew[key]), key
    assert ef["unique_tokens"] == ew["unique_tokens"]
    ws_bytes = tts_prefix_decode_workspace_size(full.desc, warm)
    ws = torch.zeros(max(ws_bytes, 1), dtype=torch.uint8, device=DEV)
    out = torch.full_like(full.out, float("nan"))
    tts_prefix_decode_attn(full.desc, warm, x.q, x.k_cache, x.v_cache, x.k_scale, x.v_scale, x.block_tables,
                           int(x.block_tables.shape[1]), x.seq_lens, wl.num_blocks, out, ws, ws_bytes)
    ref = oracle_attn_workload(wl)
    e_warm = float(np.max(np.abs(out.cpu().numpy() - ref)))
    e_full = float(np.max(np.abs(full().cpu().numpy() - ref)))
    print(f"{name}: warm plan {warm.stats()} err {e_warm:.2e}; full plan {full.meta.stats()} err {e_full:.2e}",
          flush=True)
    assert e_warm <= TOL["bf16"] and e_full <= TOL["bf16"]
