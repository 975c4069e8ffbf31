"""GPU parity of the verification attention (each beam's last q_len tokens as causal
queries over the shared prefix) against the oracle."""

from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle.attention import oracle_verify_attn
from paper_2509_00195_amd import (
    TTSError,
    make_desc,
    tts_build_prefix_meta,
    tts_build_verify_meta,
    tts_prefix_decode_attn,
    tts_prefix_decode_workspace_size,
    tts_prefix_verify_attn,
)
from tts_synth import AttnShape, CONFIGS, build_tree, make_workload, workload_from_tree
from tts_synth.device import to_device

pytestmark = pytest.mark.gpu
TOL = {"f32": 1e-4, "bf16": 1e-2, "fp8": 2e-2}


def _bits(x):
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _verify(wl, q_len, seed):
    sh = wl.shape
    rng = np.random.default_rng(seed)
    qf = rng.standard_normal((wl.num_seqs, q_len, sh.num_q_heads, sh.head_dim)).astype(np.float32)
    q = qf if sh.q_dtype == "f32" else _bits(qf)
    x = to_device(wl)
    desc = make_desc(sh.num_q_heads, sh.num_kv_heads, sh.head_dim, q_dtype=sh.q_dtype, kv_dtype=sh.kv_dtype)
    meta = tts_build_verify_meta(wl.req_seq_offsets, wl.block_tables, wl.seq_lens, q_len, 16, wl.num_blocks,
                                 desc=desc)
    wsb = tts_prefix_decode_workspace_size(desc, meta)
    ws = torch.zeros(max(wsb, 1), dtype=torch.uint8, device="cuda")
    out = torch.zeros((wl.num_seqs, q_len, sh.num_q_heads, sh.head_dim), dtype=torch.float32, device="cuda")
    dq = torch.from_numpy(q.view(np.int16) if q.dtype == np.uint16 else q).cuda()
    tts_prefix_verify_attn(desc, meta, dq, x.k_cache, x.v_cache, x.k_scale, x.v_scale, x.block_tables,
                           int(x.block_tables.shape[1]), x.seq_lens, wl.num_blocks, out, ws, wsb)
    got = out.cpu().numpy()
    ref = oracle_verify_attn(q, wl.k_cache, wl.v_cache, wl.k_scale, wl.v_scale, wl.block_tables, wl.seq_lens,
                             q_len, num_q_heads=sh.num_q_heads, num_kv_heads=sh.num_kv_heads, block_size=16,
                             q_dtype=sh.q_dtype, kv_dtype=sh.kv_dtype)
    return got, ref, meta, desc, x


@pytest.mark.parametrize("name,q_len", [("1p5b16", 2), ("1p5b16", 8), ("7b64", 4), ("tiny", 3)])
def test_verify_parity(name, q_len):
    wl = make_workload(name, 0)
    got, ref, _, _, _ = _verify(wl, q_len, 1)
    e = float(np.max(np.abs(got - ref)))
    print(f"verify {name} q_len {q_len}: err {e:.2e}", flush=True)
    assert np.isfinite(got).all() and e <= TOL[wl.shape.kv_dtype]


def test_verify_parity_fp8():
    wl = workload_from_tree(AttnShape(12, 2, 128, 16, "bf16", "fp8"), build_tree(CONFIGS["1p5b16"], 2), 2)
    got, ref, _, _, _ = _verify(wl, 5, 2)
    assert float(np.max(np.abs(got - ref))) <= TOL["fp8"]


def test_verify_one_query_equals_decode_and_decode_refuses_verify_meta():
    wl = make_workload("1p5b16", 1)
    got, ref, meta, desc, x = _verify(wl, 1, 3)
    assert float(np.max(np.abs(got - ref))) <= TOL["bf16"]
    vmeta = tts_build_verify_meta(wl.req_seq_offsets, wl.block_tables, wl.seq_lens, 2, 16, wl.num_blocks, desc=desc)
    wsb = tts_prefix_decode_workspace_size(desc, vmeta)
    ws = torch.zeros(max(wsb, 1), dtype=torch.uint8, device="cuda")
    out = torch.zeros((wl.num_seqs, 2, 12, 128), dtype=torch.float32, device="cuda")
    q = torch.zeros((wl.num_seqs, 2, 12, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(TTSError):
        tts_prefix_decode_attn(desc, vmeta, q, x.k_cache, x.v_cache, None, None, x.block_tables,
                               int(x.block_tables.shape[1]), x.seq_lens, wl.num_blocks, out, ws, wsb)


def test_verify_meta_rejects_short_beams():
    wl = make_workload("tiny", 0)
    lens = wl.seq_lens.copy()
    lens[0] = 2
    with pytest.raises(TTSError):
        tts_build_verify_meta(wl.req_seq_offsets, wl.block_tables, lens, 3, 16, wl.num_blocks)
