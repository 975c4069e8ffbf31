"""GPU parity: libtts (through its C ABI) against the CPU oracle.

Tolerances (max abs error of the fp32 outputs): 1e-4 for fp32 KV, 1e-2 for
bf16 KV (bf16 operands, fp32 accumulation, probabilities rounded to bf16
for the value product), 2e-2 for fp8 KV.
"""

import dataclasses

import numpy as np
import pytest
import torch

from oracle.attention import decode_bf16, oracle_attn_workload
from oracle.prefix_meta import oracle_prefix_meta
from paper_2509_00195_amd import TTSError
from paper_2509_00195_amd.runner import PagedAttention, PrefixAttention
from tts_synth import CONFIGS, AttnShape, BeamTree, make_workload, workload_from_tree
from tts_synth.device import to_device
from tests._paged import bf16_bits

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 1e-2, "fp8": 2e-2}


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    torch.cuda.set_device(0)


def runners(wl, lens_for_meta=None):
    x = to_device(wl)
    paged = PagedAttention(x, wl.max_seq_len, wl.num_blocks)
    pref = PrefixAttention(x, wl.req_seq_offsets, wl.block_tables,
                           wl.seq_lens if lens_for_meta is None else lens_for_meta, wl.num_blocks)
    return x, paged, pref


def outputs(wl, lens_for_meta=None):
    x, paged, pref = runners(wl, lens_for_meta)
    op = paged().cpu().numpy()
    ox = pref().cpu().numpy()
    torch.cuda.synchronize()
    return op, ox


def err(a, b, rows=None):
    if rows is not None:
        a, b = a[rows], b[rows]
    return float(np.max(np.abs(a.astype(np.float64) - b.astype(np.float64)))) if a.size else 0.0


@pytest.mark.parametrize("name", ["tiny", "1p5b16", "7b64"])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_parity_configs(name, seed):
    wl = make_workload(name, seed)
    ref = oracle_attn_workload(wl)
    op, ox = outputs(wl)
    tol = TOL[wl.shape.kv_dtype]
    print(f"{name} seed {seed}: paged {err(op, ref):.2e} prefix {err(ox, ref):.2e} (tol {tol})", flush=True)
    assert np.isfinite(op).all() and np.isfinite(ox).all()
    assert err(op, ref) <= tol
    assert err(ox, ref) <= tol


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_parity_straggler(seed):
    wl = make_workload("7b_straggler", seed)
    ref = oracle_attn_workload(wl)
    op, ox = outputs(wl)
    print(f"straggler seed {seed}: paged {err(op, ref):.2e} prefix {err(ox, ref):.2e}", flush=True)
    assert np.isfinite(op).all() and np.isfinite(ox).all()
    assert err(op, ref) <= TOL["bf16"] and err(ox, ref) <= TOL["bf16"]


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_parity_balanced_tree(seed):
    """The low-sharing balanced tree (long private tails)."""
    wl = make_workload("7b64_balanced", seed)
    ref = oracle_attn_workload(wl)
    op, ox = outputs(wl)
    print(f"balanced seed {seed}: paged {err(op, ref):.2e} prefix {err(ox, ref):.2e}", flush=True)
    assert np.isfinite(op).all() and np.isfinite(ox).all()
    assert err(op, ref) <= TOL["bf16"] and err(ox, ref) <= TOL["bf16"]


@pytest.mark.parametrize("kv,seed", [("fp8", 0), ("fp8", 1), ("fp8", 2), ("bf16", 0)])
def test_parity_longchain(kv, seed):
    """The long-chain batch at full size (its wide units hold up to 128 blocks, ids 64.. in the
    info words), every beam against the oracle: fp8 as configured (seeds 0-2) and bf16."""
    cfg = CONFIGS["7b_longchain_fp8"]
    if kv != "fp8":
        cfg = dataclasses.replace(cfg, shape=dataclasses.replace(cfg.shape, kv_dtype=kv))
    wl = make_workload(cfg, seed)
    op, ox = outputs(wl)
    assert np.isfinite(op).all() and np.isfinite(ox).all()
    ref = oracle_attn_workload(wl)
    print(f"longchain {kv} seed {seed} (all {wl.num_seqs} beams): paged {err(op, ref):.2e} "
          f"prefix {err(ox, ref):.2e}", flush=True)
    assert err(op, ref) <= TOL[kv] and err(ox, ref) <= TOL[kv]


def test_run_to_run_deterministic():
    wl = make_workload("7b64", 1)
    x, paged, pref = runners(wl)
    a1, b1 = paged().clone(), pref().clone()
    a2, b2 = paged().clone(), pref().clone()
    assert torch.equal(a1, a2) and torch.equal(b1, b2)


def _duplicate_beams(wl, picks):
    """Append exact copies (table, length, query) of the beams in `picks` to the last request."""
    offs = wl.req_seq_offsets.copy()
    offs[-1] += len(picks)
    return dataclasses.replace(
        wl, block_tables=np.vstack([wl.block_tables, wl.block_tables[picks]]),
        seq_lens=np.concatenate([wl.seq_lens, wl.seq_lens[picks]]), q=np.concatenate([wl.q, wl.q[picks]]),
        req_seq_offsets=offs)


def _max_abs_v(wl, b):
    """Largest |value| any partial state of beam b can hold: max over the beam's V rows."""
    bs = wl.shape.block_size
    nb = -(-int(wl.seq_lens[b]) // bs)
    ids = wl.block_tables[b, :nb]
    v = decode_bf16(wl.v_cache[ids])  # [nb][Hkv][D][bs]
    last = int(wl.seq_lens[b]) - (nb - 1) * bs
    vals = [v[:-1].ravel(), v[-1][..., :last].ravel()]
    return float(np.max(np.abs(np.concatenate(vals))))


def test_identical_beams_agree():
    """Beams with identical tables, lengths and queries get the same rows. The paged path computes
    them with the same instruction sequence (bit-identical); the prefix path may place the two
    beams' private blocks in different lanes of a block pair or on different waves, so their fp32
    sums associate differently, and it stores partial states as fp16 elements of at most 1 in
    magnitude times a power-of-two row scale 2^e with 2^(e-1) <= max |element|: each partial adds
    at most 2^-12 * 2^e <= 2^-11 * max |partial row| of rounding, which the merge's weights (summing
    to 1) carry into the output. Two such rows therefore agree within 2^-10 of the largest partial
    element, far inside the parity tolerance."""
    wl = make_workload("1p5b16", 0)
    picks = [0, 5, 9]
    wl2 = _duplicate_beams(wl, picks)
    op, ox = outputs(wl2)
    s = wl.num_seqs
    for i, b in enumerate(picks):
        assert np.array_equal(op[b], op[s + i])
        # the largest partial element is bounded by max |v| over the beam's values; the output
        # row's own max is a lower bound of it, so use the beam's value range directly
        assert err(ox[b], ox[s + i]) <= 2.0 ** -10 * _max_abs_v(wl2, b)
    ref = oracle_attn_workload(wl2)
    assert err(ox, ref) <= TOL["bf16"]


def test_physical_permutation_bit_exact():
    wl = make_workload("1p5b16", 2)
    op, ox = outputs(wl)
    pi = np.random.default_rng(5).permutation(wl.num_blocks)
    kc = np.empty_like(wl.k_cache)
    vc = np.empty_like(wl.v_cache)
    kc[pi] = wl.k_cache
    vc[pi] = wl.v_cache
    tables = np.where(wl.block_tables >= 0, pi[np.maximum(wl.block_tables, 0)], -1).astype(np.int32)
    wl2 = dataclasses.replace(wl, k_cache=kc, v_cache=vc, block_tables=tables)
    op2, ox2 = outputs(wl2)
    assert np.array_equal(op, op2) and np.array_equal(ox, ox2)


def _edge_tree():
    """One request whose beams have lengths 0, 1, 15, 16, 17, 32, 33 and share prefixes,
    a second request with a single beam, a third that is empty."""
    t = BeamTree(block_size=16)
    base = [t.new_alloc() for _ in range(3)]  # 48 tokens of shared prefix
    specs = [(0, 0), (1, 1), (15, 1), (16, 1), (17, 2), (32, 2), (33, 3), (48, 3), (48, 3), (50, 4)]
    for L, nshared in specs:
        blocks = list(base[:min(nshared, L // 16)])
        while len(blocks) * 16 < L:
            blocks.append(t.new_alloc())
        t.beam_allocs.append(blocks)
        t.beam_lens.append(L)
        t.beam_parent.append(-1)
    t.req_offsets.append(len(t.beam_lens))
    t.beam_allocs.append([t.new_alloc() for _ in range(7)])
    t.beam_lens.append(100)
    t.beam_parent.append(-1)
    t.req_offsets.append(len(t.beam_lens))
    t.req_offsets.append(len(t.beam_lens))  # empty request
    return t


@pytest.mark.parametrize("kv", ["bf16", "f32", "fp8"])
def test_edge_lengths(kv):
    shape = AttnShape(12, 2, 128, 16, "f32" if kv == "f32" else "bf16", kv)
    wl = workload_from_tree(shape, _edge_tree(), 3, shuffle=False)
    ref = oracle_attn_workload(wl)
    op, ox = outputs(wl)
    assert np.all(op[0] == 0) and np.all(ox[0] == 0)  # seq_len 0
    assert err(op, ref) <= TOL[kv] and err(ox, ref) <= TOL[kv]
    m = oracle_prefix_meta(wl.req_seq_offsets, wl.block_tables, wl.seq_lens, 16)
    assert m["num_segs"] >= 2


def test_head_dim_64_bf16():
    cfg = CONFIGS["1p5b16"]
    from tts_synth import build_tree
    wl = workload_from_tree(AttnShape(16, 2, 64, 16, "bf16", "bf16"), build_tree(cfg, 4), 4)
    ref = oracle_attn_workload(wl)
    op, ox = outputs(wl)
    assert err(op, ref) <= TOL["bf16"] and err(ox, ref) <= TOL["bf16"]


def _many_rows_workload(kv, head_dim):
    """320 beams x 16 query heads: more than 4096 (beam, query head) rows, so
    the merge runs its many-row kernel (sixteen lanes per row); sequences past
    1024 tokens give the paged path split partials too."""
    from tts_synth import ReqSpec, WorkloadConfig

    shape = AttnShape(16, 4, head_dim, 16, "f32" if kv == "f32" else "bf16", kv)
    spec = ReqSpec(beams=40, branch=4, prompt=(512, 512), step=(64, 256), max_len=1400)
    wl = make_workload(WorkloadConfig("many_rows", shape, (spec,) * 8), 5)
    assert len(wl.seq_lens) * shape.num_q_heads > 4096 and wl.max_seq_len > 1024
    return wl


@pytest.mark.parametrize("kv,head_dim", [("f32", 64), ("f32", 128), ("bf16", 64), ("fp8", 128)])
def test_many_rows_merge(kv, head_dim):
    wl = _many_rows_workload(kv, head_dim)
    ref = oracle_attn_workload(wl)
    op, ox = outputs(wl)
    tol = TOL[kv]
    print(f"many rows {kv} D{head_dim}: paged {err(op, ref):.2e} prefix {err(ox, ref):.2e}", flush=True)
    assert np.isfinite(op).all() and np.isfinite(ox).all()
    assert err(op, ref) <= tol and err(ox, ref) <= tol


def test_scale_override():
    wl = make_workload("tiny", 1)
    x = to_device(wl)
    pref = PrefixAttention(x, wl.req_seq_offsets, wl.block_tables, wl.seq_lens, wl.num_blocks, scale=0.37)
    paged = PagedAttention(x, wl.max_seq_len, wl.num_blocks, scale=0.37)
    ref = oracle_attn_workload(wl, scale=0.37)
    assert err(pref().cpu().numpy(), ref) <= 1e-4 and err(paged().cpu().numpy(), ref) <= 1e-4


def test_private_appends_after_build():
    """Metadata built at shorter lengths stays valid while beams only grow privately."""
    wl = make_workload("7b64", 0)
    m = oracle_prefix_meta(wl.req_seq_offsets, wl.block_tables, wl.seq_lens, 16)
    short = np.maximum(m["tail_lblock"] * 16, wl.seq_lens - 37).astype(np.int32)
    ref = oracle_attn_workload(wl)
    _, ox = outputs(wl, lens_for_meta=short)
    assert err(ox, ref) <= TOL["bf16"]


@pytest.mark.parametrize("many_rows", [False, True])
def test_bad_block_id_gives_nan_row_only(many_rows):
    """A block id outside the pool makes only that beam's row NaN: in the paged path for any table
    entry, in the prefix path for a block appended after the metadata was built (entries in use at
    build time are validated by tts_build_prefix_meta). Both merge kernels carry the NaN."""
    wl = _many_rows_workload("bf16", 128) if many_rows else make_workload("1p5b16", 0)
    m = oracle_prefix_meta(wl.req_seq_offsets, wl.block_tables, wl.seq_lens, 16)
    b = 3
    if many_rows:  # a long beam (split partials in the paged path) with a tail of two or more blocks
        b = next(i for i in range(wl.num_seqs)
                 if wl.seq_lens[i] > 1024 and (int(wl.seq_lens[i]) + 15) // 16 - 1 > m["tail_lblock"][i])
    last = (int(wl.seq_lens[b]) + 15) // 16 - 1
    assert last > m["tail_lblock"][b]  # a tail block that is not the first one
    short = wl.seq_lens.copy()
    short[b] = 16 * last  # metadata built before block `last` was appended
    x, paged, pref = runners(wl, lens_for_meta=short)
    good_p, good_x = paged().clone(), pref().clone()
    ref = oracle_attn_workload(wl)
    assert err(good_x.cpu().numpy(), ref) <= TOL["bf16"]
    x.block_tables[b, last] = wl.num_blocks + 1000
    op, ox = paged(), pref()
    torch.cuda.synchronize()
    assert torch.isnan(op[b]).all() and torch.isnan(ox[b]).all()
    others = [i for i in range(wl.num_seqs) if i != b]
    assert torch.equal(op[others], good_p[others]) and torch.equal(ox[others], good_x[others])


def test_stale_metadata_gives_nan_row():
    wl = make_workload("1p5b16", 0)
    x, paged, pref = runners(wl)
    m = oracle_prefix_meta(wl.req_seq_offsets, wl.block_tables, wl.seq_lens, 16)
    b = int(np.argmax(m["tail_lblock"]))
    lens = x.seq_lens.clone()
    lens[b] = int(m["tail_lblock"][b]) * 16 - 5
    ox = pref(seq_lens=lens)
    torch.cuda.synchronize()
    assert torch.isnan(ox[b]).all()
    assert torch.isfinite(ox[[i for i in range(wl.num_seqs) if i != b]]).all()


def test_errors_from_device_calls():
    wl = make_workload("tiny", 0)
    x, paged, pref = runners(wl)
    with pytest.raises(TTSError):  # workspace too small
        from paper_2509_00195_amd import tts_prefix_decode_attn
        tts_prefix_decode_attn(pref.desc, pref.meta, x.q, x.k_cache, x.v_cache, None, None, x.block_tables,
                               x.block_tables.shape[1], x.seq_lens, wl.num_blocks, pref.out, pref.ws, 0)
    with pytest.raises(TTSError):  # scales given for non-fp8 KV
        from paper_2509_00195_amd import tts_paged_decode_attn
        tts_paged_decode_attn(paged.desc, wl.num_seqs, x.q, x.k_cache, x.v_cache, x.seq_lens, x.seq_lens,
                              x.block_tables, x.block_tables.shape[1], x.seq_lens, wl.max_seq_len, wl.num_blocks,
                              paged.out, paged.ws, paged.ws_bytes)


def test_work_plan_stats_and_workspace():
    wl = make_workload("7b64", 0)
    x, paged, pref = runners(wl)
    units, slots = pref.meta.stats()
    assert units > 0 and slots >= wl.num_seqs
    # every merge slot of a beam is one partial row per query head: D fp16
    # elements (bf16 cache) and four fp32 words (max, sum, row scale, pad)
    assert pref.ws_bytes >= slots * wl.shape.num_q_heads * (wl.shape.head_dim * 2 + 16)
    # the host-only listing describes the plan the device got
    from paper_2509_00195_amd import tts_plan_units_host

    ncu = torch.cuda.get_device_properties(0).multi_processor_count
    rows, host_units = tts_plan_units_host(wl.req_seq_offsets, wl.block_tables, wl.seq_lens, 16, wl.num_blocks,
                                           pref.desc, ncu)
    assert host_units == units and len(rows) > 0


def test_partials_then_merge_equals_single_call():
    from paper_2509_00195_amd import tts_prefix_decode_merge, tts_prefix_decode_partials

    wl = make_workload("7b64", 2)
    x, paged, pref = runners(wl)
    ref = pref().clone()
    out = torch.full_like(ref, float("nan"))
    tts_prefix_decode_partials(pref.desc, pref.meta, x.q, x.k_cache, x.v_cache, None, None, x.block_tables,
                               x.block_tables.shape[1], x.seq_lens, wl.num_blocks, out, pref.ws, pref.ws_bytes)
    tts_prefix_decode_merge(pref.desc, pref.meta, x.seq_lens, out, pref.ws, pref.ws_bytes)
    torch.cuda.synchronize()
    assert torch.equal(out, ref)


# Error relative to the values, for bf16 and fp8 caches. The value product takes the
# probabilities rounded to bf16 (relative error <= 2^-9 each; the row is a convex combination
# of value rows, so at most 2^-9 max|V| in total), and each partial state is stored as fp16
# elements of magnitude <= 1 times a power-of-two row scale s < 2 max|partial row| (absolute
# error <= 2^-12 s < 2^-11 max|V|, carried through the merge's weights, which sum to 1); fp32
# accumulation and the scores add about 1e-6 relative. Hence, per beam,
#   max |out - oracle| <= (2^-9 + 2^-11 + 2^-14) max|V over the beam's tokens|,
# which the N(0, 1) tolerance of 1e-2 does not state for values of any size.
REL_BOUND = 2.0 ** -9 + 2.0 ** -11 + 2.0 ** -14


def _heavy_tailed_values(wl, seed):
    """Values with heavy tails: a tenth of the (block, slot) tokens scaled x30 and the rest
    scaled by |t(3)| draws per token (unused slots keep their NaN)."""
    rng = np.random.default_rng(seed)
    v = torch.from_numpy(wl.v_cache.view(np.int16)).view(torch.bfloat16).float().numpy()  # [nb][Hkv][D][16]
    nb = v.shape[0]
    f = np.abs(rng.standard_t(3, size=(nb, 1, 1, 16))) + 0.1
    f = np.where(rng.random((nb, 1, 1, 16)) < 0.1, 30.0, f)
    return dataclasses.replace(wl, v_cache=bf16_bits(v * f))


@pytest.mark.parametrize("name", ["7b64", "1p5b16"])
def test_error_relative_to_values_heavy_tails(name):
    wl = _heavy_tailed_values(make_workload(name, 0), 21)
    ref = oracle_attn_workload(wl)
    op, ox = outputs(wl)
    worst = 0.0
    for b in range(wl.num_seqs):
        vmax = _max_abs_v(wl, b)
        eb = max(err(op[b], ref[b]), err(ox[b], ref[b]))
        worst = max(worst, eb / vmax)
        assert eb <= REL_BOUND * vmax, (b, eb, vmax)
    print(f"{name} heavy-tailed values: worst error / max|V| = {worst:.2e} (bound {REL_BOUND:.2e})", flush=True)


def test_one_workspace_across_batches():
    """A search loop rebuilds its metadata every iteration and keeps its workspace: one
    workspace, filled with garbage first, serves two batches' metadata in turn (A, B, A, B).
    Every call meets the oracle, and the full call equals its partials + merge launches."""
    from paper_2509_00195_amd import tts_prefix_decode_attn, tts_prefix_decode_merge, tts_prefix_decode_partials

    runs = []
    for seed in (0, 1):
        wl = make_workload("7b64", seed)
        x, _, pref = runners(wl)
        runs.append((wl, x, pref, oracle_attn_workload(wl)))
    nbytes = max(r[2].ws_bytes for r in runs)
    ws = torch.full((nbytes,), 0xA5, dtype=torch.uint8, device="cuda:0")
    for wl, x, pref, ref in runs + runs:
        args = (pref.desc, pref.meta, x.q, x.k_cache, x.v_cache, None, None, x.block_tables,
                x.block_tables.shape[1], x.seq_lens, wl.num_blocks)
        one = torch.full_like(pref.out, float("nan"))
        two = torch.full_like(pref.out, float("nan"))
        tts_prefix_decode_attn(*args, one, ws, nbytes)
        tts_prefix_decode_partials(*args, two, ws, nbytes)
        tts_prefix_decode_merge(pref.desc, pref.meta, x.seq_lens, two, ws, nbytes)
        torch.cuda.synchronize()
        assert torch.equal(one, two)
        assert err(one.cpu().numpy(), ref) <= TOL["bf16"]
