"""Pins for the CPU prefix-metadata oracle (no GPU).

Checked against a hand-derived golden example, brute-force pairwise
longest-common-prefix over block ids, coverage/partition properties, and
statistics recomputed from the generator's own allocation records.
"""

import json
import os
from itertools import combinations

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import oracle_coverage, oracle_prefix_meta
from tts_synth import CONFIGS, AttnShape, BeamTree, build_tree, make_workload, workload_from_tree

HERE = os.path.dirname(os.path.abspath(__file__))
BS = 16
KEYS = ["perm", "seg_req", "seg_parent", "seg_lblock_begin", "seg_nblocks", "seg_beam_begin", "seg_beam_end",
        "tail_lblock"]


def load_golden():
    with open(os.path.join(HERE, "golden", "prefix_meta_example.json")) as f:
        g = json.load(f)
    return (np.array(g["req_seq_offsets"], np.int32), np.array(g["block_tables"], np.int32),
            np.array(g["seq_lens"], np.int32), g["block_size"], g["expected"])


def test_golden_example():
    offs, tables, lens, bs, exp = load_golden()
    m = oracle_prefix_meta(offs, tables, lens, bs)
    for k in KEYS:
        assert m[k].tolist() == exp[k], k
    for k in ["num_seqs", "num_segs", "unique_blocks", "unique_tokens"]:
        assert m[k] == exp[k], k


def full_path(tables, lens, b):
    return [int(x) for x in tables[b, : int(lens[b]) // BS]]


def check_meta(offs, tables, lens, m):
    """Properties every canonical metadata must satisfy, by brute force."""
    s = len(lens)
    perm = m["perm"]
    assert sorted(perm.tolist()) == list(range(s))
    pos = np.empty(s, np.int64)
    pos[perm] = np.arange(s)
    req_of = np.zeros(s, np.int64)
    for r in range(len(offs) - 1):
        req_of[offs[r]:offs[r + 1]] = r
        # Requests stay in order and contiguous in perm.
        assert sorted(pos[offs[r]:offs[r + 1]].tolist()) == list(range(offs[r], offs[r + 1]))
    nseg = m["num_segs"]
    members = []
    for sgi in range(nseg):
        bb, be = m["seg_beam_begin"][sgi], m["seg_beam_end"][sgi]
        assert be - bb >= 2
        mem = sorted(perm[bb:be].tolist())
        members.append(mem)
        assert all(req_of[b] == m["seg_req"][sgi] for b in mem)
        lb, nb = m["seg_lblock_begin"][sgi], m["seg_nblocks"][sgi]
        assert nb >= 1
        # Every member has the same full blocks over [0, lb + nb) ...
        ref = full_path(tables, lens, mem[0])
        assert len(ref) >= lb + nb
        for b in mem:
            assert full_path(tables, lens, b)[: lb + nb] == ref[: lb + nb]
        # ... and no beam outside the set shares that whole prefix.
        for b in range(offs[m["seg_req"][sgi]], offs[m["seg_req"][sgi] + 1]):
            if b not in mem:
                assert full_path(tables, lens, b)[: lb + 1] != ref[: lb + 1]
        par = m["seg_parent"][sgi]
        if par < 0:
            assert lb == 0
        else:
            assert par < sgi  # preorder
            assert m["seg_lblock_begin"][par] + m["seg_nblocks"][par] == lb
            assert set(mem) < set(members[par])
    # Pairwise: LCP of full-block paths == end of the deepest segment containing both.
    for r in range(len(offs) - 1):
        for a, b in combinations(range(offs[r], offs[r + 1]), 2):
            pa, pb = full_path(tables, lens, a), full_path(tables, lens, b)
            lcp = 0
            while lcp < min(len(pa), len(pb)) and pa[lcp] == pb[lcp]:
                lcp += 1
            deepest = 0
            for sgi in range(nseg):
                if a in members[sgi] and b in members[sgi]:
                    deepest = max(deepest, m["seg_lblock_begin"][sgi] + m["seg_nblocks"][sgi])
            assert deepest == lcp, (a, b)
    # Coverage: each used (beam, lblock) exactly once; segments then tail.
    cov = oracle_coverage(m, tables, lens, BS)
    for b in range(s):
        rows = cov[cov[:, 0] == b]
        nblk = -(-int(lens[b]) // BS)
        assert rows[:, 1].tolist() == list(range(nblk))
        seg_rows = rows[rows[:, 4] >= 0]
        assert len(seg_rows) == m["tail_lblock"][b]
        assert np.all(rows[: m["tail_lblock"][b], 4] >= 0) and np.all(rows[m["tail_lblock"][b]:, 4] == -1)
        for row in seg_rows:
            sgi = row[4]
            assert b in members[sgi]
            assert m["seg_lblock_begin"][sgi] <= row[1] < m["seg_lblock_begin"][sgi] + m["seg_nblocks"][sgi]
        assert rows[:, 3].sum() == lens[b]
    # Children ordered by smallest original beam index: within every segment's
    # range, beams of each child subtree appear in increasing order of their minimum.
    for sgi in range(nseg):
        kids = [c for c in range(nseg) if m["seg_parent"][c] == sgi]
        mins = [min(members[c]) for c in kids]
        starts = [m["seg_beam_begin"][c] for c in kids]
        assert np.all(np.argsort(mins) == np.argsort(starts))


def test_golden_properties():
    offs, tables, lens, _, _ = load_golden()
    check_meta(offs, tables, lens, oracle_prefix_meta(offs, tables, lens, BS))


@pytest.mark.parametrize("name", ["tiny", "1p5b16"])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_config_trees(name, seed):
    cfg = CONFIGS[name]
    tree = build_tree(cfg, seed)
    w = workload_from_tree(cfg.shape, tree, seed, name=name)
    m = oracle_prefix_meta(w.req_seq_offsets, w.block_tables, w.seq_lens, BS)
    check_meta(w.req_seq_offsets, w.block_tables, w.seq_lens, m)


@pytest.mark.parametrize("name", ["7b64", "7b64_balanced", "7b_straggler"])
def test_unique_tokens_two_ways(name):
    """unique_tokens/blocks from the metadata == recount from the generator's allocation records."""
    cfg = CONFIGS[name]
    tree = build_tree(cfg, 0)
    valid = {}
    for al, L in zip(tree.beam_allocs, tree.beam_lens):
        for j, a in enumerate(al):
            valid[a] = max(valid.get(a, 0), min(BS, L - j * BS))
    shape = cfg.shape
    w = workload_from_tree(AttnShape(2, 1, 8, BS, "f32", "f32"), tree, 0, name=name)  # tiny heads: fast
    m = oracle_prefix_meta(w.req_seq_offsets, w.block_tables, w.seq_lens, BS)
    assert m["unique_blocks"] == len(valid)
    assert m["unique_tokens"] == sum(valid.values())
    del shape


def test_partial_blocks_and_requests_never_shared():
    # Two beams with the same ids including the partial last block, and a
    # second request reusing the same ids.
    tables = np.array([[5, 6, 7], [5, 6, 7], [5, 6, 7]], np.int32)
    lens = np.array([40, 40, 40], np.int32)
    offs = np.array([0, 2, 3], np.int32)
    m = oracle_prefix_meta(offs, tables, lens, BS)
    assert m["num_segs"] == 1
    assert m["seg_nblocks"].tolist() == [2] and m["seg_beam_end"].tolist() == [2]
    assert m["tail_lblock"].tolist() == [2, 2, 0]
    assert m["unique_blocks"] == 3 and m["unique_tokens"] == 40


def test_non_prefix_shared_ids_get_no_sharing():
    # Same id at block 1 but different block 0: not a trie prefix.
    tables = np.array([[1, 9, 2], [3, 9, 4]], np.int32)
    lens = np.array([48, 48], np.int32)
    m = oracle_prefix_meta(np.array([0, 2], np.int32), tables, lens, BS)
    assert m["num_segs"] == 0 and m["tail_lblock"].tolist() == [0, 0]


def test_zero_and_short_lengths():
    tables = np.array([[1, 2], [1, 2], [1, 3], [1, -1]], np.int32)
    lens = np.array([0, 20, 17, 15], np.int32)
    m = oracle_prefix_meta(np.array([0, 4], np.int32), tables, lens, BS)
    check_meta(np.array([0, 4]), tables, lens, m)
    assert m["tail_lblock"].tolist() == [0, 1, 1, 0]
    assert m["perm"].tolist() == [0, 1, 2, 3] or m["perm"][0] == 0


def test_empty_batch():
    m = oracle_prefix_meta(np.array([0], np.int32), np.zeros((0, 1), np.int32), np.zeros(0, np.int32), BS)
    assert m["num_seqs"] == 0 and m["num_segs"] == 0 and m["unique_tokens"] == 0


@st.composite
def random_tree(draw):
    """Small random beam trees with forks, identical beams and ragged lengths."""
    nreq = draw(st.integers(1, 3))
    tree = BeamTree(block_size=BS)
    rng = np.random.default_rng(draw(st.integers(0, 2 ** 31)))
    for _ in range(nreq):
        nbeams = draw(st.integers(1, 7))
        beams = []
        for i in range(nbeams):
            if beams and rng.random() < 0.7:
                par_blocks, par_len = beams[int(rng.integers(len(beams)))]
                cut = int(rng.integers(0, par_len + 1))
                nfull = cut // BS
                blocks = list(par_blocks[:nfull])
                L = nfull * BS
                if cut % BS:
                    blocks.append(tree.new_alloc(par_blocks[nfull], cut % BS))
                    L = cut
            else:
                blocks, L = [], 0
            add = int(rng.integers(0, 60)) if rng.random() < 0.9 else 0
            newL = L + add
            while len(blocks) * BS < newL:
                blocks.append(tree.new_alloc())
            beams.append((blocks, newL))
        for blocks, L in beams:
            tree.beam_allocs.append(blocks)
            tree.beam_lens.append(L)
            tree.beam_parent.append(-1)
        tree.req_offsets.append(len(tree.beam_lens))
    return tree


@settings(max_examples=60, deadline=None)
@given(random_tree(), st.booleans())
def test_random_trees(tree, shuffle):
    w = workload_from_tree(AttnShape(2, 1, 8, BS, "f32", "f32"), tree, 3, shuffle=shuffle)
    m = oracle_prefix_meta(w.req_seq_offsets, w.block_tables, w.seq_lens, BS)
    check_meta(w.req_seq_offsets, w.block_tables, w.seq_lens, m)


def test_generator_is_deterministic():
    a = make_workload("1p5b16", 1)
    b = make_workload("1p5b16", 1)
    for k in ["block_tables", "seq_lens", "q", "k_cache", "v_cache"]:
        assert np.array_equal(getattr(a, k), getattr(b, k), equal_nan=True) if getattr(a, k).dtype.kind == "f" \
            else np.array_equal(getattr(a, k), getattr(b, k))
