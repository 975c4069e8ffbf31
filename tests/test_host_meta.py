"""libtts host side, no GPU: symbol exports, the C++ metadata builder
bit-exact against the oracle, coverage export, and argument validation."""

import ctypes
import os
import re

import numpy as np
import pytest
from hypothesis import given, settings

import paper_2509_00195_amd as tts
from oracle import oracle_coverage, oracle_prefix_meta
from tests.test_oracle_prefix_meta import KEYS, load_golden, random_tree
from tts_synth import CONFIGS, AttnShape, build_tree, make_workload, workload_from_tree

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BS = 16


def declared_symbols():
    with open(os.path.join(ROOT, "include", "tts.h")) as f:
        src = f.read()
    return sorted(set(re.findall(r"^\s*(?:tts_status|void|size_t|const char\*)\s+(tts_\w+)\(", src, re.M)))


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(tts.tts.LIB_PATH)
    decl = declared_symbols()
    assert len(decl) >= 10
    for name in decl:
        assert hasattr(lib, name), name
    assert sorted(tts.EXPORTED) == decl


def build(offs, tables, lens, num_blocks=None):
    nb = int(tables.max()) + 1 if num_blocks is None else num_blocks
    return tts.tts_build_prefix_meta(offs, tables, lens, BS, max(nb, 1))


def assert_same(meta_c: dict, meta_o: dict):
    for k in KEYS:
        assert meta_c[k].tolist() == meta_o[k].tolist(), k
    for k in ["num_seqs", "num_segs", "unique_blocks", "unique_tokens"]:
        assert meta_c[k] == meta_o[k], k


def test_golden_example_matches():
    offs, tables, lens, bs, exp = load_golden()
    m = build(offs, tables, lens).export()
    for k in KEYS:
        assert m[k].tolist() == exp[k], k
    assert m["unique_tokens"] == exp["unique_tokens"] and m["unique_blocks"] == exp["unique_blocks"]


@pytest.mark.parametrize("name", ["tiny", "1p5b16", "7b64", "7b64_balanced", "7b_straggler"])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_configs_bit_exact(name, seed):
    cfg = CONFIGS[name]
    tree = build_tree(cfg, seed)
    w = workload_from_tree(AttnShape(2, 1, 8, BS, "f32", "f32"), tree, seed, name=name)  # tiny values: fast
    mo = oracle_prefix_meta(w.req_seq_offsets, w.block_tables, w.seq_lens, BS)
    h = build(w.req_seq_offsets, w.block_tables, w.seq_lens, w.num_blocks)
    assert_same(h.export(), mo)
    cov = h.coverage()
    assert np.array_equal(cov, oracle_coverage(mo, w.block_tables, w.seq_lens, BS))


def test_longchain_tree_bit_exact():
    cfg = CONFIGS["7b_longchain_fp8"]
    tree = build_tree(cfg, 0)
    w = workload_from_tree(AttnShape(2, 1, 8, BS, "f32", "f32"), tree, 0, name="lc")
    mo = oracle_prefix_meta(w.req_seq_offsets, w.block_tables, w.seq_lens, BS)
    assert_same(build(w.req_seq_offsets, w.block_tables, w.seq_lens, w.num_blocks).export(), mo)


@settings(max_examples=80, deadline=None)
@given(random_tree())
def test_random_trees_bit_exact(tree):
    w = workload_from_tree(AttnShape(2, 1, 8, BS, "f32", "f32"), tree, 5)
    mo = oracle_prefix_meta(w.req_seq_offsets, w.block_tables, w.seq_lens, BS)
    h = build(w.req_seq_offsets, w.block_tables, w.seq_lens, w.num_blocks)
    assert_same(h.export(), mo)
    assert np.array_equal(h.coverage(), oracle_coverage(mo, w.block_tables, w.seq_lens, BS))


def test_coverage_with_appended_lengths():
    offs, tables, lens, _, _ = load_golden()
    mo = oracle_prefix_meta(offs, tables, lens, BS)
    h = build(offs, tables, lens)
    longer = lens.copy()
    longer[0] += 10  # private append into its partial block
    longer[6] += 1   # needs the next table entry (-1 there: pblock reported as given)
    assert np.array_equal(h.coverage(longer), oracle_coverage(mo, tables, lens, BS, seq_lens_now=longer))


def test_work_plan_stats():
    w = make_workload("tiny", 0)
    desc = tts.make_desc(4, 1, 64, 16, "f32", "f32")
    # desc given -> work list built and uploaded: needs a device; CPU-only here checks the host path only.
    h = build(w.req_seq_offsets, w.block_tables, w.seq_lens, w.num_blocks)
    with pytest.raises(tts.TTSError):
        h.stats()  # built without desc
    del desc


@pytest.mark.parametrize("mutate,code", [
    (lambda o, t, l: (np.array([1, 4], np.int32), t, l), tts.tts.TTS_ERR_INVALID_ARG),      # offsets[0] != 0
    (lambda o, t, l: (np.array([0, 3], np.int32), t, l), tts.tts.TTS_ERR_INVALID_ARG),      # offsets end != S
    (lambda o, t, l: (o, t, np.array([10, -1, 3, 4], np.int32)), tts.tts.TTS_ERR_INVALID_ARG),  # negative len
    (lambda o, t, l: (o, t, np.array([10, 100, 3, 4], np.int32)), tts.tts.TTS_ERR_INVALID_ARG),  # len > table
    (lambda o, t, l: (o, np.where(t == 2, 99, t).astype(np.int32), l), tts.tts.TTS_ERR_OUT_OF_RANGE),  # id >= NB
    (lambda o, t, l: (o, np.where(t == 2, -5, t).astype(np.int32), l), tts.tts.TTS_ERR_OUT_OF_RANGE),  # id < 0
])
def test_validation_errors(mutate, code):
    offs = np.array([0, 4], np.int32)
    tables = np.array([[0, 1, 2], [0, 1, 3], [0, 4, -1], [5, -1, -1]], np.int32)
    lens = np.array([40, 33, 20, 4], np.int32)
    build(offs, tables, lens, 6)  # valid
    o2, t2, l2 = mutate(offs, tables, lens)
    with pytest.raises(tts.TTSError) as ei:
        build(o2, t2, l2, 6)
    assert ei.value.status == code
    assert tts.load().tts_last_error().decode() != ""


def test_unused_table_entries_are_not_validated():
    offs = np.array([0, 2], np.int32)
    tables = np.array([[0, 1, -7], [0, 2, 10 ** 6]], np.int32)
    lens = np.array([20, 32], np.int32)
    m = build(offs, tables, lens, 3).export()
    assert m["unique_blocks"] == 3


def test_desc_validation_on_build():
    offs = np.array([0, 1], np.int32)
    tables = np.array([[0]], np.int32)
    lens = np.array([5], np.int32)
    for bad in [tts.make_desc(5, 2, 128), tts.make_desc(4, 1, 96), tts.make_desc(4, 1, 64, q_dtype="f32"),
                tts.make_desc(4, 1, 64, block_size=32)]:
        with pytest.raises(tts.TTSError):
            tts.tts_build_prefix_meta(offs, tables, lens, 16, 1, desc=bad)


def test_paged_workspace_size():
    d = tts.make_desc(28, 4, 128)
    assert tts.tts_paged_decode_workspace_size(d, 64, 512) == 0  # single split: written directly
    ws = tts.tts_paged_decode_workspace_size(d, 64, 4096)
    nsplit = -(-256 // 32)
    rows = 64 * nsplit * 28
    assert ws >= rows * (128 * 2 + 16)  # fp16 row + max, sum, scale, pad
    d32 = tts.make_desc(28, 4, 128, q_dtype="f32", kv_dtype="f32")
    assert tts.tts_paged_decode_workspace_size(d32, 64, 4096) >= rows * (128 * 4 + 16)
