"""The work plan (host planner), on the CPU through tts_plan_units_host.

Properties that any correct plan has, checked on every workload shape at
several workgroup counts: for every KV head, each (beam, logical block) of
the build-time sequences is covered by exactly one unit entry, with the
block's physical id and valid token count from the block tables; the
partially filled last block of a beam is flagged LIVE and lies in a narrow
unit; every beam has exactly one extension entry per KV head (for blocks
appended after the build); LIVE and extension entries sit in a unit's first
window; a window holds at most 64 entries (a unit at most 128); wide units
hold full blocks only. The number of units bounds the partial states.
"""

import dataclasses

import numpy as np
import pytest

import paper_2509_00195_amd as tts
from paper_2509_00195_amd.tts import PLAN_EXT, PLAN_LIVE, PLAN_SECOND, PLAN_WIDE
from tts_synth import CONFIGS, AttnShape, build_tree, workload_from_tree

BS = 16


def tables_of(cfg, seed):
    """The config's beam tree, block tables and lengths (the plan needs no cache contents: tiny values)."""
    return workload_from_tree(AttnShape(2, 1, 8, BS, "f32", "f32"), build_tree(cfg, seed), seed, name=cfg.name)


def plan_rows(wl, sh, nbins):
    desc = tts.make_desc(sh.num_q_heads, sh.num_kv_heads, sh.head_dim, BS, sh.q_dtype, sh.kv_dtype)
    return tts.tts_plan_units_host(wl.req_seq_offsets, wl.block_tables, wl.seq_lens, BS, wl.num_blocks, desc, nbins)


def check_plan(wl, sh, nbins):
    rows, units = plan_rows(wl, sh, nbins)
    unit, entry, kvh, beam, block, valid, flags = rows.T
    assert units >= 1 and unit.min() == 0 and unit.max() == units - 1
    ext = (flags & PLAN_EXT) != 0
    # coverage: exactly once per (kv head, beam, logical block)
    lens = np.asarray(wl.seq_lens, np.int64)
    tabs = np.asarray(wl.block_tables, np.int64)
    nblk = (lens + BS - 1) // BS
    pos = {}
    for b in range(len(lens)):
        for j in range(int(nblk[b])):
            pos[(b, int(tabs[b, j]))] = j
    seen = np.zeros((sh.num_kv_heads, len(lens), int(nblk.max()) if len(lens) else 0), np.int32)
    for u, h, b, blk, v, f in zip(unit[~ext], kvh[~ext], beam[~ext], block[~ext], valid[~ext], flags[~ext]):
        j = pos[(int(b), int(blk))]
        seen[h, b, j] += 1
        assert v == min(BS, int(lens[b]) - BS * j)
        partial = j == nblk[b] - 1 and lens[b] % BS != 0
        assert bool(f & PLAN_LIVE) == partial
        if f & PLAN_WIDE:
            assert v == BS and not partial
    for b in range(len(lens)):
        assert (seen[:, b, : nblk[b]] == 1).all(), b
    # one extension entry per (kv head, beam)
    ext_count = np.zeros((sh.num_kv_heads, len(lens)), np.int32)
    np.add.at(ext_count, (kvh[ext], beam[ext]), 1)
    assert (ext_count == 1).all()
    # windows
    assert not ((flags & (PLAN_LIVE | PLAN_EXT)) != 0)[(flags & PLAN_SECOND) != 0].any()
    for w in (0, PLAN_SECOND):
        sel = (flags & PLAN_SECOND) == w
        per_window = {}
        for u, e in zip(unit[sel], entry[sel]):
            per_window.setdefault(int(u), set()).add(int(e))
        assert all(len(es) <= 64 for es in per_window.values())
    return rows, units


@pytest.mark.parametrize("name", ["tiny", "1p5b16", "7b64", "7b64_balanced", "7b_straggler"])
@pytest.mark.parametrize("seed", [0, 1])
@pytest.mark.parametrize("nbins", [256, 40, 1])
def test_plan_covers_every_block_once(name, seed, nbins):
    cfg = CONFIGS[name]
    check_plan(tables_of(cfg, seed), cfg.shape, nbins)


def test_long_chain_plan_uses_both_windows():
    cfg = CONFIGS["7b_longchain_fp8"]
    cfg = dataclasses.replace(cfg, reqs=cfg.reqs[:4])  # a quarter of the requests keeps the check quick
    rows, units = check_plan(tables_of(cfg, 0), cfg.shape, 64)
    flags = rows[:, 6]
    assert ((flags & PLAN_SECOND) != 0).any() and ((flags & PLAN_WIDE) != 0).any()


def test_small_batch_gets_few_units():
    """A batch that fits the workgroups gets units sized by attention plus merge time, not one per entry:
    at most a few units per beam and KV head."""
    cfg = CONFIGS["1p5b16"]
    for seed in range(6):
        wl = tables_of(cfg, seed)
        _, units = plan_rows(wl, cfg.shape, 256)
        assert units <= 4 * len(wl.seq_lens) * cfg.shape.num_kv_heads, (seed, units)


def test_plan_argument_errors():
    sh = CONFIGS["tiny"].shape
    wl = tables_of(CONFIGS["tiny"], 0)
    desc = tts.make_desc(sh.num_q_heads, sh.num_kv_heads, sh.head_dim, BS, sh.q_dtype, sh.kv_dtype)
    with pytest.raises(tts.TTSError):
        tts.tts_plan_units_host(wl.req_seq_offsets, wl.block_tables, wl.seq_lens, BS, wl.num_blocks, desc, 0)
    bad = np.where(wl.block_tables == wl.block_tables[0, 0], wl.num_blocks + 5, wl.block_tables).astype(np.int32)
    with pytest.raises(tts.TTSError):
        tts.tts_plan_units_host(wl.req_seq_offsets, bad, wl.seq_lens, BS, wl.num_blocks, desc, 8)


def unit_rows(name, wide, nbins=256):
    """Query rows of each wide (or each narrow) unit in the seed-0 plan of a config."""
    cfg = CONFIGS[name]
    rows, _ = plan_rows(tables_of(cfg, 0), cfg.shape, nbins)
    unit, beam, flags = rows[:, 0], rows[:, 3], rows[:, 6]
    sel = ((flags & PLAN_WIDE) != 0) == wide
    g = cfg.shape.num_q_heads // cfg.shape.num_kv_heads
    beams = {}
    for u, b in zip(unit[sel], beam[sel]):
        beams.setdefault(int(u), set()).add(int(b))
    return [g * len(v) for v in beams.values()]


def test_row_caps_are_chosen_per_batch():
    """The planner models a batch with wide units of up to 192 rows (three row tiles per wave) and of up to 128
    (two), and a batch that fits the workgroups with narrow units of up to 64 rows and of up to 42, and keeps
    the cheaper plan: 192 / 64 for the 7B 64-beam tree, 128-row wide units for the balanced tree, 42-row
    narrow units for the 1.5B 16-beam tree."""
    r = unit_rows("7b64", wide=True)
    assert r and 128 < max(r) <= 192
    assert 42 < max(unit_rows("7b64", wide=False)) <= 64
    r = unit_rows("7b64_balanced", wide=True)
    assert r and max(r) <= 128
    assert max(unit_rows("1p5b16", wide=False)) <= 42
