"""GPU parity of the softmax's exact-maximum repeat, against the oracle.

The attention kernel weighs scores against a fixed reference maximum of 0
(log2 units) and computes a unit again, with each row's exact maximum, when
some row's maximum leaves [-64, 64]. Narrow units decide per wave (their
loop has no barrier); wide units (block pairs staged in LDS, a loop with
barriers) decide for the whole workgroup. These inputs reach every case:

(a) queries of two beams scaled x35 in the 7B 64-beam batch: only the row
    tiles of those beams leave the window, so in a wide unit only one or two
    of the four waves need the repeat and the others must take it with them;
(b) the same on a 1.5B-shaped batch of 8 beams whose plan has narrow units
    only, and through the paged call;
(c) every score far below the window: keys 2 + N(0, 0.25), queries
    -1 + N(0, 0.01), so q.k ~ -256 over D = 128; with scale 1 that is about
    -369 in log2 units (the first pass underflows every weight to 0), with
    scale 0.22 about -81;
(d) only the prompt's keys shifted (scores about +185 in log2 units there,
    ordinary elsewhere): the row's partial states then carry references
    hundreds apart and the merge must weigh the tail's states to zero.

Tolerances are the parity ones (max abs 1e-2 for bf16 KV).
"""

import dataclasses

import numpy as np
import pytest
import torch

from oracle.attention import oracle_attn_workload
from oracle.prefix_meta import oracle_prefix_meta
from paper_2509_00195_amd import tts_plan_units_host
from paper_2509_00195_amd.runner import PagedAttention, PrefixAttention, desc_for
from tests._paged import bf16_bits
from tts_synth import AttnShape, ReqSpec, WorkloadConfig, make_workload
from tts_synth.device import to_device

pytestmark = pytest.mark.gpu

TOL = 1e-2
LOG2E = 1.4426950408889634


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    torch.cuda.set_device(0)


def _bf16_f32(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).float().numpy()


def _batch(kind):
    if kind == "wide":
        return make_workload("7b64", 0)
    cfg = WorkloadConfig("narrow8", AttnShape(12, 2, 128, 16, "bf16", "bf16"),
                         (ReqSpec(beams=8, branch=4, prompt=(512, 512), step=(64, 256), max_len=2048),))
    return make_workload(cfg, 0)


def _has_wide_units(wl):
    ncu = torch.cuda.get_device_properties(0).multi_processor_count
    rows, _ = tts_plan_units_host(wl.req_seq_offsets, wl.block_tables, wl.seq_lens, 16, wl.num_blocks,
                                  desc_for(wl.shape), ncu)
    return bool(np.any(rows[:, 6] & 8)), rows


def _row_max_log2(wl, b, scale):
    """Largest scaled score of beam b over all its query heads (log2 units), from the stored inputs."""
    sh = wl.shape
    L = int(wl.seq_lens[b])
    nb = -(-L // 16)
    k = _bf16_f32(wl.k_cache[wl.block_tables[b, :nb]])  # [nb][Hkv][16][D]
    k = k.transpose(1, 0, 2, 3).reshape(sh.num_kv_heads, nb * 16, sh.head_dim)[:, :L]
    q = _bf16_f32(wl.q[b]).reshape(sh.num_kv_heads, sh.group, sh.head_dim)
    s = np.einsum("hgd,htd->hgt", q.astype(np.float64), k.astype(np.float64))
    return float(np.max(s)) * scale * LOG2E


def _run(wl, scale=0.0):
    x = to_device(wl)
    pref = PrefixAttention(x, wl.req_seq_offsets, wl.block_tables, wl.seq_lens, wl.num_blocks, scale=scale)
    paged = PagedAttention(x, wl.max_seq_len, wl.num_blocks, scale=scale)
    ox = pref().cpu().numpy()
    op = paged().cpu().numpy()
    torch.cuda.synchronize()
    return ox, op


def _err(a, b):
    return float(np.max(np.abs(a.astype(np.float64) - b.astype(np.float64))))


@pytest.mark.parametrize("kind", ["wide", "narrow"])
def test_redo_some_beams_scaled(kind):
    wl = _batch(kind)
    wide, rows = _has_wide_units(wl)
    assert wide == (kind == "wide")
    perm = oracle_prefix_meta(wl.req_seq_offsets, wl.block_tables, wl.seq_lens, 16)["perm"]
    picks = [int(perm[0]), int(perm[len(perm) // 2 + 1])]
    if kind == "wide":  # both beams sit in wide units next to beams that are not scaled
        wide_beams = set(rows[(rows[:, 6] & 8) != 0, 3].tolist())
        assert set(picks) <= wide_beams and len(wide_beams) > 2 * len(picks)
    q = _bf16_f32(wl.q)
    q[picks] *= 35.0
    wl2 = dataclasses.replace(wl, q=bf16_bits(q))
    sc = 1.0 / np.sqrt(wl.shape.head_dim)
    for b in picks:
        assert _row_max_log2(wl2, b, sc) > 64.0  # these rows leave the window...
    others = [b for b in range(wl.num_seqs) if b not in picks]
    assert max(_row_max_log2(wl2, b, sc) for b in others[:6]) < 64.0  # ...ordinary rows do not
    ref = oracle_attn_workload(wl2)
    ox, op = _run(wl2)
    print(f"redo {kind}: prefix {_err(ox, ref):.2e} paged {_err(op, ref):.2e}", flush=True)
    assert np.isfinite(ox).all() and np.isfinite(op).all()
    assert _err(ox, ref) <= TOL and _err(op, ref) <= TOL


def _shift_keys(wl, rng, blocks=None, k_mean=2.0, q_mean=-1.0):
    """Keys k_mean + N(0, 0.25) (all blocks, or only `blocks`), queries q_mean + N(0, 0.01); the
    unused slots keep their NaN."""
    kf = _bf16_f32(wl.k_cache)
    new = k_mean + 0.5 * rng.standard_normal(kf.shape)
    if blocks is not None:
        sel = np.zeros(kf.shape[0], bool)
        sel[blocks] = True
        new = np.where(sel[:, None, None, None], new, kf)
    new = np.where(np.isnan(kf), np.nan, new)
    q = q_mean + 0.1 * rng.standard_normal(wl.q.shape)
    return dataclasses.replace(wl, k_cache=bf16_bits(new), q=bf16_bits(q))


@pytest.mark.parametrize("kind", ["wide", "narrow"])
@pytest.mark.parametrize("scale", [1.0, 0.22])
def test_redo_rows_far_below_window(kind, scale):
    wl = _shift_keys(_batch(kind), np.random.default_rng(11))
    hi = max(_row_max_log2(wl, b, scale) for b in range(0, wl.num_seqs, 7))
    assert hi < -64.0 and (scale < 0.5 or hi < -126.0)
    ref = oracle_attn_workload(wl, scale=scale)
    ox, op = _run(wl, scale)
    print(f"below window {kind} scale {scale}: prefix {_err(ox, ref):.2e} paged {_err(op, ref):.2e}",
          flush=True)
    assert np.isfinite(ox).all() and np.isfinite(op).all()
    assert _err(ox, ref) <= TOL and _err(op, ref) <= TOL


@pytest.mark.parametrize("kind", ["wide", "narrow"])
def test_redo_prompt_far_above_tails(kind):
    wl = _batch(kind)
    prompt_blocks = wl.block_tables[0, :512 // 16 if kind == "narrow" else 1024 // 16]
    wl = _shift_keys(wl, np.random.default_rng(12), blocks=prompt_blocks, q_mean=1.0)
    assert _row_max_log2(wl, 0, 0.5) > 126.0
    ref = oracle_attn_workload(wl, scale=0.5)
    ox, op = _run(wl, 0.5)
    print(f"prompt above tails {kind}: prefix {_err(ox, ref):.2e} paged {_err(op, ref):.2e}", flush=True)
    assert np.isfinite(ox).all() and np.isfinite(op).all()
    assert _err(ox, ref) <= TOL and _err(op, ref) <= TOL
