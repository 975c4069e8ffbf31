"""Pins of the KV-maintenance oracle (CPU): E4M3 encoding, append, copy, fork.

The encoder is checked against what the format fixes (every code value
encodes to itself, midpoints go to the even mantissa, saturation, NaN) and
against a library routine (torch's float8_e4m3fn cast) on random values;
the append / fork oracles against hand-derived cases and invariants; the
library's host fork planner against the oracle.
"""

from __future__ import annotations

import numpy as np
import pytest

from oracle.fp8 import e4m3_table
from oracle.kv_ops import append_kv, copy_blocks, e4m3_encode, fork_tables
from paper_2509_00195_amd import TTSError, tts_fork_tables

TABLE = e4m3_table()


def test_encode_every_code_round_trips():
    for c in range(256):
        if c in (0x7F, 0xFF):
            continue
        v = np.float32(TABLE[c])
        want = c if not (c == 0x80) else 0x80  # -0.0 keeps its sign
        assert int(e4m3_encode(np.array([v]))[0]) == want, hex(c)


def test_encode_midpoints_go_to_even_mantissa():
    for c in range(126):
        lo, hi = np.float64(TABLE[c]), np.float64(TABLE[c + 1])
        mid = np.float32((lo + hi) / 2)
        assert float(mid) == (lo + hi) / 2  # exact in fp32
        even = c if c % 2 == 0 else c + 1
        assert int(e4m3_encode(np.array([mid]))[0]) == even
        assert int(e4m3_encode(np.array([-mid]))[0]) == even | 0x80
        below = np.nextafter(mid, np.float32(0))
        above = np.nextafter(mid, np.float32(1000))
        assert int(e4m3_encode(np.array([below]))[0]) == c
        assert int(e4m3_encode(np.array([above]))[0]) == c + 1


def test_encode_saturates_and_nan():
    x = np.array([448, 449, 464, 480, 1e6, np.inf, -448, -1e6, -np.inf, np.nan], np.float32)
    assert e4m3_encode(x).tolist() == [0x7E, 0x7E, 0x7E, 0x7E, 0x7E, 0x7E, 0xFE, 0xFE, 0xFE, 0x7F]


def test_encode_matches_library_cast_in_range():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.normal(0, 1, 3000), rng.normal(0, 100, 3000), rng.uniform(-448, 448, 3000),
                        rng.normal(0, 0.01, 3000)]).astype(np.float32)
    x = x[np.abs(x) <= 448]
    lib = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(e4m3_encode(x), lib)


def _fp8_cache(nb=6, hkv=2, d=8, bs=16):
    k = np.zeros((nb, hkv, bs, d), np.uint8)
    v = np.zeros((nb, hkv, d, bs), np.uint8)
    return k, v, np.ones(nb, np.float32), np.ones(nb, np.float32)


def _bits(x):
    import torch

    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def test_append_bf16_writes_one_slot():
    rng = np.random.default_rng(1)
    nb, hkv, d, bs = 5, 2, 8, 16
    k = rng.integers(0, 65535, (nb, hkv, bs, d), dtype=np.uint16)
    v = rng.integers(0, 65535, (nb, hkv, d, bs), dtype=np.uint16)
    k0, v0 = k.copy(), v.copy()
    tables = np.array([[3, 1], [4, -1], [2, 0]], np.int32)
    lens = np.array([17, 0, 5], np.int32)
    kn = rng.integers(0, 65535, (3, hkv, d), dtype=np.uint16)
    vn = rng.integers(0, 65535, (3, hkv, d), dtype=np.uint16)
    append_kv("bf16", k, v, None, None, tables, lens, kn, vn)
    assert np.array_equal(k[1, :, 0, :], kn[0]) and np.array_equal(v[1, :, :, 0], vn[0])
    assert np.array_equal(k[2, :, 4, :], kn[2]) and np.array_equal(v[2, :, :, 4], vn[2])
    mask = np.ones(k.shape, bool)
    mask[1, :, 0, :] = False
    mask[2, :, 4, :] = False
    assert np.array_equal(k[mask], k0[mask])
    mask = np.ones(v.shape, bool)
    mask[1, :, :, 0] = False
    mask[2, :, :, 4] = False
    assert np.array_equal(v[mask], v0[mask])


def test_append_fp8_scale_policy():
    k, v, ks, vs = _fp8_cache()
    tables = np.array([[2]], np.int32)
    rng = np.random.default_rng(2)
    # token 0 opens block 2: scale = amax / 448, the amax element encodes to +-448
    x0 = rng.normal(0, 1, (1, 2, 8)).astype(np.float32)
    b0 = _bits(x0)
    append_kv("fp8", k, v, ks, vs, tables, np.array([1]), b0, b0)
    amax = np.float32(np.max(np.abs((b0.astype(np.uint32) << 16).view(np.float32))))
    assert ks[2] == np.float32(amax / np.float32(448)) and vs[2] == ks[2]
    assert np.max(k[2, :, 0, :] & 0x7F) == 0x7E
    dec0 = TABLE[k[2, :, 0, :]] * ks[2]
    x0f = (b0.astype(np.uint32) << 16).view(np.float32)[0]
    assert np.all(np.abs(dec0 - x0f) <= np.abs(x0f) * 2.0 ** -4 + ks[2] * 2.0 ** -10)
    # token 1 within range: scale kept, earlier codes untouched
    s1 = ks[2]
    before = k[2, :, 0, :].copy()
    b1 = _bits(x0 * 0.5)
    append_kv("fp8", k, v, ks, vs, tables, np.array([2]), b1, b1)
    assert ks[2] == s1 and np.array_equal(k[2, :, 0, :], before)
    # token 2 four times larger: the scale grows and the earlier codes are re-encoded
    before_v = v[2, :, :, 0].copy()
    b2 = _bits(x0 * 4)
    append_kv("fp8", k, v, ks, vs, tables, np.array([3]), b2, b2)
    assert ks[2] > s1 and vs[2] == ks[2]
    assert np.array_equal(k[2, :, 0, :], e4m3_encode(TABLE[before] * s1 / ks[2]))
    assert np.array_equal(v[2, :, :, 0], e4m3_encode(TABLE[before_v] * s1 / vs[2]))
    assert np.max(k[2, :, 2, :] & 0x7F) == 0x7E
    # the re-encoded first token still decodes to its values within the new step size
    dec = TABLE[k[2, :, 0, :]] * ks[2]
    assert np.all(np.abs(dec - x0f) <= np.abs(x0f) * 2.0 ** -3 + ks[2] * 2.0 ** -9)


def test_copy_blocks_oracle():
    k, v, ks, vs = _fp8_cache()
    k[1] = 7
    v[1] = 9
    ks[1] = 0.5
    copy_blocks(k, v, ks, vs, [(1, 4), (2, 2), (9, 3)])
    assert (k[4] == 7).all() and (v[4] == 9).all() and ks[4] == 0.5 and (k[3] == 0).all()


def test_fork_tables_example_and_invariants():
    pt = np.array([[10, 11, 12, -1], [20, 21, -1, -1]], np.int32)
    pl = np.array([40, 20], np.int32)
    t, c, used = fork_tables(pt, pl, 16, [0, 0, 1, 1], [40, 33, 20, 16], [100, 101, 102, 103])
    assert t.tolist() == [[10, 11, 100, -1], [10, 11, 101, -1], [20, 102, -1, -1], [20, -1, -1, -1]]
    assert c.tolist() == [[12, 100], [12, 101], [21, 102]] and used == 3


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_host_fork_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    npar, maxb, bs = 12, 9, 16
    pl = rng.integers(0, maxb * bs + 1, npar).astype(np.int32)
    pt = np.full((npar, maxb), -1, np.int32)
    nxt = 0
    for i in range(npar):
        nblk = -(-int(pl[i]) // bs)
        pt[i, :nblk] = np.arange(nxt, nxt + nblk)
        nxt += nblk
    cp = rng.integers(0, npar, 30).astype(np.int32)
    cl = np.array([rng.integers(0, pl[p] + 1) for p in cp], np.int32)
    free = np.arange(nxt, nxt + 40, dtype=np.int32)
    t, c, u = tts_fork_tables(pt, pl, bs, cp, cl, free)
    to, co, uo = fork_tables(pt, pl, bs, cp, cl, free)
    assert np.array_equal(t, to) and np.array_equal(c, co) and u == uo


def test_host_fork_errors():
    pt = np.array([[1, 2]], np.int32)
    with pytest.raises(TTSError):
        tts_fork_tables(pt, [20], 16, [1], [5], [9])  # bad parent
    with pytest.raises(TTSError):
        tts_fork_tables(pt, [20], 16, [0], [21], [9])  # longer than the parent
    with pytest.raises(TTSError):
        tts_fork_tables(pt, [20], 16, [0, 0], [5, 6], [9])  # not enough free blocks


# ---- truncation of duplicated beams (Sec. 4.1, Alg. 1 DuplicateThenTruncate) -------------

def test_truncated_lengths_hand_derived():
    """Parents of lengths 100 and 50 with 20 and 0 speculative tokens; children 0, 0, 0, 1, 1.
    The first child of each parent is its original: 100 and 50. With R = 0.85, sigma = 0.1:
    z = 1 -> 0.95 * 20 = 19 kept -> 99; z = -2 -> 0.65 * 20 = 13 -> 93; parent 1 has nothing
    speculative -> 50 whatever z."""
    from oracle.kv_ops import truncated_lengths

    cp = [0, 0, 0, 1, 1]
    got = truncated_lengths(cp, [100, 50], [20, 0], 0.85, 0.1, [5.0, 1.0, -2.0, 0.0, -3.0])
    assert got.tolist() == [100, 99, 93, 50, 50]
    # clipping: z = 3 -> 1.15 -> 1 (all 20 kept); z = -9 -> -0.05 -> 0 (none)
    assert truncated_lengths([0, 0, 0], [100], [20], 0.85, 0.1, [0.0, 3.0, -9.0]).tolist() == [100, 100, 80]
    # R = 1 with no spread keeps everything; R = 0 drops every speculative token
    assert truncated_lengths([0, 0], [30], [7], 1.0, 0.0, [0.0, 0.5]).tolist() == [30, 30]
    assert truncated_lengths([0, 0], [30], [7], 0.0, 0.0, [0.0, 0.5]).tolist() == [30, 23]
    # z = 0 rounds R * spec half up: 0.5 * 7 = 3.5 -> 4
    assert truncated_lengths([0, 0], [30], [7], 0.5, 0.1, [0.0, 0.0]).tolist() == [30, 27]


def test_truncated_fraction_follows_the_clipped_normal():
    """Over many duplicates the kept fraction averages E[clip(N(R, sigma^2), 0, 1)], computed by
    numerical integration of the normal density (scipy), within four standard errors."""
    from scipy import integrate, stats

    from oracle.kv_ops import truncated_lengths

    rng = np.random.default_rng(11)
    n, spec = 20000, 1000
    for ratio, sigma in [(0.85, 0.1), (0.5, 0.3)]:
        z = rng.standard_normal(n + 1)
        lens = truncated_lengths(np.zeros(n + 1, np.int32), [5000], [spec], ratio, sigma, z)[1:]
        frac = (lens - (5000 - spec)) / spec
        want = integrate.quad(lambda x: min(max(ratio + sigma * x, 0.0), 1.0) * stats.norm.pdf(x), -12, 12,
                              points=[(0 - ratio) / sigma, (1 - ratio) / sigma])[0]
        assert abs(frac.mean() - want) <= 4 * frac.std() / np.sqrt(n) + 0.5 / spec
        assert frac.min() >= 0 and frac.max() <= 1


def test_library_truncated_lengths_match_oracle():
    from oracle.kv_ops import truncated_lengths
    from paper_2509_00195_amd import tts_truncated_lengths

    rng = np.random.default_rng(12)
    for _ in range(200):
        npar = int(rng.integers(1, 9))
        plens = rng.integers(0, 300, npar).astype(np.int32)
        pspec = np.array([rng.integers(0, L + 1) for L in plens], np.int32)
        cp = np.sort(rng.integers(0, npar, int(rng.integers(1, 30)))).astype(np.int32)
        ratio, sigma = float(rng.uniform(-0.2, 1.2)), float(rng.choice([0.0, 0.05, 0.1, 0.5]))
        z = rng.standard_normal(len(cp))
        z[rng.random(len(cp)) < 0.2] = 0.0  # exact halves
        assert np.array_equal(tts_truncated_lengths(cp, plens, pspec, ratio, sigma, z),
                              truncated_lengths(cp, plens, pspec, ratio, sigma, z))


def test_library_truncated_lengths_errors():
    from paper_2509_00195_amd import TTSError, tts_truncated_lengths

    with pytest.raises(TTSError):
        tts_truncated_lengths([0, 2], [10, 10], [1, 1], 0.85, 0.1, [0.0, 0.0])  # bad parent
    with pytest.raises(TTSError):
        tts_truncated_lengths([0, 0], [10], [11], 0.85, 0.1, [0.0, 0.0])  # more speculative than tokens
    with pytest.raises(TTSError):
        tts_truncated_lengths([0, 0], [10], [1], 0.85, -0.1, [0.0, 0.0])  # negative spread
    with pytest.raises(TTSError):
        tts_truncated_lengths([0, 0], [10], [1], 0.85, 0.1, [0.0, float("nan")])
