"""Pins for the CPU attention oracle (no GPU).

The oracle must match things other than itself: a float64 library routine
(torch SDPA) on dense sequences scattered into a paged cache by an
independent helper, closed forms of softmax attention, and the invariants
any correct decode attention obeys.
"""

import math

import numpy as np
import pytest
import torch

from oracle import e4m3_table, oracle_attn
from tests._paged import bf16_bits, bf16_round, dense_reference, scatter_paged

BS = 16


def run_oracle(q, kc, vc, tables, lens, hq, hkv, q_dtype="f32", kv_dtype="f32", ks=None, vsc=None, scale=None):
    return oracle_attn(q, kc, vc, ks, vsc, tables, lens, num_q_heads=hq, num_kv_heads=hkv, block_size=BS,
                       q_dtype=q_dtype, kv_dtype=kv_dtype, scale=scale)


def rand_dense(rng, lens, hkv, d):
    ks = [rng.standard_normal((hkv, L, d)).astype(np.float32) for L in lens]
    vs = [rng.standard_normal((hkv, L, d)).astype(np.float32) for L in lens]
    return ks, vs


@pytest.mark.parametrize("hq,hkv,d", [(4, 1, 64), (12, 2, 128), (28, 4, 128), (6, 6, 32)])
def test_matches_sdpa_f64_fp32_kv(hq, hkv, d):
    rng = np.random.default_rng(hq * 100 + d)
    lens = [1, 15, 16, 17, 33, 70, 0, 5]
    ks, vs = rand_dense(rng, lens, hkv, d)
    q = rng.standard_normal((len(lens), hq, d)).astype(np.float32)
    kc, vc, tables, L = scatter_paged(ks, vs, BS, rng)
    got = run_oracle(q, kc, vc, tables, L, hq, hkv)
    ref = dense_reference(q, ks, vs)
    assert np.max(np.abs(got - ref)) < 1e-5
    assert np.all(got[6] == 0.0)  # seq_len == 0 -> zero row


def test_matches_sdpa_f64_bf16_kv_and_scale():
    rng = np.random.default_rng(7)
    hq, hkv, d = 28, 4, 128
    lens = [3, 16, 200, 31]
    ks, vs = rand_dense(rng, lens, hkv, d)
    q = rng.standard_normal((len(lens), hq, d)).astype(np.float32)
    kc, vc, tables, L = scatter_paged(ks, vs, BS, rng, dtype="bf16")
    qb = bf16_bits(q)
    got = run_oracle(qb, kc, vc, tables, L, hq, hkv, "bf16", "bf16", scale=0.05)
    ref = dense_reference(bf16_round(q), [bf16_round(k) for k in ks], [bf16_round(v) for v in vs], scale=0.05)
    assert np.max(np.abs(got - ref)) < 1e-5


def test_fp8_kv_matches_library_decode():
    """fp8 codes + per-block scales vs torch's float8_e4m3fn decode in float64."""
    rng = np.random.default_rng(11)
    hq, hkv, d = 8, 2, 64
    lens = [40, 16, 9]
    s = len(lens)
    nblk = [-(-L // BS) for L in lens]
    pool = sum(nblk) + 2
    kcodes = rng.integers(0, 256, size=(pool, hkv, BS, d), dtype=np.uint8)
    vcodes = rng.integers(0, 256, size=(pool, hkv, d, BS), dtype=np.uint8)
    # Avoid NaN codes (0x7F / 0xFF) in visible slots.
    kcodes[(kcodes & 0x7F) == 0x7F] = 0x30
    vcodes[(vcodes & 0x7F) == 0x7F] = 0x31
    k_scale = rng.uniform(0.001, 0.02, size=pool).astype(np.float32)
    v_scale = rng.uniform(0.001, 0.02, size=pool).astype(np.float32)
    ids = rng.permutation(pool)
    tables = np.full((s, max(nblk)), -1, dtype=np.int32)
    n = 0
    for b in range(s):
        tables[b, : nblk[b]] = ids[n: n + nblk[b]]
        n += nblk[b]
    q = rng.standard_normal((s, hq, d)).astype(np.float32)
    got = run_oracle(q, kcodes, vcodes, tables, np.array(lens, np.int32), hq, hkv, "f32", "fp8", k_scale, v_scale)
    lib = lambda c: torch.from_numpy(c).view(torch.float8_e4m3fn).double().numpy()  # noqa: E731
    ks, vs = [], []
    for b in range(s):
        kk = np.concatenate([lib(kcodes[p]) * float(k_scale[p]) for p in tables[b, : nblk[b]]], axis=1)
        vv = np.concatenate([lib(vcodes[p]).swapaxes(1, 2) * float(v_scale[p]) for p in tables[b, : nblk[b]]], axis=1)
        ks.append(kk[:, : lens[b]])
        vs.append(vv[:, : lens[b]])
    ref = dense_reference(q, ks, vs)
    assert np.max(np.abs(got - ref)) < 1e-5


# ---------------------------------------------------------------- closed forms


def _single(q, k, v, scale=None):
    """Oracle on one beam, one KV head, dense K/V [L, D]."""
    rng = np.random.default_rng(0)
    kc, vc, tables, L = scatter_paged([k[None]], [v[None]], BS, rng)
    hq = q.shape[0]
    return run_oracle(q[None].astype(np.float32), kc, vc, tables, L, hq, 1, scale=scale)[0]


def test_single_key_returns_its_value_exactly():
    rng = np.random.default_rng(1)
    k = rng.standard_normal((1, 64)).astype(np.float32)
    v = rng.standard_normal((1, 64)).astype(np.float32)
    q = rng.standard_normal((3, 64)).astype(np.float32) * 10
    out = _single(q, k, v)
    assert np.array_equal(out, np.repeat(v, 3, axis=0))


def test_identical_keys_give_mean_of_values():
    rng = np.random.default_rng(2)
    L = 37
    k = np.repeat(rng.standard_normal((1, 64)).astype(np.float32), L, axis=0)
    v = rng.standard_normal((L, 64)).astype(np.float32)
    q = rng.standard_normal((2, 64)).astype(np.float32)
    out = _single(q, k, v)
    assert np.max(np.abs(out - v.astype(np.float64).mean(axis=0))) < 1e-6


def test_zero_query_gives_mean_of_values():
    rng = np.random.default_rng(3)
    L = 50
    k = rng.standard_normal((L, 64)).astype(np.float32)
    v = rng.standard_normal((L, 64)).astype(np.float32)
    out = _single(np.zeros((1, 64), np.float32), k, v)
    assert np.max(np.abs(out - v.astype(np.float64).mean(axis=0))) < 1e-6


def test_constant_values_are_returned():
    rng = np.random.default_rng(4)
    L = 29
    k = rng.standard_normal((L, 64)).astype(np.float32)
    v = np.full((L, 64), 0.375, np.float32)
    out = _single(rng.standard_normal((2, 64)).astype(np.float32), k, v)
    assert np.max(np.abs(out - 0.375)) < 1e-6


def test_two_keys_sigmoid_form():
    rng = np.random.default_rng(5)
    d = 64
    k = rng.standard_normal((2, d)).astype(np.float32)
    v = rng.standard_normal((2, d)).astype(np.float32)
    q = rng.standard_normal((1, d)).astype(np.float32)
    out = _single(q, k, v)[0]
    s0, s1 = (k.astype(np.float64) @ q[0].astype(np.float64)) / math.sqrt(d)
    w0 = 1.0 / (1.0 + math.exp(s1 - s0))
    ref = w0 * v[0] + (1.0 - w0) * v[1]
    assert np.max(np.abs(out - ref)) < 1e-6


def test_linear_in_values():
    rng = np.random.default_rng(6)
    L, d = 45, 64
    k = rng.standard_normal((L, d)).astype(np.float32)
    v1 = rng.standard_normal((L, d)).astype(np.float32)
    v2 = rng.standard_normal((L, d)).astype(np.float32)
    q = rng.standard_normal((2, d)).astype(np.float32)
    a, b = 0.5, -2.0
    lhs = _single(q, k, a * v1 + b * v2)
    rhs = a * _single(q, k, v1) + b * _single(q, k, v2)
    assert np.max(np.abs(lhs - rhs)) < 1e-5


def test_softmax_scale_is_inverse_sqrt_head_dim_by_default():
    rng = np.random.default_rng(8)
    L, d = 20, 64
    k = rng.standard_normal((L, d)).astype(np.float32)
    v = rng.standard_normal((L, d)).astype(np.float32)
    q = rng.standard_normal((1, d)).astype(np.float32)
    assert np.array_equal(_single(q, k, v), _single(q, k, v, scale=1.0 / math.sqrt(d)))
    assert not np.allclose(_single(q, k, v), _single(q, k, v, scale=1.0))


# ---------------------------------------------------------------- invariants


def _paged_case(rng, lens, hq=8, hkv=2, d=64):
    ks, vs = rand_dense(rng, lens, hkv, d)
    kc, vc, tables, L = scatter_paged(ks, vs, BS, rng)
    q = rng.standard_normal((len(lens), hq, d)).astype(np.float32)
    return q, kc, vc, tables, L, hq, hkv


def test_identical_beams_identical_outputs():
    rng = np.random.default_rng(9)
    q, kc, vc, tables, L, hq, hkv = _paged_case(rng, [50, 77])
    tables = np.vstack([tables, tables[1:2], tables[0:1]])
    L = np.concatenate([L, L[1:2], L[0:1]])
    q = np.concatenate([q, q[1:2], q[0:1]])
    out = run_oracle(q, kc, vc, tables, L, hq, hkv)
    assert np.array_equal(out[1], out[2]) and np.array_equal(out[0], out[3])


def test_physical_block_permutation_invariance():
    rng = np.random.default_rng(10)
    q, kc, vc, tables, L, hq, hkv = _paged_case(rng, [50, 77, 16, 3])
    out = run_oracle(q, kc, vc, tables, L, hq, hkv)
    pi = rng.permutation(kc.shape[0])  # new id of old block p is pi[p]
    kc2 = np.empty_like(kc)
    vc2 = np.empty_like(vc)
    kc2[pi] = kc
    vc2[pi] = vc
    t2 = np.where(tables >= 0, pi[np.maximum(tables, 0)], -1).astype(np.int32)
    out2 = run_oracle(q, kc2, vc2, t2, L, hq, hkv)
    assert np.array_equal(out, out2)


def test_beam_permutation_permutes_outputs():
    rng = np.random.default_rng(12)
    q, kc, vc, tables, L, hq, hkv = _paged_case(rng, [50, 77, 16, 3, 90])
    out = run_oracle(q, kc, vc, tables, L, hq, hkv)
    pi = rng.permutation(len(L))
    out2 = run_oracle(q[pi], kc, vc, tables[pi], L[pi], hq, hkv)
    assert np.array_equal(out[pi], out2)


def test_table_entries_past_length_and_unused_slots_are_ignored():
    rng = np.random.default_rng(13)
    q, kc, vc, tables, L, hq, hkv = _paged_case(rng, [18, 33])
    out = run_oracle(q, kc, vc, tables, L, hq, hkv)
    assert np.all(np.isfinite(out))  # unused slots are NaN in the cache
    t2 = tables.copy()
    for b in range(len(L)):
        t2[b, -(-int(L[b]) // BS):] = 10 ** 6  # would fault if read
    assert np.array_equal(out, run_oracle(q, kc, vc, t2, L, hq, hkv))


def test_gqa_mapping_is_contiguous_groups():
    """Query head h reads KV head h // (Hq/Hkv): zeroing KV head 1's values zeroes exactly heads 4..7."""
    rng = np.random.default_rng(14)
    q, kc, vc, tables, L, hq, hkv = _paged_case(rng, [40], hq=8, hkv=2)
    vc = vc.copy()
    vc[:, 1] = np.where(np.isnan(vc[:, 1]), np.nan, 0.0)
    out = run_oracle(q, kc, vc, tables, L, hq, hkv)
    assert np.all(out[0, 4:] == 0.0) and np.all(np.abs(out[0, :4]).sum(axis=1) > 0)


# ---------------------------------------------------------------- fp8 table


def test_e4m3_table_spot_values():
    t = e4m3_table()
    assert t[0x7E] == 448.0
    assert t[0x01] == 2.0 ** -9
    assert t[0x08] == 2.0 ** -6
    assert t[0x07] == 7 * 2.0 ** -9
    assert t[0x38] == 1.0
    assert t[0xB8] == -1.0
    assert np.isnan(t[0x7F]) and np.isnan(t[0xFF])
    assert t[0x00] == 0.0 and t[0x80] == 0.0 and math.copysign(1, t[0x80]) < 0


def test_e4m3_table_matches_torch_for_all_codes():
    codes = np.arange(256, dtype=np.uint8)
    lib = torch.from_numpy(codes).view(torch.float8_e4m3fn).float().numpy()
    t = e4m3_table()
    nan = np.isnan(lib)
    assert np.array_equal(nan, np.isnan(t))
    assert np.array_equal(lib[~nan], t[~nan])


def test_e4m3_to_bf16_is_exact():
    """Every finite E4M3 value is representable in bf16 (3 <= 7 mantissa bits)."""
    t = e4m3_table()
    fin = np.isfinite(t)
    back = torch.from_numpy(t[fin]).to(torch.bfloat16).float().numpy()
    assert np.array_equal(back, t[fin])


# ---- verification attention (each beam's last q_len tokens as causal queries) ----

def run_verify(q, kc, vc, tables, lens, q_len, hq, hkv, q_dtype="f32", kv_dtype="f32"):
    from oracle import oracle_verify_attn

    return oracle_verify_attn(q, kc, vc, None, None, tables, lens, q_len, num_q_heads=hq, num_kv_heads=hkv,
                              block_size=BS, q_dtype=q_dtype, kv_dtype=kv_dtype)


@pytest.mark.parametrize("q_len", [1, 3, 16])
def test_verify_matches_masked_sdpa_f64(q_len):
    """Against torch SDPA in float64 with an explicit mask: query i of a beam of length L sees
    keys 0 .. L - q_len + i."""
    rng = np.random.default_rng(40 + q_len)
    hq, hkv, d = 12, 2, 64
    lens = [q_len, q_len + 5, 40, 16 + q_len]
    ks, vs = rand_dense(rng, lens, hkv, d)
    q = rng.standard_normal((len(lens), q_len, hq, d)).astype(np.float32)
    kc, vc, tables, L = scatter_paged(ks, vs, BS, rng)
    got = run_verify(q, kc, vc, tables, L, q_len, hq, hkv)
    for b, ln in enumerate(lens):
        mask = np.arange(ln)[None, :] <= (ln - q_len + np.arange(q_len))[:, None]  # [q_len, L]
        qt = torch.from_numpy(q[b].transpose(1, 0, 2).astype(np.float64))  # [Hq, q_len, D]
        kt = torch.from_numpy(np.repeat(ks[b], hq // hkv, axis=0).astype(np.float64))
        vt = torch.from_numpy(np.repeat(vs[b], hq // hkv, axis=0).astype(np.float64))
        ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=torch.from_numpy(mask))
        assert np.max(np.abs(got[b] - ref.numpy().transpose(1, 0, 2))) < 1e-5


def test_verify_with_one_query_is_decode():
    rng = np.random.default_rng(50)
    hq, hkv, d = 8, 2, 32
    lens = [1, 17, 33]
    ks, vs = rand_dense(rng, lens, hkv, d)
    q = rng.standard_normal((len(lens), hq, d)).astype(np.float32)
    kc, vc, tables, L = scatter_paged(ks, vs, BS, rng)
    assert np.array_equal(run_verify(q[:, None], kc, vc, tables, L, 1, hq, hkv)[:, 0],
                          run_oracle(q, kc, vc, tables, L, hq, hkv))


def test_verify_is_causal():
    """Changing a key/value after query i's position leaves query i unchanged; at it, changes it."""
    rng = np.random.default_rng(51)
    hq, hkv, d, q_len = 4, 1, 32, 4
    lens = [21]
    ks, vs = rand_dense(rng, lens, hkv, d)
    q = rng.standard_normal((1, q_len, hq, d)).astype(np.float32)
    kc, vc, tables, L = scatter_paged(ks, vs, BS, rng)
    base = run_verify(q, kc, vc, tables, L, q_len, hq, hkv)
    pos = 21 - q_len + 1  # position of query 1
    blk, slot = tables[0, pos // BS], pos % BS
    kc2, vc2 = kc.copy(), vc.copy()
    kc2[blk, :, slot, :] += 3.0
    vc2[blk, :, :, slot] -= 2.0
    moved = run_verify(q, kc2, vc2, tables, L, q_len, hq, hkv)
    assert np.array_equal(moved[0, 0], base[0, 0])  # query 0 ends before that position
    assert np.max(np.abs(moved[0, 1] - base[0, 1])) > 1e-3  # query 1 sees it
