"""Roofline-guided KV allocation: the library's search against the oracle (CPU).

Pins of the oracle: its linear search is the best pair on the memory
boundary (brute force over boundary pairs); where both stage times fall
as their batches grow (weight-bound stages), the best pair overall lies
on the boundary, as the paper argues (brute force over every feasible
pair); unlimited memory gives one batch per stage; scaling the hardware
rates scales every time and keeps the choice. The library's search,
times and errors are then checked against the oracle, and its speed
against the paper's < 1 ms.
"""

from __future__ import annotations

import time

import numpy as np
import pytest

from oracle.kv_alloc import AllocProblem, ModelCost, brute_force, search, total_time
from paper_2509_00195_amd import TTSError, tts_kv_alloc_search, tts_kv_alloc_time
from paper_2509_00195_amd.tts import tts_alloc_problem, tts_model_cost


def _lib(p: AllocProblem) -> tts_alloc_problem:
    mc = lambda m: tts_model_cost(m.params, m.weight_bytes, m.kv_bytes_per_token, m.num_layers, m.attn_dim)  # noqa
    return tts_alloc_problem(mc(p.verifier), mc(p.generator), p.num_requests, p.verify_len, p.decode_len,
                             p.mem_bytes, p.peak_flops, p.peak_bw)


def _random_problem(rng, n=None, weight_bound=False) -> AllocProblem:
    def model():
        params = float(rng.choice([0.5e9, 1.5e9, 7e9]))
        kv = float(rng.choice([14336, 28672, 57344]))
        wb = 2 * params * (1e3 if weight_bound else 1.0)
        return ModelCost(params, wb, kv, int(rng.choice([24, 28])), int(rng.choice([1536, 3584])))

    v, g = model(), model()
    n = int(n or rng.integers(1, 80))
    s, sd = int(rng.integers(64, 4096)), int(rng.integers(64, 4096))
    need = v.kv_bytes_per_token * s + g.kv_bytes_per_token * sd
    mem = need * float(rng.uniform(1.0, 2.5 * n))
    return AllocProblem(v, g, n, s, sd, mem, float(rng.choice([80e12, 165e12, 2.5e15])),
                        float(rng.choice([1e12, 8e12])))


@pytest.mark.parametrize("seed", range(6))
def test_oracle_search_is_best_boundary_pair(seed):
    rng = np.random.default_rng(seed)
    for _ in range(20):
        p = _random_problem(rng)
        assert search(p) == brute_force(p, boundary_only=True)


def _stage_times_fall(p: AllocProblem) -> bool:
    """The paper's premise: each stage's total time does not grow with its batch."""
    n = p.num_requests
    tp = [total_time(p, b, 1)[1] for b in range(1, n + 1)]
    td = [total_time(p, 1, b)[2] for b in range(1, n + 1)]
    return all(x >= y for x, y in zip(tp, tp[1:])) and all(x >= y for x, y in zip(td, td[1:]))


@pytest.mark.parametrize("seed", range(4))
def test_boundary_is_optimal_when_stage_times_fall(seed):
    rng = np.random.default_rng(100 + seed)
    checked = 0
    for _ in range(40):
        p = _random_problem(rng, n=int(rng.choice([1, 2, 4, 8, 16, 32])), weight_bound=True)
        if not _stage_times_fall(p):
            continue
        checked += 1
        assert search(p)[2] == brute_force(p)[2]
    assert checked >= 5


def test_unlimited_memory_gives_one_batch_per_stage():
    rng = np.random.default_rng(7)
    p = _random_problem(rng, n=40, weight_bound=True)
    p.mem_bytes = 1e30
    assert search(p)[:2] == (40, 40)


def test_scaling_rates_scales_times():
    rng = np.random.default_rng(8)
    p = _random_problem(rng, n=33)
    b = search(p)
    p.peak_flops *= 0.5
    p.peak_bw *= 0.5
    b2 = search(p)
    assert b2[:2] == b[:2] and b2[2] == pytest.approx(2 * b[2], rel=1e-12)


def test_boundary_can_miss_the_optimum_with_batch_rounding():
    """With ceil(N / B) batches, a larger decode batch can cost more (same batch count, more
    work per batch): the best pair overall is then off the boundary. Documents why the
    search is only the best boundary pair."""
    # compute-bound stages (tiny weights, fast memory): a batch's time grows with its size
    v = ModelCost(1e9, 1e3, 1000.0, 1, 1)
    g = ModelCost(3e9, 1e3, 1000.0, 1, 1)
    p = AllocProblem(v, g, 3, 100, 100, 3e5, 1e12, 1e15)  # room for 3 sequences of either stage
    lin, every = search(p), brute_force(p)
    assert every[2] < lin[2]
    bp, bd = every[:2]
    from oracle.kv_alloc import fits

    assert bd < p.num_requests and fits(p, bp, bd + 1)  # the overall best leaves memory unused


@pytest.mark.parametrize("seed", range(6))
def test_library_matches_oracle(seed):
    rng = np.random.default_rng(200 + seed)
    for _ in range(25):
        p = _random_problem(rng, weight_bound=bool(seed % 2))
        want = search(p)
        got = tts_kv_alloc_search(_lib(p))
        if (got.b_pre, got.b_dec) != want[:2]:  # only a tie may differ
            assert got.t_tot == pytest.approx(want[2], rel=1e-12)
            assert total_time(p, got.b_pre, got.b_dec)[0] == pytest.approx(want[2], rel=1e-12)
        assert got.t_tot == pytest.approx(want[2], rel=1e-12)
        t = tts_kv_alloc_time(_lib(p), want[0], want[1])
        tot, tp, td = total_time(p, want[0], want[1])
        assert (t.t_tot, t.t_pre, t.t_dec) == pytest.approx((tot, tp, td), rel=1e-12)


def test_library_errors():
    rng = np.random.default_rng(9)
    p = _random_problem(rng, n=8)
    p.mem_bytes = p.verifier.kv_bytes_per_token * p.verify_len  # no room for a decode sequence
    with pytest.raises(TTSError):
        tts_kv_alloc_search(_lib(p))
    p.mem_bytes = 1e12
    p.num_requests = 0
    with pytest.raises(TTSError):
        tts_kv_alloc_search(_lib(p))
    p.num_requests = 4
    with pytest.raises(TTSError):
        tts_kv_alloc_time(_lib(p), 0, 1)


def test_search_is_fast():
    """The paper's searcher takes < 1 ms on one CPU thread; 7B generator + 1.5B verifier, 512 requests."""
    v = ModelCost(1.5e9, 3.1e9, 28 * 2 * 128 * 2 * 2, 28, 12 * 128)
    g = ModelCost(7.6e9, 15.2e9, 28 * 4 * 128 * 2 * 2, 28, 28 * 128)
    p = _lib(AllocProblem(v, g, 512, 2048, 2048, 0.9 * 288e9 - 18.3e9, 2.5e15, 8e12))
    tts_kv_alloc_search(p)
    t0 = time.perf_counter()
    for _ in range(200):
        tts_kv_alloc_search(p)
    assert (time.perf_counter() - t0) / 200 < 1e-3


# ---- hand-derived values (Sec. 4.3, T_tot and the roofline stage time) -------------------
#
# A one-layer toy pair whose counts are worked out by hand, so that a slip in the oracle's
# arithmetic (a factor in a FLOP or byte count, s^2 for s (s + 1), c = S_dec for S_dec / 2,
# floor for ceil in the batch counts) changes a number below.
#   verifier : params 1000, weights 2000 B, 10 B of KV per token, L = 1, d = 4
#   generator: params  500, weights 1000 B,  8 B of KV per token, L = 1, d = 2
#   N = 5 requests, S = 3 verifier tokens, S_dec = 4 generated tokens (c = S_dec / 2 = 2)
# Prefill of b = 2:  flops 2*1000*2*3 + 2*1*4*2*3*(3+1) = 12000 + 192 = 12192
#                    bytes 2000 + 2*10*3 = 2060;   ceil(5/2) = 3 batches
# Decode of b = 3:   flops 2*500*3 + 4*1*2*3*2 = 3000 + 48 = 3048
#                    bytes 1000 + 3*8*2 = 1048;    ceil(5/3) = 2 batches, S_dec = 4 steps each
# Memory-bound rates (P = 1000 flop/s, BW = 100 B/s): prefill max(12.192, 20.6) = 20.6 s,
#   T_pre = 3 * 20.6 = 61.8; decode max(3.048, 10.48) = 10.48 s, T_dec = 2 * 4 * 10.48 = 83.84.
# Compute-bound rates (P = 100 flop/s, BW = 1000 B/s): prefill max(121.92, 2.06) = 121.92,
#   T_pre = 365.76; decode max(30.48, 1.048) = 30.48, T_dec = 243.84.

def _toy(pf, bw, mem=1e9):
    v = ModelCost(1000.0, 2000.0, 10.0, 1, 4)
    g = ModelCost(500.0, 1000.0, 8.0, 1, 2)
    return AllocProblem(v, g, 5, 3, 4, mem, pf, bw)


@pytest.mark.parametrize("pf,bw,want", [
    (1000.0, 100.0, (61.8 + 83.84, 61.8, 83.84)),     # both stages memory-bound
    (100.0, 1000.0, (365.76 + 243.84, 365.76, 243.84)),  # both stages compute-bound
])
def test_total_time_hand_derived(pf, bw, want):
    p = _toy(pf, bw)
    assert total_time(p, 2, 3) == pytest.approx(want, rel=1e-12)
    t = tts_kv_alloc_time(_lib(p), 2, 3)
    assert (t.t_tot, t.t_pre, t.t_dec) == pytest.approx(want, rel=1e-12)


def test_search_hand_derived():
    """M = 130 B; one prefill sequence holds 10*3 = 30 B, one decode sequence 8*4 = 32 B.
    Memory-bound rates (P = 1000, BW = 100), the decode batch on the boundary:
      B_pre 1: B_dec = floor(100/32) = 3; prefill(1) max(6096/1000, 2030/100) = 20.3, 5 batches
               = 101.5; decode(3) = 83.84 (above)                            T_tot = 185.34
      B_pre 2: B_dec = floor(70/32) = 2; 61.8 + decode(2): max(2032/1000, 1032/100) = 10.32,
               ceil(5/2) * 4 * 10.32 = 123.84                                 T_tot = 185.64
      B_pre 3: B_dec = floor(40/32) = 1; prefill(3) max(18288/1000, 2090/100) = 20.9, 2 batches
               = 41.8; decode(1) max(1016/1000, 1016/100) = 10.16, 5 * 4 * 10.16 = 203.2
                                                                              T_tot = 245.0
      B_pre 4: 130 - 120 = 10 B leaves no room for a decode sequence: the search stops.
    The best pair is (1, 3) at 185.34 s."""
    p = _toy(1000.0, 100.0, mem=130.0)
    bp, bd, t = search(p)
    assert (bp, bd) == (1, 3) and t == pytest.approx(185.34, rel=1e-12)
    assert total_time(p, 2, 2)[0] == pytest.approx(185.64, rel=1e-12)
    assert total_time(p, 3, 1)[0] == pytest.approx(245.0, rel=1e-12)
    got = tts_kv_alloc_search(_lib(p))
    assert (got.b_pre, got.b_dec) == (1, 3) and got.t_tot == pytest.approx(185.34, rel=1e-12)
