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
