"""Prefix-aware scheduling (CPU): the oracle against brute force and the paper's
claims, the library against the oracle and against the canonical beam order of
the prefix metadata.

Pins of the oracle: on random beam-search trees (prefix similarities, so shared
prefixes nest) the greedy order reaches the best score over every permutation
(brute force, up to 7 CoTs), and no swap of two CoTs improves it (the paper's
local optimality); batches are maximal runs under the budget; the eviction cost
equals the sum of trie sizes minus the sum of consecutive overlaps.
"""

from __future__ import annotations

import itertools
import random

import numpy as np
import pytest

from oracle.prefix_meta import oracle_prefix_meta
from oracle.schedule import batches, eviction_cost, greedy_order, score
from paper_2509_00195_amd import tts_prefix_schedule
from tts_synth import build_tree, CONFIGS


def _tree_cots(n, rng):
    """CoTs of a random search tree: each new path branches off an existing one."""
    cots = [[0, 1]]
    nxt = 2
    while len(cots) < n:
        c = rng.choice(cots)
        d = rng.randint(1, len(c))
        k = rng.randint(1, 3)
        cots.append(c[:d] + list(range(nxt, nxt + k)))
        nxt += k
    rng.shuffle(cots)
    return cots, nxt


@pytest.mark.parametrize("seed", range(4))
def test_greedy_is_optimal_on_trees(seed):
    rng = random.Random(seed)
    for _ in range(60):
        cots, _ = _tree_cots(rng.randint(2, 7), rng)
        g = greedy_order(cots)
        best = max(score(p, cots) for p in itertools.permutations(range(len(cots))))
        assert score(g, cots) == best


@pytest.mark.parametrize("seed", range(3))
def test_no_swap_improves_greedy(seed):
    rng = random.Random(10 + seed)
    for _ in range(40):
        cots, _ = _tree_cots(rng.randint(3, 12), rng)
        g = greedy_order(cots)
        s = score(g, cots)
        for i in range(len(g)):
            for j in range(i + 1, len(g)):
                o = list(g)
                o[i], o[j] = o[j], o[i]
                assert score(o, cots) <= s


def test_batches_are_maximal_and_cost_identity():
    rng = random.Random(3)
    for _ in range(30):
        cots, nn = _tree_cots(rng.randint(2, 15), rng)
        weight = [rng.randint(1, 9) for _ in range(nn)]
        order = greedy_order(cots)
        budget = rng.randint(5, 60)
        bl = batches(order, cots, budget, weight)
        assert [c for b in bl for c in b] == order
        size = lambda b: sum(weight[v] for v in set().union(*[set(cots[c]) for c in b]))  # noqa: E731
        for i, b in enumerate(bl):
            assert len(b) == 1 or size(b) <= budget
            if i + 1 < len(bl):
                assert size(b + [bl[i + 1][0]]) > budget  # could not take the next CoT
        tries = [set().union(*[set(cots[c]) for c in b]) for b in bl]
        overlap = sum(sum(weight[v] for v in tries[i] & tries[i + 1]) for i in range(len(tries) - 1))
        assert eviction_cost(bl, cots, weight) == sum(size(b) for b in bl) - overlap


@pytest.mark.parametrize("seed", range(5))
def test_library_matches_oracle(seed):
    rng = random.Random(100 + seed)
    for _ in range(20):
        cots, nn = _tree_cots(rng.randint(1, 40), rng)
        weight = [rng.randint(1, 9) for _ in range(nn)] if seed % 2 else None
        budget = rng.randint(3, 80)
        order, bl, sc, co = tts_prefix_schedule(cots, nn, budget, weight)
        go = greedy_order(cots)
        ob = batches(go, cots, budget, weight)
        assert order.tolist() == go and bl == ob
        assert sc == score(go, cots) and co == eviction_cost(ob, cots, weight)


@pytest.mark.parametrize("name", ["1p5b16", "7b64"])
def test_schedule_is_the_metadata_beam_order(name):
    """On a beam-search tree, CoTs = each beam's block-id path: the greedy order groups the
    beams exactly as the prefix metadata's canonical permutation (children by their
    smallest beam, beams at one node in input order)."""
    from tts_synth import workload_from_tree
    from tts_synth.workload import AttnShape

    tree = build_tree(CONFIGS[name], 0)
    w = workload_from_tree(AttnShape(2, 1, 8, 16, "f32", "f32"), tree, 0, name=name)
    cots = []
    for b in range(w.num_seqs):
        nblk = int(w.seq_lens[b]) // 16  # full blocks (the shared ones); the partial block is private
        cots.append(w.block_tables[b, :nblk].tolist() + [10 ** 8 + b])  # a private leaf per beam
    order, _, _, _ = tts_prefix_schedule(cots, 10 ** 8 + w.num_seqs, 10 ** 9)
    meta = oracle_prefix_meta(w.req_seq_offsets, w.block_tables, w.seq_lens, 16)
    assert order.tolist() == list(meta["perm"])


# ---- hand-derived values (Sec. 4.2: Cost = sum_i Nodes(T_i) - P(T_i, T_{i+1})) -----------
#
# Five CoTs (node-id paths): c0 = [1,2,3], c1 = [1,5], c2 = [1,2,6], c3 = [1,2,7], c4 = [1,8].
GOLD_COTS = [[1, 2, 3], [1, 5], [1, 2, 6], [1, 2, 7], [1, 8]]


def test_eviction_cost_hand_derived():
    """CoTs c0 = [1,2,3], c1 = [1,4], c2 = [1,4,5], c3 = [1,6], c4 = [1,2,7] in the batches
    [c0 c3 c4], [c1], [c2]: tries T0 = {1,2,3,6,7}, T1 = {1,4}, T2 = {1,4,5};
    T0 & T1 = {1}, T1 & T2 = {1,4}, and the last trie has no successor.
    Unit weights: (5 - 1) + (2 - 2) + (3 - 0) = 7. With weight(v) = v: T0 = 19, T1 = 5,
    T2 = 10, overlaps 1 and 5: (19 - 1) + (5 - 5) + 10 = 28.
    Slips this separates: the previous trie's overlap instead of the next one's gives 8, the
    last trie's overlap with the first 6, dropping the last trie 4, summing per CoT instead of
    per trie (3 + 2 + 3 + 2 + 3 - 1 - 1 - 1 - 2) 8."""
    cots = [[1, 2, 3], [1, 4], [1, 4, 5], [1, 6], [1, 2, 7]]
    bl = [[0, 3, 4], [1], [2]]
    assert eviction_cost(bl, cots) == 7
    assert eviction_cost(bl, cots, list(range(8))) == 28


def test_schedule_hand_derived():
    """Greedy from c0 = [1,2,3]: shared prefixes with c1..c4 are 1, 2, 2, 1 -> c2 (earliest
    of the ties); from c2: c1 1, c3 2, c4 1 -> c3; from c3: c1 1, c4 1 -> c1; then c4.
    Order [0, 2, 3, 1, 4], score 2 + 2 + 1 + 1 = 6.
    Budget 5 (unit weights): c0 -> 3 nodes, + c2 -> 4, + c3 -> {1,2,3,6,7} = 5, + c1 would be
    6 > 5, so the batches are [0 2 3], [1 4] ({1,5,8}); cost (5 - |{1}|) + 3 = 7.
    Budget 20 with weight(v) = v: 6, 12, 19, then + 5 = 24 > 20; same batches; cost
    (19 - 1) + (1 + 5 + 8) = 32."""
    assert greedy_order(GOLD_COTS) == [0, 2, 3, 1, 4]
    assert score([0, 2, 3, 1, 4], GOLD_COTS) == 6
    assert batches([0, 2, 3, 1, 4], GOLD_COTS, 5) == [[0, 2, 3], [1, 4]]
    assert batches([0, 2, 3, 1, 4], GOLD_COTS, 20, list(range(9))) == [[0, 2, 3], [1, 4]]
    assert eviction_cost([[0, 2, 3], [1, 4]], GOLD_COTS) == 7
    order, bl, sc, co = tts_prefix_schedule(GOLD_COTS, 9, 5)
    assert order.tolist() == [0, 2, 3, 1, 4] and bl == [[0, 2, 3], [1, 4]] and sc == 6 and co == 7
    order, bl, sc, co = tts_prefix_schedule(GOLD_COTS, 9, 20, list(range(9)))
    assert bl == [[0, 2, 3], [1, 4]] and co == 32
