"""Oracle of dynamic prefix-aware scheduling (Sec. 4.2) -- test infrastructure.

The scheduler orders the active reasoning paths (CoTs) so that consecutive
ones share long prefixes: starting from the first CoT, the next is always
the remaining CoT with the largest shared prefix P(c_k, c_i) with the one
just scheduled (the paper's greedy invariant; ties to the earliest in the
input). The order is then cut into batches -- each the largest run of
consecutive CoTs whose trie fits the memory budget -- and a schedule's
eviction cost is sum_i (Nodes(T_i) - P(T_i, T_{i+1})), with Nodes the trie's
(weighted) node count and P the nodes two consecutive tries share. Plain
Python over node-id lists.
"""

from __future__ import annotations

from typing import List, Optional, Sequence


def shared_prefix(a: Sequence[int], b: Sequence[int]) -> int:
    n = 0
    for x, y in zip(a, b):
        if x != y:
            break
        n += 1
    return n


def score(order: Sequence[int], cots: Sequence[Sequence[int]]) -> int:
    """Sum of shared prefixes of consecutive CoTs."""
    return sum(shared_prefix(cots[order[k]], cots[order[k + 1]]) for k in range(len(order) - 1))


def greedy_order(cots: Sequence[Sequence[int]]) -> List[int]:
    if not cots:
        return []
    rest = list(range(1, len(cots)))
    order = [0]
    while rest:
        last = cots[order[-1]]
        best = rest[0]
        for i in rest[1:]:
            if shared_prefix(last, cots[i]) > shared_prefix(last, cots[best]):
                best = i
        rest.remove(best)
        order.append(best)
    return order


def batches(order: Sequence[int], cots: Sequence[Sequence[int]], budget: int,
            weight: Optional[Sequence[int]] = None) -> List[List[int]]:
    w = (lambda v: 1) if weight is None else (lambda v: int(weight[v]))
    out: List[List[int]] = []
    cur: List[int] = []
    nodes: set = set()
    for c in order:
        grown = nodes | set(cots[c])
        if cur and sum(w(v) for v in grown) > budget:
            out.append(cur)
            cur, nodes = [], set()
            grown = set(cots[c])
        cur.append(c)
        nodes = grown
    if cur:
        out.append(cur)
    return out


def eviction_cost(batch_list, cots, weight=None) -> int:
    w = (lambda v: 1) if weight is None else (lambda v: int(weight[v]))
    tries = [set().union(*[set(cots[c]) for c in b]) for b in batch_list]
    cost = 0
    for i, t in enumerate(tries):
        shared = tries[i + 1] & t if i + 1 < len(tries) else set()
        cost += sum(w(v) for v in t) - sum(w(v) for v in shared)
    return cost
