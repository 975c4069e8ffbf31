"""Oracle of the roofline-guided KV allocation (Sec. 4.3) -- test infrastructure.

The total time of N requests when the verifier prefills in batches of
B_pre and the generator decodes in batches of B_dec,

    T_tot = ceil(N / B_pre) T_pre(B_pre, S) + ceil(N / B_dec) S_dec T_dec(B_dec, S_dec / 2),

each batch time a roofline max(FLOPs / P, bytes / BW), under the budget
B_pre KV_v(S) + B_dec KV_g(S_dec) <= M. The paper's search walks every
prefill batch with the decode batch on the memory boundary and keeps the
fastest, ties to the larger decode batch. The FLOP and byte counts of a
stage are the reading used here of a decoder-only transformer (the paper
only names the roofline): prefill 2 params b s + 2 L d b s (s + 1) flops
and weights + b kv s bytes; decode 2 params b + 4 L d b c flops and
weights + b kv c bytes. Batches are capped at N.
"""

from __future__ import annotations

import math
from dataclasses import dataclass


@dataclass
class ModelCost:
    params: float
    weight_bytes: float
    kv_bytes_per_token: float
    num_layers: int
    attn_dim: int


@dataclass
class AllocProblem:
    verifier: ModelCost
    generator: ModelCost
    num_requests: int
    verify_len: int
    decode_len: int
    mem_bytes: float
    peak_flops: float
    peak_bw: float


def t_prefill(m: ModelCost, b: float, s: float, pf: float, bw: float) -> float:
    flops = 2.0 * m.params * b * s + 2.0 * m.num_layers * m.attn_dim * b * s * (s + 1.0)
    byts = m.weight_bytes + b * m.kv_bytes_per_token * s
    return max(flops / pf, byts / bw)


def t_decode(m: ModelCost, b: float, c: float, pf: float, bw: float) -> float:
    flops = 2.0 * m.params * b + 4.0 * m.num_layers * m.attn_dim * b * c
    byts = m.weight_bytes + b * m.kv_bytes_per_token * c
    return max(flops / pf, byts / bw)


def total_time(p: AllocProblem, b_pre: int, b_dec: int):
    n = float(p.num_requests)
    tp = t_prefill(p.verifier, float(b_pre), float(p.verify_len), p.peak_flops, p.peak_bw)
    td = t_decode(p.generator, float(b_dec), float(p.decode_len) / 2.0, p.peak_flops, p.peak_bw)
    t_pre = math.ceil(n / float(b_pre)) * tp
    t_dec = math.ceil(n / float(b_dec)) * float(p.decode_len) * td
    return t_pre + t_dec, t_pre, t_dec


def fits(p: AllocProblem, b_pre: int, b_dec: int) -> bool:
    return (b_pre * p.verifier.kv_bytes_per_token * p.verify_len
            + b_dec * p.generator.kv_bytes_per_token * p.decode_len) <= p.mem_bytes


def search(p: AllocProblem):
    """The paper's linear search: (b_pre, b_dec, t_tot) or None."""
    kv_pre = p.verifier.kv_bytes_per_token * p.verify_len
    kv_dec = p.generator.kv_bytes_per_token * p.decode_len
    best = None
    for bp in range(1, p.num_requests + 1):
        rest = p.mem_bytes - bp * kv_pre
        if rest < kv_dec:
            break
        bd = min(p.num_requests, int(math.floor(rest / kv_dec)))
        t = total_time(p, bp, bd)[0]
        if best is None or t < best[2] or (t == best[2] and bd > best[1]):
            best = (bp, bd, t)
    return best


def brute_force(p: AllocProblem, boundary_only: bool = False):
    """Every feasible pair (or only those whose decode batch cannot grow): the fastest, ties to larger b_dec."""
    best = None
    n = p.num_requests
    for bp in range(1, n + 1):
        for bd in range(n, 0, -1):
            if not fits(p, bp, bd):
                continue
            if boundary_only and bd < n and fits(p, bp, bd + 1):
                continue
            t = total_time(p, bp, bd)[0]
            if best is None or t < best[2] or (t == best[2] and bd > best[1]):
                best = (bp, bd, t)
    return best
