"""Seeded synthetic beam trees, paged block tables and KV storage.

The tree model follows the verifier-guided two-stage loop of the paper's
pattern analysis (Sec. 3.1): every iteration extends each of the N active
beams by one reasoning step of arbitrary length, then keeps N/B survivors and
duplicates each of them B times (beam search with a static branching factor).
Survivors are drawn at random because no verifier is run. A duplicate shares
all of its parent's *full* KV blocks and receives a fresh copy of the
parent's partially filled last block (copy-on-write at beam duplication,
Sec. 4.1 / Alg. 1 DuplicateThenTruncate). The final state is a snapshot taken
mid-step, so the beams' current step lengths are irregular (Sec. 3.2.1,
stragglers).

Nothing here computes attention or prefix metadata: the module produces only
inputs, in the storage formats the library consumes.

Storage formats
---------------
* ``k_cache``: ``[num_blocks][Hkv][block_size][D]`` (token-major inside a block)
* ``v_cache``: ``[num_blocks][Hkv][D][block_size]`` (dim-major inside a block)
* ``q``: ``[S][Hq][D]``
* bf16 tensors are held as ``uint16`` bit patterns, fp8 tensors as ``uint8``
  OCP E4M3FN codes with one fp32 scale per physical block for K and one for V
  (``k_scale``, ``v_scale``: ``[num_blocks]``), f32 tensors as ``float32``.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

BF16_NAN = np.uint16(0x7FC0)
FP8_NAN = np.uint8(0x7F)
FP8_MAX = 448.0


@dataclass(frozen=True)
class AttnShape:
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    block_size: int = 16
    q_dtype: str = "bf16"  # "f32" | "bf16"
    kv_dtype: str = "bf16"  # "f32" | "bf16" | "fp8"

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads


@dataclass(frozen=True)
class ReqSpec:
    """Shape of one request's beam tree.

    ``prompt`` is ``(lo, hi)``, drawn uniformly (inclusive). ``step`` is the
    uniform range of one reasoning step. ``rule`` selects when the search
    stops: ``"lmax"`` stops before an iteration whose full step could push
    the longest beam past ``max_len`` or once ``max_iters`` is reached;
    ``"fixed"`` runs ``round((target_median - prompt) / fixed_div)`` (at
    least 1) full iterations; ``"balanced"`` grows a complete tree instead
    (every beam of a level forks ``branch`` children, one step per level,
    until ``beams`` leaves) and then gives every leaf a private tail to a
    total length U[max_len / 2, max_len]. The last iteration is the snapshot:
    ``"none"`` appends the full step, ``"uniform"`` appends U[1, step],
    ``"lognormal"`` sets the beam's total length to
    ``clip(lognormal(ln median, sigma), len + 1, max_len)``.
    """

    beams: int
    branch: int
    prompt: Tuple[int, int]
    step: Tuple[int, int]
    max_len: int
    max_iters: int = 1 << 30
    rule: str = "lmax"
    snapshot: str = "uniform"
    lognormal_median: float = 1500.0
    lognormal_sigma: float = 0.55
    fixed_div: float = 160.0


@dataclass(frozen=True)
class WorkloadConfig:
    name: str
    shape: AttnShape
    reqs: Tuple[ReqSpec, ...]
    description: str = ""


def _repeat(spec: ReqSpec, n: int) -> Tuple[ReqSpec, ...]:
    return tuple([spec] * n)


# The five workload configurations (sizes from the paper's 1.5B-7B edge
# generator shapes; beam counts 8-512 per request, Sec. 6.1).
CONFIGS = {
    "tiny": WorkloadConfig(
        "tiny",
        AttnShape(4, 1, 64, 16, "f32", "f32"),
        (ReqSpec(beams=4, branch=4, prompt=(64, 64), step=(8, 24), max_len=1 << 20,
                 max_iters=1, snapshot="none"),),
        "1 request, 4 beams, Hq4/Hkv1, D64, 64-token shared prefix + U[8,24] suffix, fp32",
    ),
    "1p5b16": WorkloadConfig(
        "1p5b16",
        AttnShape(12, 2, 128, 16, "bf16", "bf16"),
        (ReqSpec(beams=16, branch=4, prompt=(512, 512), step=(64, 256), max_len=2048),),
        "1.5B-shaped: Hq12/Hkv2, D128, bf16 KV, 16 beams, 512-token prompt, branch 4, steps U[64,256], len<=2048",
    ),
    "7b64": WorkloadConfig(
        "7b64",
        AttnShape(28, 4, 128, 16, "bf16", "bf16"),
        (ReqSpec(beams=64, branch=4, prompt=(1024, 1024), step=(64, 256), max_len=4096),),
        "7B-shaped: Hq28/Hkv4, D128, bf16 KV, 64 beams, 1024-token prompt, branch 4, steps U[64,256], len<=4096",
    ),
    "7b64_balanced": WorkloadConfig(
        "7b64_balanced",
        AttnShape(28, 4, 128, 16, "bf16", "bf16"),
        (ReqSpec(beams=64, branch=4, prompt=(1024, 1024), step=(64, 256), max_len=4096, rule="balanced"),),
        "7B-shaped balanced tree (report only): 1024-token prompt -> 4 -> 16 -> 64 nodes of one U[64,256] step, "
        "then private tails to U[2048,4096] tokens, bf16 KV",
    ),
    "7b_straggler": WorkloadConfig(
        "7b_straggler",
        AttnShape(28, 4, 128, 16, "bf16", "bf16"),
        _repeat(ReqSpec(beams=32, branch=4, prompt=(256, 1024), step=(64, 256), max_len=8192,
                        rule="fixed", snapshot="lognormal"), 8),
        "7B-shaped straggler batch: 8 requests x 32 beams, prompts U[256,1024], "
        "lengths lognormal(median 1500, sigma 0.55) capped at 8192, bf16 KV",
    ),
    "7b_longchain_fp8": WorkloadConfig(
        "7b_longchain_fp8",
        AttnShape(28, 4, 128, 16, "bf16", "fp8"),
        _repeat(ReqSpec(beams=32, branch=4, prompt=(2048, 2048), step=(64, 1130), max_len=16384,
                        max_iters=24), 16),
        "7B-shaped long chain: 16 requests x 32 beams, 2048-token prompt, up to 24 steps "
        "U[64,1130], len<=16384, fp8 e4m3 KV with one fp32 scale per block",
    ),
}


# --------------------------------------------------------------------------
# Beam trees over logical block allocations
# --------------------------------------------------------------------------


@dataclass
class BeamTree:
    """Logical beam tree: per-beam allocation lists over a block allocator.

    ``allocs_src[a]``/``allocs_ncopy[a]``: allocation ``a`` is a copy of the
    first ``ncopy`` slots of allocation ``src`` (``-1`` for fresh blocks).
    ``beam_allocs[b]`` lists the allocations of beam ``b`` in logical order.
    """

    block_size: int
    allocs_src: List[int] = field(default_factory=list)
    allocs_ncopy: List[int] = field(default_factory=list)
    beam_allocs: List[List[int]] = field(default_factory=list)
    beam_lens: List[int] = field(default_factory=list)
    beam_parent: List[int] = field(default_factory=list)  # id of the beam it forked from at the last iteration
    req_offsets: List[int] = field(default_factory=lambda: [0])

    def new_alloc(self, src: int = -1, ncopy: int = 0) -> int:
        self.allocs_src.append(src)
        self.allocs_ncopy.append(ncopy)
        return len(self.allocs_src) - 1

    @property
    def num_allocs(self) -> int:
        return len(self.allocs_src)


def _fork(tree: BeamTree, blocks: List[int], length: int) -> List[int]:
    bs = tree.block_size
    nfull = length // bs
    out = list(blocks[:nfull])
    rem = length - nfull * bs
    if rem:
        out.append(tree.new_alloc(blocks[nfull], rem))
    return out


def _append(tree: BeamTree, blocks: List[int], length: int, n: int) -> int:
    bs = tree.block_size
    new_len = length + n
    while len(blocks) * bs < new_len:
        blocks.append(tree.new_alloc())
    return new_len


def _grow_request(tree: BeamTree, rng: np.random.Generator, spec: ReqSpec) -> None:
    bs = tree.block_size
    n, br = spec.beams, spec.branch
    if br < 1 or n % br:
        raise ValueError("beam count must be a multiple of the branch factor")
    p_len = int(rng.integers(spec.prompt[0], spec.prompt[1] + 1))
    prompt_blocks: List[int] = []
    _append(tree, prompt_blocks, 0, p_len)
    if spec.rule == "fixed":
        n_full = max(1, int(round((spec.lognormal_median - p_len) / spec.fixed_div)))
    else:
        n_full = None

    beams: List[Tuple[List[int], int]] = []
    parents: List[int] = []
    it = 0
    lo, hi = spec.step
    if spec.rule == "balanced":
        beams = [(_fork(tree, prompt_blocks, p_len), p_len) for _ in range(br)]
        parents = [-1] * br
        while True:
            steps = rng.integers(lo, hi + 1, size=len(beams))
            beams = [(b, _append(tree, b, ln, int(s))) for (b, ln), s in zip(beams, steps)]
            if len(beams) * br > n:
                break
            kids, kid_parent = [], []
            for i, (b, ln) in enumerate(beams):
                for _ in range(br):
                    kids.append((_fork(tree, b, ln), ln))
                    kid_parent.append(i)
            beams, parents = kids, kid_parent
        for (b, ln), par in zip(beams, parents):
            tot = int(rng.integers(spec.max_len // 2, spec.max_len + 1))
            ln = _append(tree, b, ln, max(1, tot - ln))
            tree.beam_allocs.append(b)
            tree.beam_lens.append(ln)
            tree.beam_parent.append(par)
        tree.req_offsets.append(len(tree.beam_lens))
        return
    while True:
        it += 1
        if it == 1:
            kids = [(_fork(tree, prompt_blocks, p_len), p_len) for _ in range(n)]
            kid_parent = [-1] * n
        else:
            surv = np.sort(rng.choice(n, n // br, replace=False))
            kids = []
            kid_parent = []
            for s in surv:
                for _ in range(br):
                    kids.append((_fork(tree, beams[s][0], beams[s][1]), beams[s][1]))
                    kid_parent.append(int(s))
        cur_max = max(k[1] for k in kids)
        if spec.rule == "fixed":
            final = it > n_full
        else:
            final = it >= spec.max_iters or cur_max + hi > spec.max_len
        steps = rng.integers(lo, hi + 1, size=n)
        new_beams = []
        for (blocks, length), s in zip(kids, steps):
            s = int(s)
            if final and spec.snapshot == "uniform":
                add = int(rng.integers(1, s + 1))
                add = max(1, min(add, spec.max_len - length))
            elif final and spec.snapshot == "lognormal":
                tot = float(rng.lognormal(math.log(spec.lognormal_median), spec.lognormal_sigma))
                tot = int(min(max(round(tot), length + 1), spec.max_len))
                add = tot - length
            else:
                add = s
            new_len = _append(tree, blocks, length, add)
            new_beams.append((blocks, new_len))
        beams = new_beams
        parents = kid_parent
        if final:
            break
    for (blocks, length), par in zip(beams, parents):
        tree.beam_allocs.append(blocks)
        tree.beam_lens.append(length)
        tree.beam_parent.append(par)
    tree.req_offsets.append(len(tree.beam_lens))


def build_tree(cfg: WorkloadConfig, seed: int) -> BeamTree:
    rng = np.random.default_rng([seed, 0x7A5])
    tree = BeamTree(block_size=cfg.shape.block_size)
    for spec in cfg.reqs:
        _grow_request(tree, rng, spec)
    return tree


# --------------------------------------------------------------------------
# Physical placement and KV values
# --------------------------------------------------------------------------


@dataclass
class Workload:
    name: str
    shape: AttnShape
    req_seq_offsets: np.ndarray  # int32 [R+1]
    block_tables: np.ndarray  # int32 [S, max_blocks]
    seq_lens: np.ndarray  # int32 [S]
    num_blocks: int
    q: np.ndarray  # [S, Hq, D] float32 or uint16 (bf16 bits)
    k_cache: np.ndarray  # [NB, Hkv, bs, D]
    v_cache: np.ndarray  # [NB, Hkv, D, bs]
    k_scale: Optional[np.ndarray]  # float32 [NB] for fp8
    v_scale: Optional[np.ndarray]
    seed: int = 0
    poisoned: bool = True

    @property
    def num_seqs(self) -> int:
        return int(self.seq_lens.shape[0])

    @property
    def num_reqs(self) -> int:
        return int(self.req_seq_offsets.shape[0] - 1)

    @property
    def max_blocks_per_seq(self) -> int:
        return int(self.block_tables.shape[1])

    @property
    def max_seq_len(self) -> int:
        return int(self.seq_lens.max()) if self.seq_lens.size else 0

    def kv_elem_bytes(self) -> int:
        return {"f32": 4, "bf16": 2, "fp8": 1}[self.shape.kv_dtype]


def _f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def _f32_to_e4m3_codes(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even E4M3FN encoding with saturation at +-448."""
    import torch

    y = np.clip(np.ascontiguousarray(x, dtype=np.float32), -FP8_MAX, FP8_MAX)
    t = torch.from_numpy(y).to(torch.float8_e4m3fn)
    return t.view(torch.uint8).numpy()


def workload_from_tree(
    shape: AttnShape,
    tree: BeamTree,
    seed: int,
    *,
    name: str = "custom",
    poison: bool = True,
    shuffle: bool = True,
    pool_slack: float = 0.125,
    table_slack: int = 2,
    table_fill: int = -1,
) -> Workload:
    """Place a logical tree in a shuffled physical pool and draw its values.

    * Physical ids: the allocations are mapped through a random permutation
      of a pool ``1 + pool_slack`` times larger than needed.
    * Values: Q, K, V ~ N(0, 1) in fp32, converted to the storage dtype; a
      copy-on-write block repeats the copied slots of its source.
    * ``poison``: every block or slot no beam can see holds NaN (so a kernel
      that touches it fails loudly); otherwise those slots hold finite noise.
    * ``shuffle``: beams within a request are presented in random order,
      as a serving queue would hand them over.
    """
    rng = np.random.default_rng([seed, 0xB10C])
    bs, hkv, d = shape.block_size, shape.num_kv_heads, shape.head_dim

    # Only allocations some final beam references get a physical block (the
    # blocks of pruned beams are free again); copy sources are kept for values.
    referenced = sorted({a for al in tree.beam_allocs for a in al})
    need = set(referenced)
    for a in referenced:
        src = tree.allocs_src[a]
        while src >= 0 and src not in need:
            need.add(src)
            src = tree.allocs_src[src]
    need_list = sorted(need)
    vidx = {a: i for i, a in enumerate(need_list)}
    nref = len(referenced)
    pool = max(1, int(math.ceil(nref * (1.0 + pool_slack))))
    phys_of = dict(zip(referenced, rng.permutation(pool)[:nref].tolist()))

    # Beam order within each request.
    order: List[int] = []
    for r in range(len(tree.req_offsets) - 1):
        idx = np.arange(tree.req_offsets[r], tree.req_offsets[r + 1])
        if shuffle:
            idx = rng.permutation(idx)
        order.extend(int(i) for i in idx)
    s = len(order)
    lens = np.array([tree.beam_lens[i] for i in order], dtype=np.int32)
    nblk = [len(tree.beam_allocs[i]) for i in order]
    maxb = max([1] + nblk) + table_slack
    tables = np.full((s, maxb), table_fill, dtype=np.int32)
    for row, i in enumerate(order):
        al = tree.beam_allocs[i]
        tables[row, : len(al)] = [phys_of[a] for a in al]

    # Valid slots of each referenced allocation = max over referencing beams.
    valid = np.zeros(len(need_list), dtype=np.int64)
    for i in order:
        length = tree.beam_lens[i]
        for j, a in enumerate(tree.beam_allocs[i]):
            v = min(bs, length - j * bs)
            if v > valid[vidx[a]]:
                valid[vidx[a]] = v

    # Values per needed allocation, fp32 [n, hkv, bs, d]; copies repeat their source.
    kv_rng = np.random.default_rng([seed, 0x4B56])
    nv = len(need_list)
    kvals = kv_rng.standard_normal((nv, hkv, bs, d), dtype=np.float32)
    vvals = kv_rng.standard_normal((nv, hkv, bs, d), dtype=np.float32)
    for i, a in enumerate(need_list):
        src, n = tree.allocs_src[a], tree.allocs_ncopy[a]
        if src >= 0 and n > 0:
            kvals[i, :, :n, :] = kvals[vidx[src], :, :n, :]
            vvals[i, :, :n, :] = vvals[vidx[src], :, :n, :]
    sel_rows = np.asarray([vidx[a] for a in referenced], dtype=np.int64)
    kvals, vvals, valid = kvals[sel_rows], vvals[sel_rows], valid[sel_rows]
    phys = np.asarray([phys_of[a] for a in referenced], dtype=np.int64)

    slot_ok = np.arange(bs)[None, :] < valid[:, None]  # [nref, bs]
    dt = shape.kv_dtype
    k_scale = v_scale = None
    if dt == "f32":
        kstore, vstore = kvals, vvals
        if poison:
            kc = np.full((pool, hkv, bs, d), np.nan, dtype=np.float32)
            vc = np.full((pool, hkv, bs, d), np.nan, dtype=np.float32)
        else:
            kc = kv_rng.standard_normal((pool, hkv, bs, d), dtype=np.float32)
            vc = kv_rng.standard_normal((pool, hkv, bs, d), dtype=np.float32)
    elif dt == "bf16":
        kstore, vstore = _f32_to_bf16_bits(kvals), _f32_to_bf16_bits(vvals)
        if poison:
            kc = np.full((pool, hkv, bs, d), BF16_NAN, dtype=np.uint16)
            vc = np.full((pool, hkv, bs, d), BF16_NAN, dtype=np.uint16)
        else:
            kc = _f32_to_bf16_bits(kv_rng.standard_normal((pool, hkv, bs, d), dtype=np.float32))
            vc = _f32_to_bf16_bits(kv_rng.standard_normal((pool, hkv, bs, d), dtype=np.float32))
    elif dt == "fp8":
        # One scale per block and tensor from the amax of its visible entries.
        m = slot_ok[:, None, :, None]
        kamax = np.abs(np.where(m, kvals, 0.0)).reshape(nref, -1).max(axis=1) if nref else np.zeros(0)
        vamax = np.abs(np.where(m, vvals, 0.0)).reshape(nref, -1).max(axis=1) if nref else np.zeros(0)
        ks = np.where(kamax > 0, kamax / FP8_MAX, 1.0).astype(np.float32)
        vsc = np.where(vamax > 0, vamax / FP8_MAX, 1.0).astype(np.float32)
        kstore = _f32_to_e4m3_codes(kvals / ks[:, None, None, None])
        vstore = _f32_to_e4m3_codes(vvals / vsc[:, None, None, None])
        if poison:
            kc = np.full((pool, hkv, bs, d), FP8_NAN, dtype=np.uint8)
            vc = np.full((pool, hkv, bs, d), FP8_NAN, dtype=np.uint8)
            k_scale = np.full(pool, np.nan, dtype=np.float32)
            v_scale = np.full(pool, np.nan, dtype=np.float32)
        else:
            kc = _f32_to_e4m3_codes(kv_rng.standard_normal((pool, hkv, bs, d), dtype=np.float32))
            vc = _f32_to_e4m3_codes(kv_rng.standard_normal((pool, hkv, bs, d), dtype=np.float32))
            k_scale = np.ones(pool, dtype=np.float32)
            v_scale = np.ones(pool, dtype=np.float32)
        k_scale[phys] = ks
        v_scale[phys] = vsc
    else:
        raise ValueError(f"unknown kv dtype {dt}")

    # Scatter visible slots into the pool (token-major staging, V transposed at the end).
    if poison:
        sel = slot_ok[:, None, :, None]
        kc[phys] = np.where(sel, kstore, kc[phys])
        vc[phys] = np.where(sel, vstore, vc[phys])
    else:
        kc[phys] = kstore
        vc[phys] = vstore
    vc = np.ascontiguousarray(np.swapaxes(vc, 2, 3))  # [pool, hkv, d, bs]

    q_rng = np.random.default_rng([seed, 0x51])
    qf = q_rng.standard_normal((s, shape.num_q_heads, d), dtype=np.float32)
    if shape.q_dtype == "bf16":
        q = _f32_to_bf16_bits(qf)
    elif shape.q_dtype == "f32":
        q = qf
    else:
        raise ValueError(f"unknown q dtype {shape.q_dtype}")

    return Workload(
        name=name,
        shape=shape,
        req_seq_offsets=np.asarray(tree.req_offsets, dtype=np.int32),
        block_tables=tables,
        seq_lens=lens,
        num_blocks=pool,
        q=q,
        k_cache=np.ascontiguousarray(kc),
        v_cache=vc,
        k_scale=k_scale,
        v_scale=v_scale,
        seed=seed,
        poisoned=poison,
    )


def make_workload(cfg, seed: int = 0, **kw) -> Workload:
    """Build one of ``CONFIGS`` (by name or object) for ``seed``."""
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    tree = build_tree(cfg, seed)
    return workload_from_tree(cfg.shape, tree, seed, name=cfg.name, **kw)

