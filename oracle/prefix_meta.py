"""Oracle prefix metadata: the beams' radix tree of shared KV blocks.

Definition (written from Sec. 4.2, Dynamic Prefix-Aware Scheduling: the
beams of one TTS request form a radix tree (trie) whose nodes are shared
thinking prefixes; beams spawned from the same parent are grouped while the
parents keep their relative order):

* Per request ``r`` (beams ``req_seq_offsets[r] .. req_seq_offsets[r+1]``),
  build a trie over each beam's sequence of *full* physical block ids,
  ``block_tables[b][0 : seq_lens[b] // bs]``. A node at depth ``k`` stands
  for one block-id prefix of length ``k``; its beam set is every beam whose
  full-block path starts with that prefix. Requests never share nodes, and a
  partially filled last block is never shared.
* Ordering: at every node the children and the beams whose full-block path
  ends there are visited in increasing order of the smallest original beam
  index they contain. ``perm`` lists the beams in that depth-first order
  (requests concatenated), so every node's beam set is a contiguous range of
  positions.
* Segments: nodes with at least two beams, merged into maximal parent-child
  chains with the same beam set. Each segment records its request, parent
  segment (-1 when it starts at depth 0), first logical block, block count
  and its beam range in ``perm`` positions; segments are listed in
  depth-first preorder.
* ``tail_lblock[b]``: depth of the deepest node with >= 2 beams on beam
  ``b``'s path (its private tail starts at that logical block).
* ``unique_blocks``: distinct physical ids among all (beam, logical block)
  pairs in use (``lblock < ceil(L / bs)``); ``unique_tokens``: the sum over
  those ids of the largest valid token count any beam sees in them.

This module is independent of the C++ builder; the two must agree
bit-for-bit.
"""

from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np


class _Node:
    __slots__ = ("depth", "children", "beams", "ending", "seg")

    def __init__(self, depth: int):
        self.depth = depth
        self.children: Dict[int, "_Node"] = {}
        self.beams: List[int] = []  # original indices, ascending (insertion order)
        self.ending: List[int] = []
        self.seg = -1


def _build_trie(beams: List[int], block_tables: np.ndarray, seq_lens: np.ndarray, bs: int) -> _Node:
    root = _Node(0)
    for b in beams:
        node = root
        node.beams.append(b)
        nfull = int(seq_lens[b]) // bs
        for j in range(nfull):
            pid = int(block_tables[b, j])
            child = node.children.get(pid)
            if child is None:
                child = _Node(node.depth + 1)
                node.children[pid] = child
            child.beams.append(b)
            node = child
        node.ending.append(b)
    return root


def oracle_prefix_meta(
    req_seq_offsets: np.ndarray,
    block_tables: np.ndarray,
    seq_lens: np.ndarray,
    block_size: int,
) -> dict:
    """Canonical prefix metadata as a dict of numpy int32 arrays / ints."""
    offs = [int(x) for x in req_seq_offsets]
    s_all = int(seq_lens.shape[0])
    perm: List[int] = []
    seg_req: List[int] = []
    seg_parent: List[int] = []
    seg_lb: List[int] = []
    seg_nb: List[int] = []
    seg_bb: List[int] = []
    seg_be: List[int] = []
    tail = [0] * s_all
    node_seg_paths: Dict[int, List[int]] = {}

    for r in range(len(offs) - 1):
        beams = list(range(offs[r], offs[r + 1]))
        root = _build_trie(beams, block_tables, seq_lens, block_size)
        # Depth-first walk with an explicit stack (paths can be 1000s of blocks deep).
        # A stack entry is (node, parent_node) for a subtree or ("beam", b).
        stack: list = [(root, None)]
        while stack:
            item = stack.pop()
            if item[0] == "beam":
                perm.append(item[1])
                continue
            node, parent = item
            if node is not root and len(node.beams) >= 2:
                if parent is not root and len(parent.beams) == len(node.beams):
                    node.seg = parent.seg
                    seg_nb[node.seg] += 1
                else:
                    node.seg = len(seg_req)
                    seg_req.append(r)
                    seg_parent.append(parent.seg if parent is not root else -1)
                    seg_lb.append(node.depth - 1)
                    seg_nb.append(1)
                    seg_bb.append(len(perm))
                    seg_be.append(len(perm) + len(node.beams))
            items = [(c.beams[0], 0, c) for c in node.children.values()]
            items += [(b, 1, b) for b in node.ending]
            items.sort(key=lambda t: t[0])
            for key, kind, obj in reversed(items):
                stack.append(("beam", obj) if kind == 1 else (obj, node))
        # Tails and per-block segment ids along each beam's path.
        for b in beams:
            node = root
            segs: List[int] = []
            nfull = int(seq_lens[b]) // block_size
            for j in range(nfull):
                node = node.children[int(block_tables[b, j])]
                if len(node.beams) < 2:
                    break
                segs.append(node.seg)
            tail[b] = len(segs)
            node_seg_paths[b] = segs

    # Unique physical blocks / tokens over every (beam, logical block) in use.
    best: Dict[int, int] = {}
    for b in range(s_all):
        length = int(seq_lens[b])
        nblk = -(-length // block_size)
        for j in range(nblk):
            pid = int(block_tables[b, j])
            v = min(block_size, length - j * block_size)
            if v > best.get(pid, 0):
                best[pid] = v

    i32 = lambda x: np.asarray(x, dtype=np.int32)  # noqa: E731
    return {
        "num_seqs": s_all,
        "num_segs": len(seg_req),
        "perm": i32(perm),
        "seg_req": i32(seg_req),
        "seg_parent": i32(seg_parent),
        "seg_lblock_begin": i32(seg_lb),
        "seg_nblocks": i32(seg_nb),
        "seg_beam_begin": i32(seg_bb),
        "seg_beam_end": i32(seg_be),
        "tail_lblock": i32(tail),
        "unique_blocks": len(best),
        "unique_tokens": int(sum(best.values())),
        "_block_seg": node_seg_paths,
    }


def oracle_coverage(meta: dict, block_tables: np.ndarray, seq_lens: np.ndarray, block_size: int,
                    seq_lens_now: Optional[np.ndarray] = None) -> np.ndarray:
    """Rows ``(beam, lblock, pblock, ntok, src)`` covering every used block once.

    Beams in original order; each beam's logical blocks in order, which is
    also the merge order (segments root to leaf, then the tail). ``src`` is
    the covering segment id, or -1 for tail blocks. ``seq_lens_now`` may be
    larger than the lengths the metadata was built from (private appends).
    """
    lens = seq_lens if seq_lens_now is None else seq_lens_now
    rows = []
    for b in range(int(lens.shape[0])):
        length = int(lens[b])
        segs = meta["_block_seg"][b]
        for j in range(-(-length // block_size)):
            src = segs[j] if j < len(segs) else -1
            rows.append((b, j, int(block_tables[b, j]), min(block_size, length - j * block_size), src))
    return np.asarray(rows, dtype=np.int32).reshape(-1, 5)
