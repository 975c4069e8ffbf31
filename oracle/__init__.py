"""CPU oracle for prefix-shared beam decode attention -- TEST INFRASTRUCTURE.

This package is the parity reference for the HIP library. It is plain,
slow and written to be checked by eye against its definitions:

* ``attention.oracle_attn`` -- single-query softmax attention per beam and
  query head over the beam's fully materialised key/value sequence, read
  through its block table (the paged KV cache of the paper's serving
  substrate, Sec. 2.3), in fp32; ``attention.oracle_verify_attn`` -- the
  same with each beam's last q_len tokens as causal queries (the verifier
  pass over the current and speculative steps, Sec. 4.1).
* ``prefix_meta.oracle_prefix_meta`` -- the beams of each request arranged
  as a radix tree (trie) of shared full-block prefixes, grouped so that beams
  spawned from the same parent are adjacent while the parents keep their
  relative order (Sec. 4.2, Dynamic Prefix-Aware Scheduling).
* ``fp8.e4m3_table`` -- the 256 OCP E4M3FN code values from the bit formula.
* ``kv_ops`` -- the KV-cache steps around decode: E4M3 encoding by nearest
  table value, appending each beam's token (with the fp8 block-scale rule),
  block copies, the block tables of duplicated beams
  (DuplicateThenTruncate, Sec. 3.1 and Alg. 1) and the lengths the
  duplicates keep after speculation (truncation drawn around the ratio R,
  Sec. 4.1).
* ``schedule`` -- dynamic prefix-aware scheduling (Sec. 4.2): the greedy
  shared-prefix order, budgeted batches and the eviction cost.
* ``kv_alloc`` -- roofline-guided KV allocation (Sec. 4.3): the modelled
  total time of a (prefill batch, decode batch) choice and the search over
  the memory boundary, with a brute force over every pair.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. The product path (the HIP library and
its Python binding) never imports, links or calls it, and the oracle never
imports the product package: the two share no code. Inputs come from the
independent ``tts_synth`` generator.

No part of this oracle is "parity unpinned": every function is checked in
``tests/test_oracle_*.py`` against brute force, closed forms, a library
routine or hand-derived golden fixtures.
"""

from .attention import decode_bf16, oracle_attn, oracle_attn_row, oracle_verify_attn  # noqa: F401
from .fp8 import e4m3_table  # noqa: F401
from .kv_ops import append_kv, copy_blocks, e4m3_encode, fork_tables, truncated_lengths  # noqa: F401
from .prefix_meta import oracle_coverage, oracle_prefix_meta  # noqa: F401
