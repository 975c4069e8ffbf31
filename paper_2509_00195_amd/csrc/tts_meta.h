// Host-side prefix metadata and kernel work list (pure C++, no HIP).
//
// The beams of each request form a radix tree (trie) of shared thinking
// prefixes (FastTTS Sec. 4.2). Here the trie is built over physical KV block
// ids: a node is a prefix of full blocks, its beam set the beams whose
// full-block path starts with it. Maximal chains of nodes with the same set
// of >= 2 beams are "segments"; each segment's blocks are read once for all
// of its beams. Beams are ordered depth-first with children sorted by their
// smallest original beam index, which groups siblings while the parents keep
// their relative order (Sec. 4.2), and makes each segment's beams a
// contiguous range of positions.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "tts_work.h"

namespace tts {

struct MetaInput {
  int32_t num_reqs = 0;
  const int32_t* req_seq_offsets = nullptr;
  int32_t num_seqs = 0;
  const int32_t* block_tables = nullptr;
  int32_t max_blocks = 0;
  const int32_t* seq_lens = nullptr;
  int32_t block_size = 16;
  int32_t num_blocks = 0;
};

struct HostMeta {
  int32_t num_seqs = 0;
  int32_t block_size = 16;
  int32_t max_blocks = 0;
  // canonical arrays
  std::vector<int32_t> perm;  // position -> original beam
  std::vector<int32_t> seg_req, seg_parent, seg_lblock_begin, seg_nblocks, seg_beam_begin, seg_beam_end;
  std::vector<int32_t> tail_lblock;  // by original beam
  int64_t unique_blocks = 0, unique_tokens = 0;
  // per beam: covering segment of each logical block below tail_lblock (CSR)
  std::vector<int32_t> path_seg_off, path_seg;
  // build-time copies
  std::vector<int32_t> tables, seq_lens;
  std::vector<int32_t> pos_of;  // original beam -> position
  std::vector<int32_t> req_off; // [num_reqs + 1] request offsets (positions of a request are contiguous)
};

// Validates the input and builds the canonical metadata. Returns 0 on
// success or a negative tts_status code with a message in *err.
int build_host_meta(const MetaInput& in, HostMeta* out, std::string* err);

// Coverage rows (beam, lblock, pblock, ntok, src) for the given lengths
// (build-time lengths when seq_lens is null). Returns the number of rows;
// writes at most cap rows.
int64_t coverage_rows(const HostMeta& m, const int32_t* seq_lens, int32_t* rows, int64_t cap);

// Kernel work list for one attention shape (see build_work_plan).
struct WorkPlan {
  std::vector<UnitRec> recs;      // record k < num_bins: workgroup k's first unit
  std::vector<int32_t> slot_off;  // [S + 1] by original beam: CSR into slot_rows
  std::vector<int32_t> slot_rows; // partial row of the beam's row 0 (KV head 0), merge order
  // The same lists as a dense table for the merge kernel: beam b's row
  // holds its slot count, then its slots; slot_stride ints per beam.
  std::vector<int32_t> slot_tab;
  int32_t slot_stride = 0;
  std::vector<int32_t> build_len; // [S] lengths the plan was built for
  int32_t rows_per_head = 0;      // partial rows per KV head
  int32_t num_bins = 0;
  bool two_windows = false;       // some record has a second entry window
  int64_t num_units = 0;          // records with work
  int64_t num_slots = 0;          // slot_rows.size()
  // The planner's choices, for a warm re-plan of the next batch: the target
  // unit cost (us), the modelled work per workgroup it was chosen for, and
  // whether the units were chained (more units than workgroups).
  double target_us = 0, work_us = 0;
  bool chained = false;
  int32_t wide_rows = 0;    // the row caps of the wide and the narrow units
  int32_t narrow_rows = 0;  // the plan chose
};

struct PlanShape {
  int32_t num_q_heads, num_kv_heads, head_dim, kv_bytes;
  int32_t num_bins;  // persistent workgroups (one per compute unit)
};

// warm: a plan of an earlier batch of the same shape (e.g. before a fork);
// when given, its target unit cost, scaled by the change in work, is used
// instead of searching one (the search is most of a plan's host time).
void build_work_plan(const HostMeta& m, const PlanShape& shape, WorkPlan* plan, const WorkPlan* warm = nullptr);

}  // namespace tts
