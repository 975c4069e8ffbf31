// Work-unit and kernel-parameter layouts shared by the host planner and the
// HIP kernels. Plain C++ (no HIP types) so the planner builds with any
// host compiler.
#pragma once

#include <cstdint>

namespace tts {

// Rows of one KV head handled by one workgroup: 4 waves x 16 rows, cut at
// whole beams (a unit covers floor(64 / g) beams).
constexpr int kRowsPerUnit = 64;
constexpr int kUnitInts = 12;

enum UnitKind : int32_t { kSegmentPiece = 0, kTailSplit = 1 };

// One workgroup's share of the decode step: query rows of one KV head
// against one contiguous run of KV blocks.
//
// Rows: the beams at positions [pos0, pos0 + nbeams) of the canonical order
// each contribute g = Hq/Hkv rows (beam-major, then query head); the unit
// owns rows [row0, row0 + nrows) of those nbeams * g.
// Blocks: a segment piece reads seg_blocks[blk_off .. blk_off + nblk), all
// full; a tail split reads split blk_off of nblk equal parts of the beam's
// private blocks [tail_lblock, ceil(seq_len / block_size)), from the live
// block table (last block possibly partial).
// Output: a partial softmax state written to slot `slot` of every covered
// beam (slot order = merge order). A unit with nrows == 0 is padding.
struct Unit {
  int32_t kvh;
  int32_t kind;
  int32_t pos0;
  int32_t nbeams;
  int32_t row0;
  int32_t nrows;
  int32_t blk_off;
  int32_t nblk;
  int32_t slot;
  int32_t pad0, pad1, pad2;
};
static_assert(sizeof(Unit) == kUnitInts * 4, "Unit layout");

struct AttnParams {
  const void* q;
  const void* k_cache;
  const void* v_cache;
  const float* k_scale;
  const float* v_scale;
  const int32_t* block_tables;
  const int32_t* seq_lens;
  float* out;
  float* part_o;   // [slots][Hq][D]
  float* part_ml;  // [slots][Hq][2]: running max (log2 units), sum
  // prefix path (null for the paged path)
  const int32_t* perm;
  const int32_t* tail_lblock;
  const int32_t* slot_base;
  const int32_t* seg_blocks;
  const Unit* units;
  int32_t max_blocks;
  int32_t num_blocks;
  int32_t num_seqs;
  int32_t hq;
  int32_t hkv;
  int32_t g;
  float scale_log2;     // softmax scale * log2(e)
  int32_t paged_nsplit; // paged path: splits per beam (1: write the output directly)
  int32_t paged_max_len;
  int32_t pad;
};


struct MergeParams {
  const float* part_o;
  const float* part_ml;
  const int32_t* slot_base;    // [S + 1]; null for the paged path
  const int32_t* seq_lens;
  const int32_t* tail_lblock;  // prefix path: stale-metadata check (else null)
  float* out;
  int32_t num_seqs;
  int32_t hq;
  int32_t paged_nsplit;
  int32_t pad;
};

}  // namespace tts
