// Work-unit records and kernel parameters shared by the host planner and
// the HIP kernels. Plain C++ (no HIP types) so the planner builds with any
// host compiler.
#pragma once

#include <cstdint>

namespace tts {

// One workgroup handles at most this many query rows of one KV head
// (4 row tiles of 16); a row is one (beam, query head of the KV group).
constexpr int kMaxRows = 64;
// Block entries per window (one per lane of a wave). A unit has two
// windows: the first holds its LIVE and extension entries, the second up to
// kMaxEntries more static entries.
constexpr int kMaxEntries = 64;
constexpr int kMaxUnitEntries = 2 * kMaxEntries;
// Beams per unit.
constexpr int kMaxUnitBeams = 16;

// Entry info word: rows [r0, r1) of the unit that attend to the block, and
// its valid token count (static; see the flags). Wide units' blocks apply
// to all of their rows and are full; their info words are not read.
//   bits  0..5   r0
//   bits  6..11  r1 - 1
//   bits 12..15  valid - 1
//   bit  16      kEntLive: the beam's partially filled last block at build
//                time; valid grows with the beam's live length
//   bit  17      kEntExt: not a block; the beam (id = its slot in the unit)
//                may have grown past its build-time blocks, which are then
//                read from the live block table
constexpr uint32_t kEntLive = 1u << 16;
constexpr uint32_t kEntExt = 1u << 17;

inline constexpr uint32_t ent_info(int r0, int r1, int valid, uint32_t flags) {
  return static_cast<uint32_t>(r0) | (static_cast<uint32_t>(r1 - 1) << 6) |
         (static_cast<uint32_t>(valid - 1) << 12) | flags;
}

// Wide units (kModeWide): up to kMaxWideRows rows of one segment piece;
// each of the 4 waves owns a quarter of the row tiles (at most 3) and
// every block applies to every row.
constexpr int kMaxWideRows = 192;
constexpr int kMaxWideBeams = 64;
enum UnitMode : int32_t { kModeNarrow = 0, kModeWide = 1 };

// One unit of work: query rows of up to kMaxUnitBeams beams (kMaxWideBeams
// for a wide unit), consecutive in the canonical order, for one KV head,
// against a list of KV blocks, each applying to a contiguous range of those
// rows. Rows are beam-major: row r belongs to the unit's beam r / g and
// query head kvh * g + r % g. The unit writes one partial softmax state per
// row to partial row kvh * rows_per_head + prow0 + r.
struct UnitRec {
  int32_t kvh;
  int32_t nrows;     // 0: nothing to do (an idle workgroup)
  int32_t nstatic;   // first window: block entries (pairs are entries 2i, 2i+1)
  int32_t nent;      // first window: block entries + extension entries (these come last)
  int32_t prow0;
  int32_t next;      // next record of the same workgroup, -1 at the end
  int32_t mode;      // UnitMode
  int32_t nstatic2;  // second window: block entries (no LIVE or extension entries)
  int32_t beams[kMaxWideBeams];  // original beam index of each unit beam
  int32_t ent_id[kMaxEntries];   // physical block id (extension: beam slot)
  uint32_t ent_info[kMaxEntries];
  int32_t ent_id2[kMaxEntries];  // second window
  uint32_t ent_info2[kMaxEntries];
};
static_assert(sizeof(UnitRec) == 32 + 4 * kMaxWideBeams + 16 * kMaxEntries, "UnitRec layout");

// Partial softmax state of one query row over a subset of its tokens:
// the reference maximum m (log2 units), the sum l of 2^(score - m), the
// row's elements and their factor z, with element x z = o / l (the
// normalised value average). For bf16 and fp8 caches the elements are o
// divided by a power of two 2^e chosen so that every element lies in
// [-1, 1], in fp16 (2 bytes per element instead of 4; scaled so, the
// elements keep fp16's full relative precision and never overflow), and
// z = 2^e / l; for fp32 caches they are o / l in fp32 and z = 1. The D
// elements of a row are stored in lane order: element 32 q + 4 t + j (for
// D = 128; generally (D / 4) q + 4 t + j) holds dimension 16 t + 4 q + j,
// the order in which the attention kernel's lanes hold the row.
constexpr int kPartMl = 4;  // floats per row of part_ml: m, l, z, 0

struct AttnParams {
  const void* q;
  const void* k_cache;
  const void* v_cache;
  const float* k_scale;
  const float* v_scale;
  const int32_t* block_tables;
  const int32_t* seq_lens;
  float* out;
  void* part_o;    // [rows][D] fp16 (fp32 for fp32 caches), lane order
  float* part_ml;  // [rows][kPartMl]: m, l, z, 0
  // prefix path (null recs: paged path)
  const UnitRec* recs;
  const int32_t* build_len;  // [S] lengths the metadata was built for
  int32_t rows_per_head;     // partial rows of one KV head
  int32_t max_blocks;
  int32_t num_blocks;
  int32_t num_seqs;
  int32_t hq;
  int32_t hkv;
  int32_t g;
  float scale_log2;      // softmax scale * log2(e)
  int32_t paged_nsplit;  // paged path: splits per beam (1: write the output directly)
  int32_t paged_max_len;
  // Verification: every beam's last q_len tokens are queries, each a
  // virtual beam vb = b * q_len + i over beam b's table with length
  // seq_lens[b] - (q_len - 1 - i) (causal). 1 for decode.
  int32_t q_len;
  // Some unit of the plan has a second entry window: selects the kernel
  // build that reads them (the other keeps the pair loop's registers).
  int32_t two_windows;
};

// Slots the merge kernel reads per round trip (and the smallest slot-table
// stride - 1, so that a beam's first round of slots is always in its row).
constexpr int kMergeBatch = 16;
// Readable int32 words after the start of any slot-table row (the table is
// followed by this many zeros): the merges read a row's first entries in
// the same round trip as its count, without waiting for the count.
constexpr int kSlotTabReadAhead = 65;

struct MergeParams {
  const void* part_o;
  const float* part_ml;
  // [S][slot_stride]: slot count, then the partial row of the beam's row 0
  // (KV head 0) for each slot in merge order; null for the paged path
  const int32_t* slot_tab;
  int32_t slot_stride;
  int32_t pad0;
  const int32_t* seq_lens;
  const int32_t* build_len;  // prefix path: stale-metadata check (else null)
  float* out;
  int32_t num_seqs;
  int32_t hq;
  int32_t g;
  int32_t rows_per_head;
  int32_t paged_nsplit;
  int32_t q_len;  // as in AttnParams (lengths of virtual beams)
};

}  // namespace tts
