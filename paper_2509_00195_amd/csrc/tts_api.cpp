// C ABI of libtts (include/tts.h): argument validation, metadata handles
// and kernel launches.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "tts.h"
#include "tts_meta.h"
#include "tts_work.h"

namespace tts {
hipError_t launch_attn(const AttnParams& p, int grid, int head_dim, int kv_kind, hipStream_t stream);
hipError_t launch_merge(const MergeParams& p, int head_dim, int kv_kind, hipStream_t stream);
hipError_t scratch_buffer(void** ptr, size_t* bytes);
hipError_t launch_append(const void* k_new, const void* v_new, const int32_t* block_tables, const int32_t* seq_lens,
                         void* k_cache, void* v_cache, float* k_scale, float* v_scale, int num_seqs, int max_blocks,
                         int num_blocks, int hkv, int head_dim, int kv_kind, hipStream_t stream);
void alloc_time(const tts_alloc_problem& pr, int64_t b_pre, int64_t b_dec, tts_alloc_result* out);
struct SchedInput {
  int32_t num_cots;
  const int32_t* cot_off;
  const int32_t* cot_nodes;
  const int64_t* weight;
  int64_t budget;
};
struct SchedOutput {
  std::vector<int32_t> order, batch_off;
  int64_t score = 0, cost = 0;
};
void prefix_schedule(const SchedInput& in, SchedOutput* out);
bool alloc_search(const tts_alloc_problem& pr, tts_alloc_result* out);
hipError_t launch_copy_blocks(const int32_t* pairs, int num_pairs, void* k_cache, void* v_cache, float* k_scale,
                              float* v_scale, int64_t blk_bytes, int num_blocks, hipStream_t stream);
}  // namespace tts

namespace tts {
// A product the compiler may not fuse with a following addition (an FMA
// would round once where the oracle rounds twice).
double mul_unfused(double a, double b) {
  volatile double r = a * b;
  return r;
}
}  // namespace tts

namespace {

thread_local std::string g_last_error;

tts_status fail(tts_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

tts_status ok() {
  g_last_error.clear();
  return TTS_OK;
}

// Paged path: blocks per split of a long sequence.
constexpr int32_t kPagedSplitBlocks = 32;

tts_status check_desc(const tts_attn_desc* d) {
  if (!d) return fail(TTS_ERR_INVALID_ARG, "desc is NULL");
  if (d->num_q_heads <= 0 || d->num_kv_heads <= 0 || d->num_q_heads % d->num_kv_heads != 0)
    return fail(TTS_ERR_INVALID_ARG, "num_q_heads must be a positive multiple of num_kv_heads");
  if (d->num_q_heads / d->num_kv_heads > tts::kMaxRows)
    return fail(TTS_ERR_UNSUPPORTED, "more than 64 query heads per KV head");
  if (d->head_dim != 64 && d->head_dim != 128) return fail(TTS_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (d->block_size != 16) return fail(TTS_ERR_UNSUPPORTED, "block_size must be 16");
  const bool f32 = d->q_dtype == TTS_F32 && d->kv_dtype == TTS_F32;
  const bool bf = d->q_dtype == TTS_BF16 && (d->kv_dtype == TTS_BF16 || d->kv_dtype == TTS_FP8_E4M3);
  if (!f32 && !bf) return fail(TTS_ERR_UNSUPPORTED, "unsupported (q_dtype, kv_dtype) combination");
  if (d->out_dtype != TTS_F32) return fail(TTS_ERR_UNSUPPORTED, "out_dtype must be F32");
  if (!std::isfinite(d->scale)) return fail(TTS_ERR_INVALID_ARG, "scale is not finite");
  return TTS_OK;
}

int kv_kind(const tts_attn_desc* d) { return d->kv_dtype == TTS_F32 ? 0 : (d->kv_dtype == TTS_BF16 ? 1 : 2); }
int kv_bytes(const tts_attn_desc* d) { return d->kv_dtype == TTS_F32 ? 4 : (d->kv_dtype == TTS_BF16 ? 2 : 1); }

float scale_log2(const tts_attn_desc* d) {
  const double s = d->scale > 0.f ? d->scale : 1.0 / std::sqrt(static_cast<double>(d->head_dim));
  return static_cast<float>(s * 1.4426950408889634);
}

tts_status check_scales(const tts_attn_desc* d, const float* ks, const float* vs) {
  if (d->kv_dtype == TTS_FP8_E4M3) {
    if (!ks || !vs) return fail(TTS_ERR_INVALID_ARG, "fp8 KV needs k_scale and v_scale");
  } else if (ks || vs) {
    return fail(TTS_ERR_INVALID_ARG, "k_scale/v_scale must be NULL unless kv_dtype is FP8_E4M3");
  }
  return TTS_OK;
}

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

// Partial-state elements: fp16 for bf16 and fp8 caches, fp32 for fp32 caches.
size_t part_o_bytes(const tts_attn_desc* d, size_t rows) {
  return align256(rows * d->head_dim * (d->kv_dtype == TTS_F32 ? 4 : 2));
}

}  // namespace

struct tts_prefix_meta {
  tts::HostMeta host;
  bool has_plan = false;
  tts_attn_desc desc{};
  tts::WorkPlan plan;
  int32_t num_blocks = 0;
  int32_t q_len = 1;  // > 1: a verification metadata (q_len virtual beams per beam)
  // device buffer: unit records | slot table | build_len
  void* dev = nullptr;
  size_t off_recs = 0, off_slot_tab = 0, off_build = 0;
};

extern "C" {

const char* tts_last_error(void) { return g_last_error.c_str(); }

static tts_status build_meta_impl(int32_t num_reqs, const int32_t* req_seq_offsets, int32_t num_seqs,
                                  const int32_t* block_tables, int32_t max_blocks_per_seq, const int32_t* seq_lens,
                                  int32_t block_size, int32_t num_blocks, const tts_attn_desc* desc,
                                  hipStream_t stream, int32_t q_len, tts_prefix_meta** out,
                                  const tts::WorkPlan* warm = nullptr) {
  if (!out) return fail(TTS_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (desc) {
    tts_status s = check_desc(desc);
    if (s != TTS_OK) return s;
    if (desc->block_size != block_size) return fail(TTS_ERR_INVALID_ARG, "desc->block_size != block_size");
  }
  tts_prefix_meta* m = new (std::nothrow) tts_prefix_meta();
  if (!m) return fail(TTS_ERR_NOMEM, "out of host memory");
  tts::MetaInput in;
  in.num_reqs = num_reqs;
  in.req_seq_offsets = req_seq_offsets;
  in.num_seqs = num_seqs;
  in.block_tables = block_tables;
  in.max_blocks = max_blocks_per_seq;
  in.seq_lens = seq_lens;
  in.block_size = block_size;
  in.num_blocks = num_blocks;
  std::string err;
  int rc;
  try {
    rc = tts::build_host_meta(in, &m->host, &err);
  } catch (const std::bad_alloc&) {
    delete m;
    return fail(TTS_ERR_NOMEM, "out of host memory");
  }
  if (rc != 0) {
    delete m;
    return fail(static_cast<tts_status>(rc), err);
  }
  m->num_blocks = num_blocks;
  m->q_len = q_len;
  if (desc) {
    m->has_plan = true;
    m->desc = *desc;
    int dev_id = 0, ncu = 0;
    if (hipGetDevice(&dev_id) != hipSuccess ||
        hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev_id) != hipSuccess || ncu <= 0) {
      delete m;
      return fail(TTS_ERR_HIP, "cannot query the device's compute-unit count");
    }
    try {
      tts::build_work_plan(m->host, {desc->num_q_heads, desc->num_kv_heads, desc->head_dim, kv_bytes(desc), ncu},
                           &m->plan, warm);
    } catch (const std::bad_alloc&) {
      delete m;
      return fail(TTS_ERR_NOMEM, "out of host memory");
    }
    const size_t S = static_cast<size_t>(num_seqs);
    const auto& pl = m->plan;
    m->off_recs = 0;
    m->off_slot_tab = align256(m->off_recs + pl.recs.size() * sizeof(tts::UnitRec));
    m->off_build = align256(m->off_slot_tab + (pl.slot_tab.size() + tts::kSlotTabReadAhead) * 4);
    const size_t total = align256(m->off_build + S * 4);
    std::vector<unsigned char> img(total, 0);
    std::memcpy(img.data() + m->off_recs, pl.recs.data(), pl.recs.size() * sizeof(tts::UnitRec));
    if (!pl.slot_tab.empty()) std::memcpy(img.data() + m->off_slot_tab, pl.slot_tab.data(), pl.slot_tab.size() * 4);
    if (S) std::memcpy(img.data() + m->off_build, pl.build_len.data(), S * 4);
    hipError_t e = hipMalloc(&m->dev, total);
    if (e != hipSuccess) {
      m->dev = nullptr;
      delete m;
      return fail(e == hipErrorOutOfMemory ? TTS_ERR_NOMEM : TTS_ERR_HIP,
                  std::string("hipMalloc: ") + hipGetErrorString(e));
    }
    e = hipMemcpyAsync(m->dev, img.data(), total, hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);  // img is a temporary host buffer
    if (e != hipSuccess) {
      hipFree(m->dev);
      delete m;
      return fail(TTS_ERR_HIP, std::string("upload: ") + hipGetErrorString(e));
    }
  }
  *out = m;
  return ok();
}

tts_status tts_build_prefix_meta(int32_t num_reqs, const int32_t* req_seq_offsets, int32_t num_seqs,
                                 const int32_t* block_tables, int32_t max_blocks_per_seq, const int32_t* seq_lens,
                                 int32_t block_size, int32_t num_blocks, const tts_attn_desc* desc,
                                 hipStream_t stream, tts_prefix_meta** out) {
  return build_meta_impl(num_reqs, req_seq_offsets, num_seqs, block_tables, max_blocks_per_seq, seq_lens, block_size,
                         num_blocks, desc, stream, 1, out);
}

tts_status tts_build_verify_meta(int32_t num_reqs, const int32_t* req_seq_offsets, int32_t num_seqs,
                                 const int32_t* block_tables, int32_t max_blocks_per_seq, const int32_t* seq_lens,
                                 int32_t q_len, int32_t block_size, int32_t num_blocks, const tts_attn_desc* desc,
                                 hipStream_t stream, tts_prefix_meta** out) {
  if (!out) return fail(TTS_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (q_len < 1) return fail(TTS_ERR_INVALID_ARG, "q_len must be >= 1");
  if (num_reqs < 0 || num_seqs < 0 || max_blocks_per_seq < 0) return fail(TTS_ERR_INVALID_ARG, "negative size");
  if ((num_seqs > 0 && (!seq_lens || !block_tables)) || !req_seq_offsets)
    return fail(TTS_ERR_INVALID_ARG, "NULL host array");
  const int64_t vs = static_cast<int64_t>(num_seqs) * q_len;
  if (vs > 0x7FFFFFFF / 2) return fail(TTS_ERR_UNSUPPORTED, "too many query rows");
  for (int32_t b = 0; b < num_seqs; ++b)
    if (seq_lens[b] < q_len) return fail(TTS_ERR_INVALID_ARG, "a beam is shorter than q_len");
  // Virtual beams b * q_len + i: beam b's table, its first len - (q_len - 1 - i) tokens.
  std::vector<int32_t> voff(num_reqs + 1), vlen(vs), vtab(static_cast<size_t>(vs) * max_blocks_per_seq);
  for (int32_t r = 0; r <= num_reqs; ++r) voff[r] = req_seq_offsets[r] * q_len;
  for (int32_t b = 0; b < num_seqs; ++b)
    for (int32_t i = 0; i < q_len; ++i) {
      const int64_t v = static_cast<int64_t>(b) * q_len + i;
      vlen[v] = seq_lens[b] - (q_len - 1 - i);
      std::memcpy(vtab.data() + v * max_blocks_per_seq, block_tables + static_cast<int64_t>(b) * max_blocks_per_seq,
                  sizeof(int32_t) * max_blocks_per_seq);
    }
  return build_meta_impl(num_reqs, voff.data(), static_cast<int32_t>(vs), vtab.data(), max_blocks_per_seq,
                         vlen.data(), block_size, num_blocks, desc, stream, q_len, out);
}

tts_status tts_fork_prefix_meta(const tts_prefix_meta* prev, int32_t num_reqs, const int32_t* req_seq_offsets,
                                int32_t num_seqs, const int32_t* block_tables, int32_t max_blocks_per_seq,
                                const int32_t* seq_lens, int32_t block_size, int32_t num_blocks, hipStream_t stream,
                                tts_prefix_meta** out) {
  if (out) *out = nullptr;
  if (!prev) return fail(TTS_ERR_INVALID_ARG, "prev is NULL");
  if (!prev->has_plan) return fail(TTS_ERR_INVALID_ARG, "prev was built without a desc");
  if (prev->q_len != 1) return fail(TTS_ERR_INVALID_ARG, "prev is a verification metadata");
  return build_meta_impl(num_reqs, req_seq_offsets, num_seqs, block_tables, max_blocks_per_seq, seq_lens, block_size,
                         num_blocks, &prev->desc, stream, 1, out, &prev->plan);
}

tts_status tts_truncated_lengths(int32_t num_children, const int32_t* child_parent, const int32_t* parent_lens,
                                 const int32_t* parent_spec, int32_t num_parents, double ratio, double sigma,
                                 const double* z, int32_t* child_lens) {
  if (num_children < 0 || num_parents < 0) return fail(TTS_ERR_INVALID_ARG, "negative count");
  if (num_children > 0 && (!child_parent || !z || !child_lens || !parent_lens || !parent_spec))
    return fail(TTS_ERR_INVALID_ARG, "NULL host array");
  if (!std::isfinite(ratio) || !std::isfinite(sigma) || sigma < 0)
    return fail(TTS_ERR_INVALID_ARG, "ratio must be finite and sigma finite and >= 0");
  for (int32_t c = 0; c < num_children; ++c) {
    const int32_t p = child_parent[c];
    if (p < 0 || p >= num_parents) return fail(TTS_ERR_OUT_OF_RANGE, "child_parent out of range");
    if (parent_spec[p] < 0 || parent_spec[p] > parent_lens[p])
      return fail(TTS_ERR_INVALID_ARG, "parent_spec must lie in [0, parent length]");
    if (!std::isfinite(z[c])) return fail(TTS_ERR_INVALID_ARG, "z is not finite");
  }
  std::vector<char> seen(static_cast<size_t>(num_parents), 0);
  for (int32_t c = 0; c < num_children; ++c) {
    const int32_t p = child_parent[c];
    if (!seen[p]) {  // the original keeps every token
      seen[p] = 1;
      child_lens[c] = parent_lens[p];
      continue;
    }
    // A duplicate keeps the fraction clip(ratio + sigma z, 0, 1) of its
    // parent's speculative tokens, rounded half up (two roundings: the
    // product, then the sum, never fused, as the oracle computes it).
    const double dz = tts::mul_unfused(sigma, z[c]);
    double f = ratio + dz;
    f = f < 0.0 ? 0.0 : (f > 1.0 ? 1.0 : f);
    const int32_t spec = parent_spec[p];
    const int32_t kept = static_cast<int32_t>(std::floor(tts::mul_unfused(f, static_cast<double>(spec)) + 0.5));
    child_lens[c] = parent_lens[p] - spec + (kept > spec ? spec : kept);
  }
  return ok();
}

void tts_prefix_meta_destroy(tts_prefix_meta* m) {
  if (!m) return;
  if (m->dev) hipFree(m->dev);
  delete m;
}

tts_status tts_prefix_meta_export(const tts_prefix_meta* m, tts_prefix_meta_view* v) {
  if (!m || !v) return fail(TTS_ERR_INVALID_ARG, "NULL argument");
  const auto& h = m->host;
  v->num_seqs = h.num_seqs;
  v->num_segs = static_cast<int32_t>(h.seg_req.size());
  v->perm = h.perm.data();
  v->seg_req = h.seg_req.data();
  v->seg_parent = h.seg_parent.data();
  v->seg_lblock_begin = h.seg_lblock_begin.data();
  v->seg_nblocks = h.seg_nblocks.data();
  v->seg_beam_begin = h.seg_beam_begin.data();
  v->seg_beam_end = h.seg_beam_end.data();
  v->tail_lblock = h.tail_lblock.data();
  v->unique_blocks = h.unique_blocks;
  v->unique_tokens = h.unique_tokens;
  return ok();
}

tts_status tts_prefix_meta_coverage(const tts_prefix_meta* m, const int32_t* seq_lens_host, int32_t* out_rows,
                                    int64_t cap, int64_t* n_rows) {
  if (!m || !n_rows) return fail(TTS_ERR_INVALID_ARG, "NULL argument");
  if (cap < 0 || (cap > 0 && !out_rows)) return fail(TTS_ERR_INVALID_ARG, "bad out_rows/cap");
  if (seq_lens_host) {
    for (int32_t b = 0; b < m->host.num_seqs; ++b) {
      if (seq_lens_host[b] < 0 || static_cast<int64_t>(seq_lens_host[b]) >
                                      static_cast<int64_t>(m->host.max_blocks) * m->host.block_size)
        return fail(TTS_ERR_INVALID_ARG, "seq_lens_host entry outside [0, max_blocks * block_size]");
    }
  }
  *n_rows = tts::coverage_rows(m->host, seq_lens_host, out_rows, cap);
  if (*n_rows > cap) return fail(TTS_ERR_WORKSPACE, "cap too small for the coverage rows");
  return ok();
}

tts_status tts_plan_units_host(int32_t num_reqs, const int32_t* req_seq_offsets, int32_t num_seqs,
                               const int32_t* block_tables, int32_t max_blocks_per_seq, const int32_t* seq_lens,
                               int32_t block_size, int32_t num_blocks, const tts_attn_desc* desc,
                               int32_t num_workgroups, int32_t* out_rows, int64_t cap, int64_t* n_rows,
                               int64_t* num_units) {
  if (!desc || !n_rows || !num_units) return fail(TTS_ERR_INVALID_ARG, "NULL argument");
  if (num_workgroups < 1) return fail(TTS_ERR_INVALID_ARG, "num_workgroups must be >= 1");
  if (cap < 0 || (cap > 0 && !out_rows)) return fail(TTS_ERR_INVALID_ARG, "bad out_rows/cap");
  tts_status s = check_desc(desc);
  if (s != TTS_OK) return s;
  if (desc->block_size != block_size) return fail(TTS_ERR_INVALID_ARG, "desc->block_size != block_size");
  tts::MetaInput in;
  in.num_reqs = num_reqs;
  in.req_seq_offsets = req_seq_offsets;
  in.num_seqs = num_seqs;
  in.block_tables = block_tables;
  in.max_blocks = max_blocks_per_seq;
  in.seq_lens = seq_lens;
  in.block_size = block_size;
  in.num_blocks = num_blocks;
  tts::HostMeta host;
  tts::WorkPlan plan;
  std::string err;
  try {
    const int rc = tts::build_host_meta(in, &host, &err);
    if (rc != 0) return fail(static_cast<tts_status>(rc), err);
    tts::build_work_plan(host, {desc->num_q_heads, desc->num_kv_heads, desc->head_dim, kv_bytes(desc), num_workgroups},
                         &plan);
  } catch (const std::bad_alloc&) {
    return fail(TTS_ERR_NOMEM, "out of host memory");
  }
  const int32_t g = desc->num_q_heads / desc->num_kv_heads;
  int64_t n = 0, units = 0;
  auto emit = [&](int32_t unit, int32_t entry, int32_t kvh, int32_t beam, int32_t block, int32_t valid, int32_t flags) {
    if (n < cap) {
      int32_t* r = out_rows + 7 * n;
      r[0] = unit, r[1] = entry, r[2] = kvh, r[3] = beam, r[4] = block, r[5] = valid, r[6] = flags;
    }
    ++n;
  };
  for (const tts::UnitRec& r : plan.recs) {
    if (r.nrows <= 0) continue;
    const int32_t u = static_cast<int32_t>(units++);
    const int32_t nbeams = r.nrows / g;
    if (r.mode == tts::kModeWide) {
      for (int32_t e = 0; e < r.nstatic; ++e) {
        const int32_t second = e >= tts::kMaxEntries;
        const int32_t id = second ? r.ent_id2[e - tts::kMaxEntries] : r.ent_id[e];
        for (int32_t i = 0; i < nbeams; ++i) emit(u, e, r.kvh, r.beams[i], id, block_size, 8 | (second ? 4 : 0));
      }
      continue;
    }
    for (int32_t e = 0; e < r.nent + r.nstatic2; ++e) {
      const bool second = e >= r.nent;
      const int32_t id = second ? r.ent_id2[e - r.nent] : r.ent_id[e];
      const uint32_t inf = second ? r.ent_info2[e - r.nent] : r.ent_info[e];
      const int32_t r0 = static_cast<int32_t>(inf & 63), r1 = static_cast<int32_t>((inf >> 6) & 63) + 1;
      const bool ext = (inf & tts::kEntExt) != 0;
      const int32_t flags = ((inf & tts::kEntLive) ? 1 : 0) | (ext ? 2 : 0) | (second ? 4 : 0);
      const int32_t valid = ext ? 0 : static_cast<int32_t>((inf >> 12) & 15) + 1;
      for (int32_t i = r0 / g; i < (r1 + g - 1) / g && i < nbeams; ++i)
        emit(u, e, r.kvh, r.beams[i], ext ? -1 : id, valid, flags);
    }
  }
  *n_rows = n;
  *num_units = units;
  if (n > cap) return fail(TTS_ERR_WORKSPACE, "cap too small for the plan rows");
  return ok();
}

tts_status tts_prefix_meta_stats(const tts_prefix_meta* m, int64_t* num_units, int64_t* num_slots) {
  if (!m || !num_units || !num_slots) return fail(TTS_ERR_INVALID_ARG, "NULL argument");
  if (!m->has_plan) return fail(TTS_ERR_INVALID_ARG, "metadata was built without a desc");
  *num_units = m->plan.num_units;
  *num_slots = m->plan.num_slots;
  return ok();
}

static int32_t paged_nsplit(int32_t max_seq_len) {
  const int32_t nblk = (max_seq_len + 15) / 16;
  const int32_t n = (nblk + kPagedSplitBlocks - 1) / kPagedSplitBlocks;
  return n < 1 ? 1 : n;
}

size_t tts_paged_decode_workspace_size(const tts_attn_desc* d, int32_t num_seqs, int32_t max_seq_len) {
  if (!d || check_desc(d) != TTS_OK || num_seqs < 0 || max_seq_len < 0) return 0;
  const int32_t ns = paged_nsplit(max_seq_len);
  if (ns == 1) return 0;
  const size_t rows = static_cast<size_t>(num_seqs) * ns * d->num_q_heads;
  return part_o_bytes(d, rows) + align256(rows * tts::kPartMl * 4);
}

tts_status tts_paged_decode_attn(const tts_attn_desc* d, int32_t num_seqs, const void* q, const void* k_cache,
                                 const void* v_cache, const float* k_scale, const float* v_scale,
                                 const int32_t* block_tables, int32_t max_blocks_per_seq, const int32_t* seq_lens,
                                 int32_t max_seq_len, int32_t num_blocks, void* out, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream) {
  tts_status s = check_desc(d);
  if (s != TTS_OK) return s;
  if ((s = check_scales(d, k_scale, v_scale)) != TTS_OK) return s;
  if (num_seqs < 0 || max_blocks_per_seq < 0 || max_seq_len < 0 || num_blocks < 0)
    return fail(TTS_ERR_INVALID_ARG, "negative size");
  if (static_cast<int64_t>(max_seq_len) > static_cast<int64_t>(max_blocks_per_seq) * 16)
    return fail(TTS_ERR_INVALID_ARG, "max_seq_len exceeds max_blocks_per_seq * block_size");
  if (num_seqs == 0) return ok();
  if (!q || !k_cache || !v_cache || !block_tables || !seq_lens || !out)
    return fail(TTS_ERR_INVALID_ARG, "NULL device pointer");
  const int32_t ns = paged_nsplit(max_seq_len);
  const size_t need = tts_paged_decode_workspace_size(d, num_seqs, max_seq_len);
  if (need > 0 && (!workspace || workspace_bytes < need))
    return fail(TTS_ERR_WORKSPACE, "workspace smaller than tts_paged_decode_workspace_size");
  const size_t rows = static_cast<size_t>(num_seqs) * ns * d->num_q_heads;
  if (rows > 0x7FFFFFFFu) return fail(TTS_ERR_UNSUPPORTED, "more than 2^31 - 1 partial rows");
  tts::AttnParams p{};
  p.q = q;
  p.k_cache = k_cache;
  p.v_cache = v_cache;
  p.k_scale = k_scale;
  p.v_scale = v_scale;
  p.block_tables = block_tables;
  p.seq_lens = seq_lens;
  p.out = static_cast<float*>(out);
  p.part_o = ns > 1 ? workspace : nullptr;
  p.part_ml = ns > 1 ? reinterpret_cast<float*>(static_cast<char*>(workspace) + part_o_bytes(d, rows))
                     : nullptr;

  p.max_blocks = max_blocks_per_seq;
  p.num_blocks = num_blocks;
  p.num_seqs = num_seqs;
  p.hq = d->num_q_heads;
  p.hkv = d->num_kv_heads;
  p.g = d->num_q_heads / d->num_kv_heads;
  p.scale_log2 = scale_log2(d);
  p.paged_nsplit = ns;
  p.paged_max_len = max_seq_len;
  p.q_len = 1;
  p.two_windows = 0;
  const int64_t units = static_cast<int64_t>(num_seqs) * d->num_kv_heads * ns;
  if (units > 0x7FFFFFFF) return fail(TTS_ERR_UNSUPPORTED, "grid too large");
  hipError_t e = tts::launch_attn(p, static_cast<int>(units), d->head_dim, kv_kind(d), stream);
  if (e != hipSuccess) return fail(TTS_ERR_HIP, std::string("attention launch: ") + hipGetErrorString(e));
  if (ns > 1) {
    tts::MergeParams mp{};
    mp.part_o = p.part_o;
    mp.part_ml = p.part_ml;
    mp.seq_lens = seq_lens;
    mp.out = p.out;
    mp.num_seqs = num_seqs;
    mp.hq = d->num_q_heads;
    mp.g = d->num_q_heads / d->num_kv_heads;
    mp.paged_nsplit = ns;
    e = tts::launch_merge(mp, d->head_dim, kv_kind(d), stream);
    if (e != hipSuccess) return fail(TTS_ERR_HIP, std::string("merge launch: ") + hipGetErrorString(e));
  }
  return ok();
}

size_t tts_prefix_decode_workspace_size(const tts_attn_desc* d, const tts_prefix_meta* m) {
  if (!d || !m || !m->has_plan || check_desc(d) != TTS_OK) return 0;
  const size_t rows = static_cast<size_t>(m->plan.rows_per_head) * d->num_kv_heads;
  return part_o_bytes(d, rows) + align256(rows * tts::kPartMl * 4);
}

namespace {

// Validation shared by the prefix-path entry points; fills the kernel
// parameters on success.
tts_status prefix_params(const tts_attn_desc* d, const tts_prefix_meta* m, const void* q, const void* k_cache,
                         const void* v_cache, const float* k_scale, const float* v_scale,
                         const int32_t* block_tables, int32_t max_blocks_per_seq, const int32_t* seq_lens,
                         int32_t num_blocks, void* out, void* workspace, size_t workspace_bytes, bool need_kv,
                         tts::AttnParams* p) {
  tts_status s = check_desc(d);
  if (s != TTS_OK) return s;
  if (need_kv && (s = check_scales(d, k_scale, v_scale)) != TTS_OK) return s;
  if (!m) return fail(TTS_ERR_INVALID_ARG, "metadata is NULL");
  if (!m->has_plan || !m->dev) return fail(TTS_ERR_INVALID_ARG, "metadata was built without a desc");
  if (m->desc.num_q_heads != d->num_q_heads || m->desc.num_kv_heads != d->num_kv_heads ||
      m->desc.head_dim != d->head_dim)
    return fail(TTS_ERR_INVALID_ARG, "desc shape differs from the one the metadata was built for");
  if (need_kv) {
    if (max_blocks_per_seq != m->host.max_blocks)
      return fail(TTS_ERR_INVALID_ARG, "max_blocks_per_seq differs from the metadata's");
    if (num_blocks < m->num_blocks) return fail(TTS_ERR_INVALID_ARG, "num_blocks smaller than at build time");
  }
  const int32_t S = m->host.num_seqs;
  if (S == 0) return TTS_OK;
  if (!seq_lens || !out || (need_kv && (!q || !k_cache || !v_cache || !block_tables)))
    return fail(TTS_ERR_INVALID_ARG, "NULL device pointer");
  const size_t need = tts_prefix_decode_workspace_size(d, m);
  if (!workspace || workspace_bytes < need)
    return fail(TTS_ERR_WORKSPACE, "workspace smaller than tts_prefix_decode_workspace_size");
  const size_t rows = static_cast<size_t>(m->plan.rows_per_head) * d->num_kv_heads;
  if (rows > 0x7FFFFFFFu) return fail(TTS_ERR_UNSUPPORTED, "more than 2^31 - 1 partial rows");
  const char* dev = static_cast<const char*>(m->dev);
  *p = tts::AttnParams{};
  p->q = q;
  p->k_cache = k_cache;
  p->v_cache = v_cache;
  p->k_scale = k_scale;
  p->v_scale = v_scale;
  p->block_tables = block_tables;
  p->seq_lens = seq_lens;
  p->out = static_cast<float*>(out);
  p->part_o = workspace;
  p->part_ml = reinterpret_cast<float*>(static_cast<char*>(workspace) + part_o_bytes(d, rows));
  p->recs = reinterpret_cast<const tts::UnitRec*>(dev + m->off_recs);
  p->build_len = reinterpret_cast<const int32_t*>(dev + m->off_build);
  p->rows_per_head = m->plan.rows_per_head;
  p->max_blocks = max_blocks_per_seq;
  p->num_blocks = num_blocks;
  p->num_seqs = S;
  p->hq = d->num_q_heads;
  p->hkv = d->num_kv_heads;
  p->g = d->num_q_heads / d->num_kv_heads;
  p->scale_log2 = scale_log2(d);
  p->q_len = m->q_len;
  p->two_windows = m->plan.two_windows ? 1 : 0;
  return TTS_OK;
}

tts_status launch_partials(const tts_attn_desc* d, const tts_prefix_meta* m, const tts::AttnParams& p,
                           hipStream_t stream) {
  hipError_t e = tts::launch_attn(p, m->plan.num_bins, d->head_dim, kv_kind(d), stream);
  if (e != hipSuccess) return fail(TTS_ERR_HIP, std::string("attention launch: ") + hipGetErrorString(e));
  return TTS_OK;
}

tts_status launch_prefix_merge(const tts_attn_desc* d, const tts_prefix_meta* m, const tts::AttnParams& p,
                               hipStream_t stream) {
  const char* dev = static_cast<const char*>(m->dev);
  tts::MergeParams mp{};
  mp.part_o = p.part_o;
  mp.part_ml = p.part_ml;
  mp.slot_tab = reinterpret_cast<const int32_t*>(dev + m->off_slot_tab);
  mp.slot_stride = m->plan.slot_stride;
  mp.seq_lens = p.seq_lens;
  mp.build_len = p.build_len;
  mp.out = p.out;
  mp.num_seqs = p.num_seqs;
  mp.hq = d->num_q_heads;
  mp.g = p.g;
  mp.q_len = p.q_len;
  mp.rows_per_head = p.rows_per_head;
  hipError_t e = tts::launch_merge(mp, d->head_dim, kv_kind(d), stream);
  if (e != hipSuccess) return fail(TTS_ERR_HIP, std::string("merge launch: ") + hipGetErrorString(e));
  return TTS_OK;
}

}  // namespace

tts_status tts_prefix_decode_attn(const tts_attn_desc* d, const tts_prefix_meta* m, const void* q,
                                  const void* k_cache, const void* v_cache, const float* k_scale,
                                  const float* v_scale, const int32_t* block_tables, int32_t max_blocks_per_seq,
                                  const int32_t* seq_lens, int32_t num_blocks, void* out, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream) {
  if (m && m->q_len != 1)
    return fail(TTS_ERR_INVALID_ARG, "verification metadata (q_len > 1): use tts_prefix_verify_attn");
  tts::AttnParams p;
  tts_status s = prefix_params(d, m, q, k_cache, v_cache, k_scale, v_scale, block_tables, max_blocks_per_seq,
                               seq_lens, num_blocks, out, workspace, workspace_bytes, true, &p);
  if (s != TTS_OK || m->host.num_seqs == 0) return s == TTS_OK ? ok() : s;
  if ((s = launch_partials(d, m, p, stream)) != TTS_OK) return s;
  if ((s = launch_prefix_merge(d, m, p, stream)) != TTS_OK) return s;
  return ok();
}

tts_status tts_prefix_decode_attn_noalloc(const tts_attn_desc* d, const tts_prefix_meta* m, const void* q,
                                          const void* k_cache, const void* v_cache, const float* k_scale,
                                          const float* v_scale, const int32_t* block_tables,
                                          int32_t max_blocks_per_seq, const int32_t* seq_lens, int32_t num_blocks,
                                          void* out, hipStream_t stream) {
  if (m && m->q_len != 1)
    return fail(TTS_ERR_INVALID_ARG, "verification metadata (q_len > 1): use tts_prefix_verify_attn");
  // The library's own scratch array on the current device (no allocation).
  void* scratch = nullptr;
  size_t scratch_bytes = 0;
  const hipError_t e = tts::scratch_buffer(&scratch, &scratch_bytes);
  if (e != hipSuccess) return fail(TTS_ERR_HIP, std::string("scratch lookup: ") + hipGetErrorString(e));
  if (d && m && m->has_plan && check_desc(d) == TTS_OK) {
    const size_t need = tts_prefix_decode_workspace_size(d, m);
    if (need > scratch_bytes)
      return fail(TTS_ERR_WORKSPACE, "the plan needs " + std::to_string(need) + " bytes of partial states; the "
                  "allocation-free call holds " + std::to_string(scratch_bytes) + " (use tts_prefix_decode_attn "
                  "with a workspace)");
  }
  tts::AttnParams p;
  tts_status s = prefix_params(d, m, q, k_cache, v_cache, k_scale, v_scale, block_tables, max_blocks_per_seq,
                               seq_lens, num_blocks, out, scratch, scratch_bytes, true, &p);
  if (s != TTS_OK || m->host.num_seqs == 0) return s == TTS_OK ? ok() : s;
  if ((s = launch_partials(d, m, p, stream)) != TTS_OK) return s;
  if ((s = launch_prefix_merge(d, m, p, stream)) != TTS_OK) return s;
  return ok();
}

tts_status tts_prefix_verify_attn(const tts_attn_desc* d, const tts_prefix_meta* m, const void* q,
                                  const void* k_cache, const void* v_cache, const float* k_scale,
                                  const float* v_scale, const int32_t* block_tables, int32_t max_blocks_per_seq,
                                  const int32_t* seq_lens, int32_t num_blocks, void* out, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream) {
  tts::AttnParams p;
  tts_status s = prefix_params(d, m, q, k_cache, v_cache, k_scale, v_scale, block_tables, max_blocks_per_seq,
                               seq_lens, num_blocks, out, workspace, workspace_bytes, true, &p);
  if (s != TTS_OK || m->host.num_seqs == 0) return s == TTS_OK ? ok() : s;
  if ((s = launch_partials(d, m, p, stream)) != TTS_OK) return s;
  if ((s = launch_prefix_merge(d, m, p, stream)) != TTS_OK) return s;
  return ok();
}

tts_status tts_prefix_decode_partials(const tts_attn_desc* d, const tts_prefix_meta* m, const void* q,
                                      const void* k_cache, const void* v_cache, const float* k_scale,
                                      const float* v_scale, const int32_t* block_tables,
                                      int32_t max_blocks_per_seq, const int32_t* seq_lens, int32_t num_blocks,
                                      void* out, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  tts::AttnParams p;
  tts_status s = prefix_params(d, m, q, k_cache, v_cache, k_scale, v_scale, block_tables, max_blocks_per_seq,
                               seq_lens, num_blocks, out, workspace, workspace_bytes, true, &p);
  if (s != TTS_OK || m->host.num_seqs == 0) return s == TTS_OK ? ok() : s;
  if ((s = launch_partials(d, m, p, stream)) != TTS_OK) return s;
  return ok();
}

tts_status tts_prefix_decode_merge(const tts_attn_desc* d, const tts_prefix_meta* m, const int32_t* seq_lens,
                                   void* out, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  tts::AttnParams p;
  tts_status s = prefix_params(d, m, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0, seq_lens, 0, out,
                               workspace, workspace_bytes, false, &p);
  if (s != TTS_OK || m->host.num_seqs == 0) return s == TTS_OK ? ok() : s;
  if ((s = launch_prefix_merge(d, m, p, stream)) != TTS_OK) return s;
  return ok();
}

// ---- KV maintenance ----------------------------------------------------------

tts_status tts_append_kv(const tts_attn_desc* d, int32_t num_seqs, const void* k_new, const void* v_new,
                         const int32_t* block_tables, int32_t max_blocks_per_seq, const int32_t* seq_lens,
                         int32_t num_blocks, void* k_cache, void* v_cache, float* k_scale, float* v_scale,
                         hipStream_t stream) {
  tts_status s = check_desc(d);
  if (s != TTS_OK) return s;
  if ((s = check_scales(d, k_scale, v_scale)) != TTS_OK) return s;
  if (num_seqs < 0 || max_blocks_per_seq < 0 || num_blocks < 0) return fail(TTS_ERR_INVALID_ARG, "negative size");
  if (num_seqs == 0) return ok();
  if (!k_new || !v_new || !block_tables || !seq_lens || !k_cache || !v_cache)
    return fail(TTS_ERR_INVALID_ARG, "NULL device pointer");
  hipError_t e = tts::launch_append(k_new, v_new, block_tables, seq_lens, k_cache, v_cache, k_scale, v_scale, num_seqs,
                                    max_blocks_per_seq, num_blocks, d->num_kv_heads, d->head_dim, kv_kind(d), stream);
  if (e != hipSuccess) return fail(TTS_ERR_HIP, std::string("append launch: ") + hipGetErrorString(e));
  return ok();
}

tts_status tts_copy_blocks(const tts_attn_desc* d, int32_t num_pairs, const int32_t* pairs, int32_t num_blocks,
                           void* k_cache, void* v_cache, float* k_scale, float* v_scale, hipStream_t stream) {
  tts_status s = check_desc(d);
  if (s != TTS_OK) return s;
  if ((s = check_scales(d, k_scale, v_scale)) != TTS_OK) return s;
  if (num_pairs < 0 || num_blocks < 0) return fail(TTS_ERR_INVALID_ARG, "negative size");
  if (num_pairs == 0) return ok();
  if (!pairs || !k_cache || !v_cache) return fail(TTS_ERR_INVALID_ARG, "NULL device pointer");
  const int64_t eb = d->kv_dtype == TTS_F32 ? 4 : (d->kv_dtype == TTS_BF16 ? 2 : 1);
  const int64_t blk_bytes = static_cast<int64_t>(d->num_kv_heads) * d->block_size * d->head_dim * eb;
  hipError_t e = tts::launch_copy_blocks(pairs, num_pairs, k_cache, v_cache, k_scale, v_scale, blk_bytes, num_blocks,
                                         stream);
  if (e != hipSuccess) return fail(TTS_ERR_HIP, std::string("copy launch: ") + hipGetErrorString(e));
  return ok();
}

tts_status tts_fork_tables(int32_t num_parents, const int32_t* parent_tables, int32_t max_blocks_per_seq,
                           const int32_t* parent_lens, int32_t block_size, int32_t num_children,
                           const int32_t* child_parent, const int32_t* child_lens, const int32_t* free_ids,
                           int32_t num_free, int32_t* child_tables, int32_t* copies, int32_t* num_copies,
                           int32_t* num_free_used) {
  if (num_parents < 0 || num_children < 0 || max_blocks_per_seq < 0 || num_free < 0 || block_size <= 0)
    return fail(TTS_ERR_INVALID_ARG, "negative size");
  if (!num_copies || !num_free_used) return fail(TTS_ERR_INVALID_ARG, "NULL output count");
  *num_copies = 0;
  *num_free_used = 0;
  if (num_children == 0) return ok();
  if (!child_parent || !child_lens || !child_tables || !copies || (num_parents > 0 && (!parent_tables || !parent_lens)))
    return fail(TTS_ERR_INVALID_ARG, "NULL host array");
  // Validate everything before writing anything.
  int32_t need = 0;
  for (int32_t c = 0; c < num_children; ++c) {
    const int32_t par = child_parent[c];
    if (par < 0 || par >= num_parents) return fail(TTS_ERR_OUT_OF_RANGE, "child_parent outside [0, num_parents)");
    const int32_t pl = parent_lens[par], cl = child_lens[c];
    if (pl < 0 || static_cast<int64_t>(pl) > static_cast<int64_t>(max_blocks_per_seq) * block_size)
      return fail(TTS_ERR_INVALID_ARG, "parent length outside [0, max_blocks_per_seq * block_size]");
    if (cl < 0 || cl > pl) return fail(TTS_ERR_INVALID_ARG, "child length outside [0, parent length]");
    if (cl % block_size) ++need;
  }
  if (need > num_free) return fail(TTS_ERR_NOMEM, "not enough free blocks for the copied partial blocks");
  for (int32_t c = 0; c < num_children; ++c) {
    const int32_t par = child_parent[c], cl = child_lens[c];
    const int32_t* prow = parent_tables + static_cast<int64_t>(par) * max_blocks_per_seq;
    int32_t* crow = child_tables + static_cast<int64_t>(c) * max_blocks_per_seq;
    const int32_t full = cl / block_size;
    for (int32_t j = 0; j < max_blocks_per_seq; ++j) crow[j] = j < full ? prow[j] : -1;
    if (cl % block_size) {
      const int32_t dst = free_ids[(*num_free_used)++];
      crow[full] = dst;
      copies[2 * *num_copies] = prow[full];
      copies[2 * *num_copies + 1] = dst;
      ++*num_copies;
    }
  }
  return ok();
}

// ---- roofline-guided KV allocation --------------------------------------------

static tts_status check_alloc(const tts_alloc_problem* pr) {
  if (!pr) return fail(TTS_ERR_INVALID_ARG, "problem is NULL");
  if (pr->num_requests < 1 || pr->verify_len < 1 || pr->decode_len < 1)
    return fail(TTS_ERR_INVALID_ARG, "num_requests, verify_len and decode_len must be >= 1");
  if (!(pr->mem_bytes > 0) || !(pr->peak_flops > 0) || !(pr->peak_bw > 0))
    return fail(TTS_ERR_INVALID_ARG, "mem_bytes, peak_flops and peak_bw must be > 0");
  const tts_model_cost* ms[2] = {&pr->verifier, &pr->generator};
  for (const tts_model_cost* m : ms)
    if (!(m->kv_bytes_per_token > 0) || !(m->params >= 0) || !(m->weight_bytes >= 0) || m->num_layers < 0 ||
        m->attn_dim < 0)
      return fail(TTS_ERR_INVALID_ARG, "model cost fields out of range (kv_bytes_per_token must be > 0)");
  return TTS_OK;
}

tts_status tts_kv_alloc_time(const tts_alloc_problem* pr, int64_t b_pre, int64_t b_dec, tts_alloc_result* out) {
  tts_status s = check_alloc(pr);
  if (s != TTS_OK) return s;
  if (!out) return fail(TTS_ERR_INVALID_ARG, "out is NULL");
  if (b_pre < 1 || b_dec < 1) return fail(TTS_ERR_INVALID_ARG, "batch sizes must be >= 1");
  tts::alloc_time(*pr, b_pre, b_dec, out);
  return ok();
}

tts_status tts_kv_alloc_search(const tts_alloc_problem* pr, tts_alloc_result* out) {
  tts_status s = check_alloc(pr);
  if (s != TTS_OK) return s;
  if (!out) return fail(TTS_ERR_INVALID_ARG, "out is NULL");
  if (!tts::alloc_search(*pr, out))
    return fail(TTS_ERR_NOMEM, "the budget does not hold one prefill and one decode sequence");
  return ok();
}

// ---- prefix-aware scheduling -------------------------------------------------

tts_status tts_prefix_schedule(int32_t num_cots, const int32_t* cot_offsets, const int32_t* cot_nodes,
                               int32_t num_nodes, const int64_t* node_weight, int64_t budget, int32_t* order,
                               int32_t* batch_offsets, int32_t* num_batches, int64_t* score, int64_t* cost) {
  if (num_cots < 0 || num_nodes < 0) return fail(TTS_ERR_INVALID_ARG, "negative size");
  if (!num_batches || !score || !cost) return fail(TTS_ERR_INVALID_ARG, "NULL output");
  if (num_cots > 0 && (!cot_offsets || !order || !batch_offsets)) return fail(TTS_ERR_INVALID_ARG, "NULL host array");
  if (num_cots > 0 && cot_offsets[0] != 0) return fail(TTS_ERR_INVALID_ARG, "cot_offsets[0] must be 0");
  for (int32_t c = 0; c < num_cots; ++c)
    if (cot_offsets[c + 1] < cot_offsets[c]) return fail(TTS_ERR_INVALID_ARG, "cot_offsets not monotone");
  const int32_t total = num_cots > 0 ? cot_offsets[num_cots] : 0;
  if (total > 0 && !cot_nodes) return fail(TTS_ERR_INVALID_ARG, "NULL cot_nodes");
  for (int32_t j = 0; j < total; ++j)
    if (cot_nodes[j] < 0 || cot_nodes[j] >= num_nodes) return fail(TTS_ERR_OUT_OF_RANGE, "node id outside [0, num_nodes)");
  if (node_weight)
    for (int32_t v = 0; v < num_nodes; ++v)
      if (node_weight[v] < 0) return fail(TTS_ERR_INVALID_ARG, "negative node weight");
  tts::SchedInput in{num_cots, cot_offsets, cot_nodes, node_weight, budget};
  tts::SchedOutput out;
  try {
    tts::prefix_schedule(in, &out);
  } catch (const std::bad_alloc&) {
    return fail(TTS_ERR_NOMEM, "host allocation failed");
  }
  std::copy(out.order.begin(), out.order.end(), order);
  if (num_cots > 0) std::copy(out.batch_off.begin(), out.batch_off.end(), batch_offsets);
  *num_batches = num_cots > 0 ? static_cast<int32_t>(out.batch_off.size()) - 1 : 0;
  *score = out.score;
  *cost = out.cost;
  return ok();
}

#ifdef TTS_PROFILE_UNITS
// Tuning builds only: copy the unit records of a handle.
int64_t tts_prof_recs(const tts_prefix_meta* m, void* out, int64_t cap) {
  const int64_t n = static_cast<int64_t>(m->plan.recs.size());
  if (out) std::memcpy(out, m->plan.recs.data(), sizeof(tts::UnitRec) * static_cast<size_t>(std::min(n, cap)));
  return n;
}
#endif

}  // extern "C"
