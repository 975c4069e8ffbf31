// HIP kernels (gfx950) for prefix-shared beam decode attention.
//
// One kernel processes "work units" (tts_work.h): up to 64 query rows of one
// KV head against a run of KV blocks. Four waves share every K/V chunk the
// workgroup stages in LDS: when the unit has many rows (a segment shared by
// many beams) each wave takes 16 rows and all waves read the same chunk;
// when it has few rows (a private tail) the waves split the chunk's blocks
// and combine their softmax states at the end. Both products run on MFMA:
//   S^T = K Q^T  (M = 16 tokens, N = 16 rows, K = head dim)
//   O^T += V^T P^T (M = 16 dims, N = 16 rows, K = 16 tokens)
// Computing S transposed leaves each lane with 4 tokens of one row, so the
// softmax reductions are mostly lane-local, and the probabilities feed the
// second product straight from the accumulator registers. Values are stored
// dim-major inside a block, which makes the token run each lane needs for
// that product contiguous.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "tts_work.h"

namespace tts {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kTok = 16;  // tokens per KV block
constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr float kNegInf = -__builtin_inff();

enum KvKind : int { kKvF32 = 0, kKvBf16 = 1, kKvFp8 = 2 };

template <int KV>
struct KvTraits;
template <>
struct KvTraits<kKvF32> {
  static constexpr int bytes = 4;
};
template <>
struct KvTraits<kKvBf16> {
  static constexpr int bytes = 2;
};
template <>
struct KvTraits<kKvFp8> {
  static constexpr int bytes = 1;
};

template <int D, int KV>
struct Geo {
  static constexpr int eb = KvTraits<KV>::bytes;
  static constexpr int row_bytes = D * eb;           // one token of K
  static constexpr int c16 = row_bytes / 16;          // 16-byte columns per K row
  static constexpr int blk_bytes = kTok * row_bytes;  // one (block, head) of K or V
  static constexpr int vec_per_blk = blk_bytes / 16;
  static constexpr int vrow_bytes = kTok * eb;        // one dim of V (16 tokens)
  static constexpr int chunk = (16384 / blk_bytes) < 2 ? 2 : ((16384 / blk_bytes) > 8 ? 8 : (16384 / blk_bytes));
  static constexpr int stage_bytes = chunk * 2 * blk_bytes;
  static constexpr int vpt = (vec_per_blk + kThreads - 1) / kThreads;  // 16-byte loads per thread per block/tensor
  static constexpr int combine_bytes = kWaves * (kTok * D + 2 * kTok) * 4;
  static constexpr int lds_bytes = (2 * stage_bytes) > combine_bytes ? (2 * stage_bytes) : combine_bytes;
};

__device__ __forceinline__ uint32_t f32_bits(float x) { return __builtin_bit_cast(uint32_t, x); }

// Two OCP E4M3 codes (byte pair `hi` of w) -> two bf16 in one dword. The
// conversion to fp32 is exact and every E4M3 value fits bf16 exactly, so
// dropping the low half of the fp32 pattern is exact too.
template <bool kHi>
__device__ __forceinline__ uint32_t fp8x2_to_bf16x2(uint32_t w) {
  f32x2 f = __builtin_amdgcn_cvt_pk_f32_fp8(w, kHi);
  return (f32_bits(f.x) >> 16) | (f32_bits(f.y) & 0xFFFF0000u);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  // Round to nearest even (finite inputs: probabilities in [0, 1] times a scale).
  uint32_t ua = f32_bits(a), ub = f32_bits(b);
  ua += 0x7FFFu + ((ua >> 16) & 1u);
  ub += 0x7FFFu + ((ub >> 16) & 1u);
  return (ua >> 16) | (ub & 0xFFFF0000u);
}

__device__ __forceinline__ float wave_max16(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  x = fmaxf(x, __shfl_xor(x, 32));
  return x;
}
__device__ __forceinline__ float wave_sum16(float x) {
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 32);
  return x;
}

// Block run of one unit, resolved from the metadata or the live tables.
struct Run {
  const int32_t* ids;  // block ids (segment) or table row (tail)
  int32_t first;       // first index into ids
  int32_t nblk;        // blocks in this unit
  int32_t len;         // tail: beam length (last block may be partial); segment: unused
  bool tail;
  bool bad;
};

template <int D, int KV>
__global__ __launch_bounds__(kThreads) void attn_units_kernel(AttnParams p) {
  using G = Geo<D, KV>;
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int ln = lane & 15;  // row (N) / token (M) index inside a 16x16 tile
  const int lq = lane >> 4;  // k-group of the lane

  // ---- the unit ----------------------------------------------------------
  Unit u;
  if (p.units) {
    u = p.units[blockIdx.x];
  } else {  // paged path: unit = (beam, kv head, split), no sharing
    const int j = blockIdx.x % p.paged_nsplit;
    const int bh = blockIdx.x / p.paged_nsplit;
    u.kvh = bh % p.hkv;
    u.kind = kTailSplit;
    u.pos0 = bh / p.hkv;
    u.nbeams = 1;
    u.row0 = 0;
    u.nrows = p.g;
    u.blk_off = j;
    u.nblk = p.paged_nsplit;
    u.slot = j;
  }

  Run run;
  run.bad = false;
  run.len = 0;
  if (u.kind == kSegmentPiece) {
    run.tail = false;
    run.ids = p.seg_blocks;
    run.first = u.blk_off;
    run.nblk = u.nblk;
  } else {
    run.tail = true;
    const int b = p.perm ? p.perm[u.pos0] : u.pos0;
    const int L = p.seq_lens[b];
    const int t0 = p.tail_lblock ? p.tail_lblock[b] : 0;
    int nb_all = (L + kTok - 1) / kTok;
    if (L < 0 || nb_all > p.max_blocks || (!p.perm && L > p.paged_max_len) || nb_all < t0) {
      run.bad = true;
      nb_all = t0;
    }
    const int tb = nb_all - t0;
    const int per = (tb + u.nblk - 1) / u.nblk;
    int a = t0 + u.blk_off * per;
    int e = a + per;
    if (e > nb_all) e = nb_all;
    if (a > e) a = e;
    run.ids = p.block_tables + static_cast<int64_t>(b) * p.max_blocks;
    run.first = a;
    run.nblk = e - a;
    run.len = L;
  }

  // ---- wave roles --------------------------------------------------------
  const int nrt = (u.nrows + 15) >> 4;
  const int wr = nrt >= 3 ? 4 : nrt;  // waves splitting rows
  const int wt = kWaves / wr;         // waves splitting blocks
  const int rt = wave % wr;
  const int tl = wave / wr;
  const int rloc = rt * 16 + ln;
  const bool row_ok = rloc < u.nrows;
  const bool wave_active = rt * 16 < u.nrows;
  int beam = 0, qh = 0;
  {
    const int r = u.row0 + (row_ok ? rloc : 0);
    const int pos = u.pos0 + r / p.g;
    beam = p.perm ? p.perm[pos] : pos;
    qh = u.kvh * p.g + r % p.g;
  }

  // ---- query fragments (B operand of S^T = K Q^T) ------------------------
  constexpr int kQf = (KV == kKvF32) ? D / 16 : D / 32;
  typedef typename std::conditional<KV == kKvF32, f32x4, bf16x8>::type QFrag;
  QFrag qf[kQf];
  if (KV == kKvF32) {
    const float* qrow = static_cast<const float*>(p.q) + (static_cast<int64_t>(beam) * p.hq + qh) * D;
#pragma unroll
    for (int j = 0; j < kQf; ++j) {
      f32x4 v = row_ok ? *reinterpret_cast<const f32x4*>(qrow + 16 * j + 4 * lq) : f32x4{0.f, 0.f, 0.f, 0.f};
      qf[j] = __builtin_bit_cast(QFrag, v);
    }
  } else {
    const uint16_t* qrow = static_cast<const uint16_t*>(p.q) + (static_cast<int64_t>(beam) * p.hq + qh) * D;
#pragma unroll
    for (int j = 0; j < kQf; ++j) {
      uint4 v = row_ok ? *reinterpret_cast<const uint4*>(qrow + 32 * j + 8 * lq) : uint4{0u, 0u, 0u, 0u};
      qf[j] = __builtin_bit_cast(QFrag, v);
    }
  }

  // ---- running softmax state (rows n = ln; O^T in C layout) --------------
  f32x4 o[D / 16];
#pragma unroll
  for (int i = 0; i < D / 16; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = kNegInf;
  float l_run = 0.f;

  const size_t kv_head_stride = G::blk_bytes;
  const size_t kv_blk_stride = static_cast<size_t>(p.hkv) * G::blk_bytes;
  const unsigned char* kbase_g = static_cast<const unsigned char*>(p.k_cache) + u.kvh * kv_head_stride;
  const unsigned char* vbase_g = static_cast<const unsigned char*>(p.v_cache) + u.kvh * kv_head_stride;

  // Block id / valid tokens of the i-th block of the run (ids are validated
  // on the host for segments and checked here for tails).
  auto block_of = [&](int i, int* valid) -> int {
    int id = run.ids[run.first + i];
    if (run.tail) {
      const int lb = run.first + i;
      int v = run.len - lb * kTok;
      *valid = v < kTok ? v : kTok;
      if (id < 0 || id >= p.num_blocks) {
        run.bad = true;
        id = 0;
        *valid = 0;
      }
    } else {
      *valid = kTok;
    }
    return id;
  };

  // Register staging of one chunk: per block, K then V, vpt 16-byte vectors each.
  uint4 stg[G::chunk][2][G::vpt];
  int stg_valid[G::chunk];
  const int nchunks = (run.nblk + G::chunk - 1) / G::chunk;

  auto load_chunk = [&](int c) {
#pragma unroll
    for (int bi = 0; bi < G::chunk; ++bi) {
      const int i = c * G::chunk + bi;
      stg_valid[bi] = 0;
      if (i < run.nblk) {
        int valid;
        const int id = block_of(i, &valid);
        stg_valid[bi] = valid;
        const unsigned char* kp = kbase_g + static_cast<size_t>(id) * kv_blk_stride;
        const unsigned char* vp = vbase_g + static_cast<size_t>(id) * kv_blk_stride;
#pragma unroll
        for (int t = 0; t < G::vpt; ++t) {
          const int vec = tid + t * kThreads;
          if (vec < G::vec_per_blk && valid > 0) {
            stg[bi][0][t] = *reinterpret_cast<const uint4*>(kp + vec * 16);
            stg[bi][1][t] = *reinterpret_cast<const uint4*>(vp + vec * 16);
          }
        }
      }
    }
  };

  // Write the staged chunk to LDS stage `s`; masked slots become zero. K rows
  // are XOR-swizzled by token so the 16 lanes reading one column of 16
  // tokens hit distinct banks.
  auto store_chunk = [&](int c, int s) {
    unsigned char* st = lds + s * G::stage_bytes;
#pragma unroll
    for (int bi = 0; bi < G::chunk; ++bi) {
      const int i = c * G::chunk + bi;
      if (i >= run.nblk) continue;
      const int valid = stg_valid[bi];
      unsigned char* kd = st + bi * 2 * G::blk_bytes;
      unsigned char* vd = kd + G::blk_bytes;
#pragma unroll
      for (int t = 0; t < G::vpt; ++t) {
        const int vec = tid + t * kThreads;
        if (vec >= G::vec_per_blk) continue;
        uint4 kv = stg[bi][0][t];
        uint4 vv = stg[bi][1][t];
        const int krow = vec / G::c16;
        const int kcol = vec % G::c16;
        if (krow >= valid) kv = uint4{0u, 0u, 0u, 0u};
        if (valid < kTok) {
          // V vector = tokens [tok0, tok0 + 16/eb) of one dim.
          constexpr int per = 16 / G::eb;
          constexpr uint32_t emask = G::eb == 4 ? 0xFFFFFFFFu : ((1u << ((G::eb * 8) & 31)) - 1u);
          const int tok0 = (vec % G::eb) * per;
          uint32_t w[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
          for (int e = 0; e < per; ++e) {
            if (tok0 + e >= valid) {
              const int bit = e * G::eb * 8;
              w[bit >> 5] &= ~(emask << (bit & 31));
            }
          }
          vv = uint4{w[0], w[1], w[2], w[3]};
        }
        *reinterpret_cast<uint4*>(kd + krow * G::row_bytes + ((kcol ^ (krow & (G::c16 - 1))) << 4)) = kv;
        *reinterpret_cast<uint4*>(vd + vec * 16) = vv;
      }
    }
  };

  // One 16-token block for this wave's 16 rows: S tile, online softmax, PV.
  auto do_block = [&](const unsigned char* kd, const unsigned char* vd, int valid, float kscale, float vscale) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    const unsigned char* krow = kd + ln * G::row_bytes;
    const int sw = ln & (G::c16 - 1);
    if constexpr (KV == kKvF32) {
#pragma unroll
      for (int j = 0; j < D / 16; ++j) {
        const f32x4 a = *reinterpret_cast<const f32x4*>(krow + (((4 * j + lq) ^ sw) << 4));
        const f32x4 b = __builtin_bit_cast(f32x4, qf[j]);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, b.x, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, b.y, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, b.z, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, b.w, acc, 0, 0, 0);
      }
    } else if constexpr (KV == kKvBf16) {
#pragma unroll
      for (int kk = 0; kk < D / 32; ++kk) {
        const uint4 a = *reinterpret_cast<const uint4*>(krow + (((4 * kk + lq) ^ sw) << 4));
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                      __builtin_bit_cast(bf16x8, qf[kk]), acc, 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int kk = 0; kk < D / 32; ++kk) {
        const int col = 2 * kk + (lq >> 1);
        const uint2 w = *reinterpret_cast<const uint2*>(krow + ((col ^ sw) << 4) + 8 * (lq & 1));
        const uint4 a = {fp8x2_to_bf16x2<false>(w.x), fp8x2_to_bf16x2<true>(w.x), fp8x2_to_bf16x2<false>(w.y),
                         fp8x2_to_bf16x2<true>(w.y)};
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                      __builtin_bit_cast(bf16x8, qf[kk]), acc, 0, 0, 0);
      }
    }
    // acc[i] = S[row ln][token 4*lq + i]
    const float sc = p.scale_log2 * kscale;
    float s[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) s[i] = (4 * lq + i < valid) ? acc[i] * sc : kNegInf;
    float tmax = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
    tmax = wave_max16(tmax);
    const float m_new = fmaxf(m_run, tmax);
    const float m_use = (m_new == kNegInf) ? 0.f : m_new;
    const float alpha = exp2f(m_run - m_use);
    float pr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) pr[i] = exp2f(s[i] - m_use);
    l_run = l_run * alpha + ((pr[0] + pr[1]) + (pr[2] + pr[3]));
    m_run = m_new;
#pragma unroll
    for (int i = 0; i < D / 16; ++i) o[i] *= alpha;
    if constexpr (KV == kKvF32) {
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        const f32x4 a = *reinterpret_cast<const f32x4*>(vd + (16 * dt + ln) * G::vrow_bytes + 16 * lq);
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, pr[0], o[dt], 0, 0, 0);
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, pr[1], o[dt], 0, 0, 0);
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, pr[2], o[dt], 0, 0, 0);
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, pr[3], o[dt], 0, 0, 0);
      }
    } else {
      const uint2 pb = {pack_bf16x2(pr[0] * vscale, pr[1] * vscale), pack_bf16x2(pr[2] * vscale, pr[3] * vscale)};
      const bf16x4 bfr = __builtin_bit_cast(bf16x4, pb);
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        uint2 a;
        if constexpr (KV == kKvBf16) {
          a = *reinterpret_cast<const uint2*>(vd + (16 * dt + ln) * G::vrow_bytes + 8 * lq);
        } else {
          const uint32_t w = *reinterpret_cast<const uint32_t*>(vd + (16 * dt + ln) * G::vrow_bytes + 4 * lq);
          a = uint2{fp8x2_to_bf16x2<false>(w), fp8x2_to_bf16x2<true>(w)};
        }
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(bf16x4, a), bfr, o[dt], 0, 0, 0);
      }
    }
  };

  // ---- main loop: double-buffered LDS stages ------------------------------
  if (nchunks > 0) load_chunk(0);
  for (int c = 0; c < nchunks; ++c) {
    const int s = c & 1;
    store_chunk(c, s);
    __syncthreads();
    if (c + 1 < nchunks) load_chunk(c + 1);
    if (wave_active) {
      const unsigned char* st = lds + s * G::stage_bytes;
      const int nb = (run.nblk - c * G::chunk) < G::chunk ? (run.nblk - c * G::chunk) : G::chunk;
      for (int bi = tl; bi < nb; bi += wt) {
        int valid = kTok;
        float ks = 1.f, vs = 1.f;
        if (run.tail) {
          const int lb = run.first + c * G::chunk + bi;
          valid = run.len - lb * kTok;
          valid = valid < kTok ? valid : kTok;
        }
        if constexpr (KV == kKvFp8) {
          int v2;
          const int id = block_of(c * G::chunk + bi, &v2);
          ks = p.k_scale[id];
          vs = p.v_scale[id];
        }
        do_block(st + bi * 2 * G::blk_bytes, st + bi * 2 * G::blk_bytes + G::blk_bytes, valid, ks, vs);
      }
    }
  }

  // ---- combine the waves that split blocks, then write -------------------
  float l_tot = wave_sum16(l_run);
  if (wt > 1) {
    __syncthreads();  // stages are free now
    float* cb = reinterpret_cast<float*>(lds);
    float* my = cb + (tl * wr + rt) * (kTok * D + 2 * kTok);
    if (wave_active) {
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt)
        *reinterpret_cast<f32x4*>(my + ln * D + 16 * dt + 4 * lq) = o[dt];
      if (lq == 0) {
        my[kTok * D + ln] = m_run;
        my[kTok * D + kTok + ln] = l_tot;
      }
    }
    __syncthreads();
    if (tl == 0 && wave_active) {
      float mt[kWaves];
      float mx = kNegInf;
      for (int t = 0; t < wt; ++t) {
        const float* ot = cb + (t * wr + rt) * (kTok * D + 2 * kTok);
        mt[t] = ot[kTok * D + ln];
        mx = fmaxf(mx, mt[t]);
      }
      const float mu = (mx == kNegInf) ? 0.f : mx;
      l_tot = 0.f;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int t = 0; t < wt; ++t) {
        const float* ot = cb + (t * wr + rt) * (kTok * D + 2 * kTok);
        const float f = exp2f(mt[t] - mu);
        l_tot += ot[kTok * D + kTok + ln] * f;
#pragma unroll
        for (int dt = 0; dt < D / 16; ++dt)
          o[dt] += *reinterpret_cast<const f32x4*>(ot + ln * D + 16 * dt + 4 * lq) * f;
      }
      m_run = mx;
    }
  }
  if (tl != 0 || !row_ok) return;
  if (run.bad) m_run = __builtin_nanf("");

  if (!p.units && p.paged_nsplit == 1) {
    // Whole sequence in this unit: write the normalised result.
    float* orow = p.out + (static_cast<int64_t>(beam) * p.hq + qh) * D;
    const float inv = (l_tot > 0.f) ? 1.f / l_tot : 0.f;
    const bool nan = m_run != m_run;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) {
      f32x4 v = o[dt] * inv;
      if (nan) v = f32x4{m_run, m_run, m_run, m_run};
      *reinterpret_cast<f32x4*>(orow + 16 * dt + 4 * lq) = v;
    }
    return;
  }
  int64_t prow;
  if (p.units)
    prow = static_cast<int64_t>(p.slot_base[beam] + u.slot) * p.hq + qh;
  else
    prow = (static_cast<int64_t>(beam) * p.paged_nsplit + u.slot) * p.hq + qh;
  float* po = p.part_o + prow * D;
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) *reinterpret_cast<f32x4*>(po + 16 * dt + 4 * lq) = o[dt];
  if (lq == 0) {
    p.part_ml[prow * 2] = m_run;
    p.part_ml[prow * 2 + 1] = l_tot;
  }
}

// Exact merge of partial softmax states, in slot order (segments root to
// leaf, then tail splits): m = max m_k, l = sum l_k 2^(m_k - m),
// out = sum o_k 2^(m_k - m) / l. One wave per (beam, query head).
template <int D>
__global__ __launch_bounds__(kThreads) void merge_kernel(MergeParams p) {
  const int w = (blockIdx.x * kThreads + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  if (w >= p.num_seqs * p.hq) return;
  const int b = w / p.hq;
  const int qh = w % p.hq;
  constexpr int kPer = D / 64;
  float* orow = p.out + static_cast<int64_t>(w) * D;
  const int L = p.seq_lens[b];
  int64_t base;
  int n;
  if (p.slot_base) {
    base = p.slot_base[b];
    n = p.slot_base[b + 1] - p.slot_base[b];
  } else {
    base = static_cast<int64_t>(b) * p.paged_nsplit;
    n = p.paged_nsplit;
  }
  bool stale = p.tail_lblock && L < p.tail_lblock[b] * p.block_size;
  float mx = kNegInf;
  bool nan = stale;
  for (int k = 0; k < n; ++k) {
    const float mk = p.part_ml[((base + k) * p.hq + qh) * 2];
    nan |= (mk != mk);
    mx = fmaxf(mx, mk);
  }
  float acc[kPer];
#pragma unroll
  for (int i = 0; i < kPer; ++i) acc[i] = 0.f;
  float l = 0.f;
  if (!nan && mx != kNegInf && L > 0) {
    for (int k = 0; k < n; ++k) {
      const int64_t r = (base + k) * p.hq + qh;
      const float f = exp2f(p.part_ml[r * 2] - mx);
      l += p.part_ml[r * 2 + 1] * f;
#pragma unroll
      for (int i = 0; i < kPer; ++i) acc[i] += p.part_o[r * D + lane * kPer + i] * f;
    }
  }
  const float inv = (l > 0.f) ? 1.f / l : 0.f;
#pragma unroll
  for (int i = 0; i < kPer; ++i) orow[lane * kPer + i] = nan ? __builtin_nanf("") : acc[i] * inv;
}

template <int D, int KV>
static hipError_t launch_attn_t(const AttnParams& p, int num_units, hipStream_t stream) {
  using G = Geo<D, KV>;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_units_kernel<D, KV>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, G::lds_bytes);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((attn_units_kernel<D, KV>), dim3(num_units), dim3(kThreads), G::lds_bytes, stream, p);
  return hipGetLastError();
}

hipError_t launch_attn_units(const AttnParams& p, int num_units, int head_dim, int kv_kind, hipStream_t stream) {
  if (num_units <= 0) return hipSuccess;
  if (head_dim == 128) {
    if (kv_kind == kKvBf16) return launch_attn_t<128, kKvBf16>(p, num_units, stream);
    if (kv_kind == kKvFp8) return launch_attn_t<128, kKvFp8>(p, num_units, stream);
    return launch_attn_t<128, kKvF32>(p, num_units, stream);
  }
  if (kv_kind == kKvBf16) return launch_attn_t<64, kKvBf16>(p, num_units, stream);
  if (kv_kind == kKvFp8) return launch_attn_t<64, kKvFp8>(p, num_units, stream);
  return launch_attn_t<64, kKvF32>(p, num_units, stream);
}

hipError_t launch_merge(const MergeParams& p, int head_dim, hipStream_t stream) {
  const int waves = p.num_seqs * p.hq;
  if (waves <= 0) return hipSuccess;
  const int blocks = (waves * 64 + kThreads - 1) / kThreads;
  if (head_dim == 128)
    hipLaunchKernelGGL((merge_kernel<128>), dim3(blocks), dim3(kThreads), 0, stream, p);
  else
    hipLaunchKernelGGL((merge_kernel<64>), dim3(blocks), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace tts
