// HIP kernels (gfx950) for prefix-shared beam decode attention.
//
// One kernel processes "work units" (tts_work.h): the query rows of up to
// 64 / g whole beams for one KV head against a run of KV blocks.
//
// Products on MFMA, two 16-token blocks ("a pair") at a time:
//   S^T = K Q^T   : 2 x v_mfma_f32_16x16x32_bf16 per 32-dim slice
//                   (M = 16 tokens, N = 16 query rows, K = head dim)
//   O^T += V^T P^T: 1 x v_mfma_f32_16x16x32_bf16 per 16 output dims
//                   (M = 16 dims, N = 16 rows, K = the pair's 32 tokens)
// The two S tiles of a pair take their 16 token rows in an interleaved
// order (tile t, row m -> token 8*(m/4) + 4*t + m%4), so after the first
// product every lane holds the scores of 8 consecutive tokens of one row:
// exactly the B operand the second product needs, with no data movement.
// Values are stored dim-major inside a block, so the matching A operand is
// one contiguous 16-byte read.
//
// Softmax is online with a lazy reference maximum: probabilities are
// exp2(s - m_ref) and O/l are rescaled only when some score exceeds m_ref
// by more than kRescale (a wave vote decides), which keeps the common path
// free of cross-lane reductions and accumulator rescaling.
//
// Units with more than 16 rows stage each chunk of K/V blocks in LDS once
// and every wave (16 rows each) reads it; units with at most 16 rows (a
// private tail, a two-beam segment) let each wave stream its own block
// pairs straight into registers. Partial softmax states go to the
// workspace, and a second kernel merges each (beam, query head)'s partial
// states in a fixed order (deterministic).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "tts_work.h"

namespace tts {

#ifdef TTS_PROFILE_UNITS
// Per-unit timestamps for tuning builds only: start, end of the block loop,
// end, and the XCC / HW_ID registers of the workgroup.
constexpr int kProfSlots = 1 << 16;
__device__ uint64_t g_prof[kProfSlots][4];
#define TTS_PROF_MARK(k) \
  do { if (threadIdx.x == 0 && blockIdx.x < kProfSlots) g_prof[blockIdx.x][k] = wall_clock64(); } while (0)
#else
#define TTS_PROF_MARK(k) do {} while (0)
#endif

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kTok = 16;  // tokens per KV block
constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr float kNegInf = -__builtin_inff();
constexpr float kRescale = 8.0f;  // log2 headroom before O and l are rescaled

enum KvKind : int { kKvF32 = 0, kKvBf16 = 1, kKvFp8 = 2 };

template <int KV>
struct KvBytes {
  static constexpr int value = KV == kKvF32 ? 4 : (KV == kKvBf16 ? 2 : 1);
};

template <int D, int KV>
struct Geo {
  static constexpr int eb = KvBytes<KV>::value;
  static constexpr int row_bytes = D * eb;            // one token of K
  static constexpr int c16 = row_bytes / 16;           // 16-byte columns per K row
  static constexpr int blk_bytes = kTok * row_bytes;   // one (block, head) of K or V
  static constexpr int vrow_bytes = kTok * eb;         // one dim of V (16 tokens)
  // LDS stages of one block pair (K0, V0, K1, V1) for the staged path:
  // four when a stage is at most 16 KB, else two.
  static constexpr int stage_bytes = 4 * blk_bytes;
  static constexpr int stages = stage_bytes <= 16384 ? 4 : 2;
  static constexpr int dma_per_wave = blk_bytes / 1024;  // 1-KB wave loads per tensor
  // Per-wave softmax state exchanged at the end: 16 rows of D floats padded
  // by 4 (bank spread) plus m and l; it reuses a stage.
  static constexpr int combine_bytes = (kTok * (D + 4) + 2 * kTok) * 4;
  static constexpr int stage_alloc = stage_bytes > combine_bytes ? stage_bytes : combine_bytes;
  static_assert(blk_bytes % 1024 == 0, "whole 1-KB wave loads");
};

__device__ __forceinline__ uint32_t f32_bits(float x) { return __builtin_bit_cast(uint32_t, x); }

// Two OCP E4M3 codes (byte pair kHi of w) -> two bf16 in one dword. The
// conversion to fp32 is exact and every E4M3 value fits bf16 exactly, so
// dropping the low half of the fp32 pattern is exact too.
template <bool kHi>
__device__ __forceinline__ uint32_t fp8x2_to_bf16x2(uint32_t w) {
  f32x2 f = __builtin_amdgcn_cvt_pk_f32_fp8(w, kHi);
  return (f32_bits(f.x) >> 16) | (f32_bits(f.y) & 0xFFFF0000u);
}

__device__ __forceinline__ uint4 fp8x8_to_bf16x8(uint2 w) {
  return uint4{fp8x2_to_bf16x2<false>(w.x), fp8x2_to_bf16x2<true>(w.x), fp8x2_to_bf16x2<false>(w.y),
               fp8x2_to_bf16x2<true>(w.y)};
}

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, bf16x2));  // RNE
}

__device__ __forceinline__ float xlane_max16(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  return fmaxf(x, __shfl_xor(x, 32));
}
__device__ __forceinline__ float xlane_sum16(float x) {
  x += __shfl_xor(x, 16);
  return x + __shfl_xor(x, 32);
}

// Per-lane operands of one block pair: K fragments of the two S tiles and
// V^T fragments of every 16-dim slice (bf16 compute: bf16 bits; f32
// compute: raw floats).
template <int D, int KV>
struct PairFrags {
  static constexpr bool f32 = KV == kKvF32;
  static constexpr int kk = f32 ? D / 16 : D / 32;  // K-fragment slices per tile
  typedef typename std::conditional<f32, f32x4, uint4>::type KF;
  KF k[2][kk];
  // V^T: lane (d = 16*dt + ln, tokens 8*lq .. 8*lq+7)
  typedef typename std::conditional<f32, f32x4, uint4>::type VF;
  VF v[D / 16][f32 ? 2 : 1];
};

// Softmax state of one wave's 16 rows (lane ln = row, lq = token group).
template <int D>
struct RowState {
  f32x4 o[D / 16];
  float m;  // reference max (log2 units), uniform over the 4 lanes of a row
  float l;  // per-lane partial sum
};

template <int D, int KV>
__device__ __forceinline__ void pair_step(const PairFrags<D, KV>& f, const void* qf_, RowState<D>& st, int lq,
                                          float sc0, float sc1, float vs0, float vs1, int valid0, int valid1,
                                          bool masked) {
  using F = PairFrags<D, KV>;
  f32x4 acc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
  if constexpr (F::f32) {
    const f32x4* qf = static_cast<const f32x4*>(qf_);
#pragma unroll
    for (int j = 0; j < F::kk; ++j) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(f.k[t][j].x, qf[j].x, acc[t], 0, 0, 0);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(f.k[t][j].y, qf[j].y, acc[t], 0, 0, 0);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(f.k[t][j].z, qf[j].z, acc[t], 0, 0, 0);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(f.k[t][j].w, qf[j].w, acc[t], 0, 0, 0);
      }
    }
  } else {
    const uint4* qf = static_cast<const uint4*>(qf_);
#pragma unroll
    for (int j = 0; j < F::kk; ++j) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, f.k[t][j]),
                                                         __builtin_bit_cast(bf16x8, qf[j]), acc[t], 0, 0, 0);
    }
  }
  // Lane (ln, lq) holds row ln, tokens 8*lq + 4*t + i of the pair; they all
  // lie in block lq >> 1 of the pair, at slots 8*(lq & 1) + 4*t + i.
  // bf16/fp32 scores stay unscaled (their scale is positive, so it
  // preserves the maximum) and the scale is applied inside the exponent:
  // p = 2^(acc * sc - m).
  const bool hi = lq >= 2;
  const float sc = hi ? sc1 : sc0;
  // fp8 block scales are caller data (any sign): scale first there.
  constexpr bool kPreScale = KV == kKvFp8;
  float s[8];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) s[4 * t + i] = kPreScale ? acc[t][i] * sc : acc[t][i];
  if (masked) {
    const int valid = hi ? valid1 : valid0;
    const int slot0 = 8 * (lq & 1);
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (slot0 + 4 * t + i >= valid) s[4 * t + i] = kNegInf;
  }
  float smax = fmaxf(fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3])), fmaxf(fmaxf(s[4], s[5]), fmaxf(s[6], s[7])));
  const float lm = kPreScale ? smax : smax * sc;  // largest scaled score of this lane (-inf if all masked)
  if (__builtin_amdgcn_ballot_w64(lm > st.m + kRescale) != 0) {
    // Rare: move the reference maximum up for every row of the wave.
    const float rmax = xlane_max16(lm);
    const float m_new = fmaxf(st.m, rmax);
    const float alpha = (st.m == kNegInf) ? 0.f : __builtin_amdgcn_exp2f(st.m - m_new);
    st.l *= alpha;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) st.o[dt] *= alpha;
    st.m = m_new;
  }
  const float mu = (st.m == kNegInf) ? 0.f : st.m;
  float p[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) p[i] = __builtin_amdgcn_exp2f(kPreScale ? s[i] - mu : __builtin_fmaf(s[i], sc, -mu));
  st.l += ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
  if constexpr (F::f32) {
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) {
      const f32x4 a0 = f.v[dt][0], a1 = f.v[dt][1];
      f32x4 o = st.o[dt];
      o = __builtin_amdgcn_mfma_f32_16x16x4f32(a0.x, p[0], o, 0, 0, 0);
      o = __builtin_amdgcn_mfma_f32_16x16x4f32(a0.y, p[1], o, 0, 0, 0);
      o = __builtin_amdgcn_mfma_f32_16x16x4f32(a0.z, p[2], o, 0, 0, 0);
      o = __builtin_amdgcn_mfma_f32_16x16x4f32(a0.w, p[3], o, 0, 0, 0);
      o = __builtin_amdgcn_mfma_f32_16x16x4f32(a1.x, p[4], o, 0, 0, 0);
      o = __builtin_amdgcn_mfma_f32_16x16x4f32(a1.y, p[5], o, 0, 0, 0);
      o = __builtin_amdgcn_mfma_f32_16x16x4f32(a1.z, p[6], o, 0, 0, 0);
      o = __builtin_amdgcn_mfma_f32_16x16x4f32(a1.w, p[7], o, 0, 0, 0);
      st.o[dt] = o;
    }
  } else {
    float pv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) pv[i] = (KV == kKvFp8) ? p[i] * (hi ? vs1 : vs0) : p[i];
    const uint4 pb = {pack_bf16x2(pv[0], pv[1]), pack_bf16x2(pv[2], pv[3]), pack_bf16x2(pv[4], pv[5]),
                      pack_bf16x2(pv[6], pv[7])};
    const bf16x8 pbf = __builtin_bit_cast(bf16x8, pb);
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt)
      st.o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, f.v[dt][0]), pbf, st.o[dt], 0,
                                                        0, 0);
  }
}

// LDS swizzles of the staged path (bank-conflict-free fragment reads).
// K: an S tile reads rows {0-3, 8-11} or {4-7, 12-15} of both blocks of a
// pair, so the 16-byte column of (block b, row r) is XORed with
// (r & 3) | ((r >> 3) & 1) << 2 | b << 3 (cut to the columns a row has).
// V^T: lanes read 16 consecutive dims at a 32-byte stride; the two 16-byte
// halves of a dim row swap on odd groups of 8 dims.
template <int C16>
__device__ __forceinline__ int k_swz(int b, int r) {
  return ((r & 3) | (((r >> 3) & 1) << 2) | (b << 3)) & (C16 - 1);
}
__device__ __forceinline__ int v_half_swz(int d) { return (d >> 3) & 1; }

// Token row of S tile t, MFMA row m inside a pair (see the header).
__device__ __forceinline__ int pair_token(int t, int m) { return ((m >> 2) << 3) + (t << 2) + (m & 3); }

// K fragments of one pair straight from global memory.
template <int D, int KV>
__device__ __forceinline__ void load_k_global(PairFrags<D, KV>& f, const unsigned char* kb0,
                                              const unsigned char* kb1, int ln, int lq) {
  using G = Geo<D, KV>;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int tok = pair_token(t, ln);
    const unsigned char* kr = (tok < 16 ? kb0 : kb1) + (tok & 15) * G::row_bytes;
#pragma unroll
    for (int j = 0; j < PairFrags<D, KV>::kk; ++j) {
      if constexpr (KV == kKvF32) {
        f.k[t][j] = *reinterpret_cast<const f32x4*>(kr + (4 * j + lq) * 16);
      } else if constexpr (KV == kKvBf16) {
        f.k[t][j] = *reinterpret_cast<const uint4*>(kr + (4 * j + lq) * 16);
      } else {
        f.k[t][j] = fp8x8_to_bf16x8(*reinterpret_cast<const uint2*>(kr + 32 * j + 8 * lq));
      }
    }
  }
}

// V^T fragments of one pair (lane: dim 16*dt + ln, tokens 8*lq .. 8*lq+7)
// from two blocks laid out dim-major; works for global memory and LDS.
template <int D, int KV>
__device__ __forceinline__ void load_v(PairFrags<D, KV>& f, const unsigned char* vb0, const unsigned char* vb1, int ln,
                                       int lq) {
  using G = Geo<D, KV>;
  const unsigned char* vb = (lq >= 2 ? vb1 : vb0) + (lq & 1) * 8 * G::eb + ln * G::vrow_bytes;
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    const unsigned char* vr = vb + 16 * dt * G::vrow_bytes;
    if constexpr (KV == kKvF32) {
      f.v[dt][0] = *reinterpret_cast<const f32x4*>(vr);
      f.v[dt][1] = *reinterpret_cast<const f32x4*>(vr + 16);
    } else if constexpr (KV == kKvBf16) {
      f.v[dt][0] = *reinterpret_cast<const uint4*>(vr);
    } else {
      f.v[dt][0] = fp8x8_to_bf16x8(*reinterpret_cast<const uint2*>(vr));
    }
  }
}

// LDS fragment reads of the staged path are written as inline asm: the
// compiler's wait insertion cannot tell which stage an in-flight
// global-to-LDS copy targets once the read sits behind a branch, and would
// otherwise drain every copy before each read. lds_ready() then waits for
// this wave's LDS reads and ties each value to that wait, so no use can be
// scheduled before it.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) void*)(p)));
}
__device__ __forceinline__ u32x4 lds_rd128(const unsigned char* p) {
  u32x4 v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(lds_addr(p)) : "memory");
  return v;
}
__device__ __forceinline__ u32x2 lds_rd64(const unsigned char* p) {
  u32x2 v;
  asm volatile("ds_read_b64 %0, %1" : "=v"(v) : "v"(lds_addr(p)) : "memory");
  return v;
}
__device__ __forceinline__ void lds_wait_all() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
template <typename T>
__device__ __forceinline__ void lds_tie(T& v) { asm volatile("" : "+v"(v)); }

// V^T fragments of one pair from an LDS stage (bf16: halves swizzled).
// K and V^T fragments of one pair from an LDS stage (K rows XOR-swizzled,
// bf16 V^T halves swizzled; see k_swz / v_half_swz).
template <int D, int KV>
__device__ __forceinline__ void load_pair_lds(PairFrags<D, KV>& f, const unsigned char* k0, const unsigned char* k1,
                                              const unsigned char* v0, const unsigned char* v1, int ln, int lq) {
  using G = Geo<D, KV>;
  constexpr int kk = PairFrags<D, KV>::kk;
  constexpr bool wide = KV != kKvFp8;  // 16-byte reads (fp8: 8 bytes)
  typedef typename std::conditional<wide, u32x4, u32x2>::type R;
  R rk[2][kk];
  R rv[D / 16][KV == kKvF32 ? 2 : 1];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int tok = pair_token(t, ln);
    const int r = tok & 15;
    const unsigned char* kr = (tok < 16 ? k0 : k1) + r * G::row_bytes;
    const int sw = k_swz<G::c16>(tok >> 4, r);
#pragma unroll
    for (int j = 0; j < kk; ++j) {
      if constexpr (wide) {
        rk[t][j] = lds_rd128(kr + (((4 * j + lq) ^ sw) << 4));
      } else {
        const int col = 2 * j + (lq >> 1);
        rk[t][j] = lds_rd64(kr + ((col ^ sw) << 4) + 8 * (lq & 1));
      }
    }
  }
  const unsigned char* vb = lq >= 2 ? v1 : v0;
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    const int d = 16 * dt + ln;
    if constexpr (KV == kKvBf16) {
      rv[dt][0] = lds_rd128(vb + d * G::vrow_bytes + 16 * ((lq & 1) ^ v_half_swz(d)));
    } else if constexpr (KV == kKvF32) {
      const unsigned char* vr = vb + d * G::vrow_bytes + (lq & 1) * 32;
      rv[dt][0] = lds_rd128(vr);
      rv[dt][1] = lds_rd128(vr + 16);
    } else {
      rv[dt][0] = lds_rd64(vb + d * G::vrow_bytes + (lq & 1) * 8);
    }
  }
  lds_wait_all();
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int j = 0; j < kk; ++j) lds_tie(rk[t][j]);
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt)
#pragma unroll
    for (int h = 0; h < (KV == kKvF32 ? 2 : 1); ++h) lds_tie(rv[dt][h]);
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int j = 0; j < kk; ++j) {
      if constexpr (KV == kKvF32) {
        f.k[t][j] = __builtin_bit_cast(f32x4, rk[t][j]);
      } else if constexpr (KV == kKvBf16) {
        f.k[t][j] = __builtin_bit_cast(uint4, rk[t][j]);
      } else {
        f.k[t][j] = fp8x8_to_bf16x8(__builtin_bit_cast(uint2, rk[t][j]));
      }
    }
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    if constexpr (KV == kKvF32) {
      f.v[dt][0] = __builtin_bit_cast(f32x4, rv[dt][0]);
      f.v[dt][1] = __builtin_bit_cast(f32x4, rv[dt][1]);
    } else if constexpr (KV == kKvBf16) {
      f.v[dt][0] = __builtin_bit_cast(uint4, rv[dt][0]);
    } else {
      f.v[dt][0] = fp8x8_to_bf16x8(__builtin_bit_cast(uint2, rv[dt][0]));
    }
  }
}

// Zero the V^T fragments of tokens past `valid` in this lane's block, so
// unused slots of a partial block never reach the value product.
template <int D, int KV>
__device__ __forceinline__ void mask_v(PairFrags<D, KV>& f, int lq, int valid0, int valid1) {
  const int valid = lq >= 2 ? valid1 : valid0;
  const int slot0 = 8 * (lq & 1);
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    if constexpr (KV == kKvF32) {
      float* a = reinterpret_cast<float*>(&f.v[dt][0]);
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (slot0 + e >= valid) a[e] = 0.f;
    } else {
      uint32_t* a = reinterpret_cast<uint32_t*>(&f.v[dt][0]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t keep =
            (slot0 + 2 * e < valid ? 0x0000FFFFu : 0u) | (slot0 + 2 * e + 1 < valid ? 0xFFFF0000u : 0u);
        a[e] &= keep;
      }
    }
  }
}

// Block run of one unit, resolved from the metadata or the live tables.
struct Run {
  const int32_t* ids;  // block ids (segment) or table row (tail)
  int32_t first;       // first index into ids
  int32_t nblk;        // blocks in this unit
  int32_t len;         // tail: beam length (last block may be partial)
  bool tail;
};

// Per-lane view of up to 64 consecutive blocks of a run: lane i holds the
// id, valid token count and (fp8) scales of block w0 + i; a wave reads any
// of them with a uniform index. Bad ids become valid = 0.
struct Window {
  int id, valid;
  float ks, vs;
};

template <int KV>
__device__ __forceinline__ Window load_window(const Run& run, int w0, int lane, const AttnParams& p, bool* bad) {
  Window w{-1, 0, 1.f, 1.f};
  const int i = w0 + lane;
  bool b = false;
  if (i < run.nblk) {
    int id = run.ids[run.first + i];
    int v = kTok;
    if (run.tail) {
      v = run.len - (run.first + i) * kTok;
      v = v < kTok ? v : kTok;
      if (id < 0 || id >= p.num_blocks) {
        b = true;
        id = -1;
        v = 0;
      }
    }
    w.id = id;
    w.valid = v;
    if constexpr (KV == kKvFp8) {
      if (id >= 0) {
        w.ks = p.k_scale[id];
        w.vs = p.v_scale[id];
      }
    }
  }
  if (__builtin_amdgcn_ballot_w64(b) != 0) *bad = true;
  return w;
}

// Workgroup barrier for the staged pipeline: LDS writes of this wave have
// completed, then s_barrier. Unlike __syncthreads() it does not wait for
// outstanding global loads (whose results are still travelling to their
// registers), which is what keeps several pairs in flight across it.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ __forceinline__ int rl(int x, int i) { return __builtin_amdgcn_readlane(x, i); }
__device__ __forceinline__ float rlf(float x, int i) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), i));
}

template <int D, int KV>
__global__ __launch_bounds__(kThreads, 2) void attn_units_kernel(AttnParams p) {
  using G = Geo<D, KV>;
  using F = PairFrags<D, KV>;
  // Four distinct LDS stages (the last two are stubs when only two are used).
  __shared__ __attribute__((aligned(16))) unsigned char lds_s0[G::stage_alloc];
  __shared__ __attribute__((aligned(16))) unsigned char lds_s1[G::stage_alloc];
  __shared__ __attribute__((aligned(16))) unsigned char lds_s2[G::stages > 2 ? G::stage_alloc : 16];
  __shared__ __attribute__((aligned(16))) unsigned char lds_s3[G::stages > 3 ? G::stage_alloc : 16];
  // Stage i (i is a compile-time constant wherever this is used).
  auto stage_of = [&](int i) -> unsigned char* {
    return i == 0 ? lds_s0 : (i == 1 ? lds_s1 : (i == 2 ? lds_s2 : lds_s3));
  };

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int ln = lane & 15;
  const int lq = lane >> 4;

  TTS_PROF_MARK(0);
  // ---- the unit ----------------------------------------------------------
  Unit u;
  if (p.units) {
    u = p.units[blockIdx.x];
    if (u.nrows <= 0) return;  // padding unit
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
  bool bad = false;
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
      bad = true;
      nb_all = t0;
    }
    const int tb = nb_all - t0;
    // Splits cover whole pairs so only a sequence's last pair is ragged.
    const int npairs = (tb + 1) >> 1;
    const int per = 2 * ((npairs + u.nblk - 1) / u.nblk);
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
  const int wt = kWaves / wr;         // waves splitting block pairs
  const int rt = wave % wr;
  const int tl = wave / wr;
  const int rloc = rt * 16 + ln;
  const bool row_ok = rloc < u.nrows;
  const bool wave_active = rt * 16 < u.nrows;
  int beam, qh;
  {
    const int r = u.row0 + (row_ok ? rloc : 0);
    const int pos = u.pos0 + r / p.g;
    beam = p.perm ? p.perm[pos] : pos;
    qh = u.kvh * p.g + r % p.g;
  }

  // ---- query fragments (B operand of S^T = K Q^T) ------------------------
  typename F::KF qf[F::kk];
  if constexpr (KV == kKvF32) {
    const float* qrow = static_cast<const float*>(p.q) + (static_cast<int64_t>(beam) * p.hq + qh) * D;
#pragma unroll
    for (int j = 0; j < F::kk; ++j)
      qf[j] = row_ok ? *reinterpret_cast<const f32x4*>(qrow + 16 * j + 4 * lq) : f32x4{0.f, 0.f, 0.f, 0.f};
  } else {
    const uint16_t* qrow = static_cast<const uint16_t*>(p.q) + (static_cast<int64_t>(beam) * p.hq + qh) * D;
#pragma unroll
    for (int j = 0; j < F::kk; ++j)
      qf[j] = row_ok ? *reinterpret_cast<const uint4*>(qrow + 32 * j + 8 * lq) : uint4{0u, 0u, 0u, 0u};
  }

  RowState<D> st;
#pragma unroll
  for (int i = 0; i < D / 16; ++i) st.o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  st.m = kNegInf;
  st.l = 0.f;

  const size_t kv_blk_stride = static_cast<size_t>(p.hkv) * G::blk_bytes;
  const unsigned char* kbase_g = static_cast<const unsigned char*>(p.k_cache) + u.kvh * G::blk_bytes;
  const unsigned char* vbase_g = static_cast<const unsigned char*>(p.v_cache) + u.kvh * G::blk_bytes;
  const float sc_log2 = p.scale_log2;

  if (nrt == 1) {
    // ---- direct path: each wave streams its own block pairs -------------
    for (int w0 = 0; w0 < run.nblk; w0 += 64) {
      const Window win = load_window<KV>(run, w0, lane, p, &bad);
      const int nw = (run.nblk - w0) < 64 ? (run.nblk - w0) : 64;
      const int npairs = (nw + 1) >> 1;
      for (int pp = tl; pp < npairs; pp += wt) {
        const int i0 = 2 * pp, i1 = 2 * pp + 1;
        const int v0 = rl(win.valid, i0);
        const int v1 = i1 < nw ? rl(win.valid, i1) : 0;
        if (v0 <= 0 && v1 <= 0) continue;
        const int id0 = rl(win.id, i0);
        const int id1 = i1 < nw ? rl(win.id, i1) : -1;
        // A missing or bad block re-reads a valid one and is fully masked.
        const int r0 = v0 > 0 ? id0 : id1;
        const int r1 = v1 > 0 ? id1 : r0;
        F f;
        load_k_global<D, KV>(f, kbase_g + r0 * kv_blk_stride, kbase_g + r1 * kv_blk_stride, ln, lq);
        load_v<D, KV>(f, vbase_g + r0 * kv_blk_stride, vbase_g + r1 * kv_blk_stride, ln, lq);
        float ks0 = 1.f, ks1 = 1.f, vs0 = 1.f, vs1 = 1.f;
        if constexpr (KV == kKvFp8) {
          ks0 = rlf(win.ks, v0 > 0 ? i0 : i1);
          vs0 = rlf(win.vs, v0 > 0 ? i0 : i1);
          ks1 = v1 > 0 ? rlf(win.ks, i1) : ks0;
          vs1 = v1 > 0 ? rlf(win.vs, i1) : vs0;
        }
        const bool masked = v0 < kTok || v1 < kTok;
        if (masked) mask_v<D, KV>(f, lq, v0, v1);
        pair_step<D, KV>(f, qf, st, lq, sc_log2 * ks0, sc_log2 * ks1, vs0, vs1, v0, v1, masked);
      }
    }
  } else {
    // ---- staged path: pairs land in LDS, every wave reads them -----------
    // Each stage holds K0, V0, K1, V1 of one pair; wave w copies tensor w
    // straight from global memory into LDS (no registers). The stages are
    // distinct LDS objects indexed at compile time so that the compiler does
    // not make reads of one stage wait for copies into another; kStages - 2
    // pairs stay in flight across each barrier.
    constexpr int kStages = G::stages;
    constexpr int kDma = G::dma_per_wave;
    const bool is_v = wave & 1;
    const int blk_sel = wave >> 1;
    for (int w0 = 0; w0 < run.nblk; w0 += 64) {
      const Window win = load_window<KV>(run, w0, lane, p, &bad);
      __builtin_amdgcn_s_waitcnt(0x0F70);  // window and query loads done
      const int nw = (run.nblk - w0) < 64 ? (run.nblk - w0) : 64;
      const int npairs = (nw + 1) >> 1;
      // Any valid block of the window stands in for invalid ones (loaded, never used).
      const uint64_t any_valid = __builtin_amdgcn_ballot_w64(lane < nw && win.valid > 0);
      if (any_valid == 0) continue;  // uniform: nothing to read in this window
      const int fill_id = rl(win.id, static_cast<int>(__builtin_ctzll(any_valid)));
      auto pair_ids = [&](int pp, int* r0, int* r1, int* v0, int* v1) {
        const int i0 = 2 * pp, i1 = 2 * pp + 1;
        *v0 = rl(win.valid, i0);
        *v1 = i1 < nw ? rl(win.valid, i1) : 0;
        const int id0 = rl(win.id, i0);
        const int id1 = i1 < nw ? rl(win.id, i1) : -1;
        *r0 = *v0 > 0 ? id0 : (*v1 > 0 ? id1 : fill_id);
        *r1 = *v1 > 0 ? id1 : *r0;
      };
      // Copy pair pp (clamped to the window) into stage `dst`: always exactly
      // kDma loads per wave, so the wait counts below are constants.
      auto issue = [&](int pp, unsigned char* dst) {
        pp = pp < npairs ? pp : npairs - 1;
        int r0, r1, v0, v1;
        pair_ids(pp, &r0, &r1, &v0, &v1);
        const int rid = blk_sel ? r1 : r0;
        const unsigned char* src = (is_v ? vbase_g : kbase_g) + static_cast<size_t>(rid) * kv_blk_stride;
        unsigned char* d = dst + wave * G::blk_bytes;
#pragma unroll
        for (int j = 0; j < kDma; ++j) {
          const int pos = j * 64 + lane;  // 16-byte slot of this lane in the tensor
          int off;
          if (!is_v) {
            const int r = pos / G::c16;
            off = r * G::row_bytes + (((pos % G::c16) ^ k_swz<G::c16>(blk_sel, r)) << 4);
          } else if constexpr (KV == kKvBf16) {
            const int dd = pos >> 1;
            off = dd * G::vrow_bytes + 16 * ((pos & 1) ^ v_half_swz(dd));
          } else {
            off = pos * 16;
          }
          __builtin_amdgcn_global_load_lds(src + off, (__attribute__((address_space(3))) void*)(d + j * 1024),
                                           16, 0, 0);
        }
      };
      auto consume = [&](int pp, const unsigned char* stage) {
        int r0, r1, v0, v1;
        pair_ids(pp, &r0, &r1, &v0, &v1);
        if (!wave_active || (pp % wt) != tl || (v0 <= 0 && v1 <= 0)) return;
        F f;
        load_pair_lds<D, KV>(f, stage, stage + 2 * G::blk_bytes, stage + G::blk_bytes, stage + 3 * G::blk_bytes, ln,
                             lq);
        float ks0 = 1.f, ks1 = 1.f, vs0 = 1.f, vs1 = 1.f;
        if constexpr (KV == kKvFp8) {
          const int i0 = 2 * pp, i1 = 2 * pp + 1;
          ks0 = rlf(win.ks, v0 > 0 ? i0 : i1);
          vs0 = rlf(win.vs, v0 > 0 ? i0 : i1);
          ks1 = v1 > 0 ? rlf(win.ks, i1) : ks0;
          vs1 = v1 > 0 ? rlf(win.vs, i1) : vs0;
        }
        const bool masked = v0 < kTok || v1 < kTok;
        if (masked) mask_v<D, KV>(f, lq, v0, v1);
        pair_step<D, KV>(f, qf, st, lq, sc_log2 * ks0, sc_log2 * ks1, vs0, vs1, v0, v1, masked);
      };
#pragma unroll
      for (int j = 0; j < kStages - 1; ++j) issue(j, stage_of(j));
      for (int p0 = 0; p0 < npairs; p0 += kStages) {
#pragma unroll
        for (int s = 0; s < kStages; ++s) {
          const int pp = p0 + s;
          if (pp < npairs) {
            // Pairs pp + 1 .. pp + kStages - 2 may still be in flight.
            __builtin_amdgcn_s_waitcnt(0x0F70 | (((kStages - 2) * kDma) & 15) | ((((kStages - 2) * kDma) >> 4) << 14));
            lds_barrier();
            issue(pp + kStages - 1, stage_of((s + kStages - 1) % kStages));
            consume(pp, stage_of(s));
          }
        }
      }
      __builtin_amdgcn_s_waitcnt(0x0F70);  // the clamped trailing copies
      __syncthreads();                      // every wave is done with the stages
    }
  }

  TTS_PROF_MARK(1);
  // A bad block id may have been seen by one wave only.
  bad = __syncthreads_or(bad ? 1 : 0) != 0;

  // ---- combine the waves that split block pairs --------------------------
  float l_tot = xlane_sum16(st.l);
  float m_fin = st.m;
  if (wt > 1) {
    // Waves 1..3 of a row tile publish their state in stages 0..2 (wt >= 2
    // means at most two row tiles: slot = (tl - 1) * wr + rt < 3).
    static_assert(G::stages > 2 || G::stage_alloc >= 2 * G::combine_bytes, "third combine slot");
    auto region = [&](int t) {
      const int slot = (t - 1) * wr + rt;
      unsigned char* c = slot == 0 ? lds_s0 : (slot == 1 ? lds_s1 : (G::stages > 2 ? lds_s2 : lds_s0 + G::combine_bytes));
      return reinterpret_cast<float*>(c);
    };
    float* my = tl > 0 ? region(tl) : nullptr;
    // Rows are padded by 4 floats so the 16 lanes of a column hit distinct banks.
    constexpr int kRow = D + 4;
    if (tl > 0 && wave_active) {
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) *reinterpret_cast<f32x4*>(my + ln * kRow + 16 * dt + 4 * lq) = st.o[dt];
      if (lq == 0) {
        my[kTok * kRow + ln] = st.m;
        my[kTok * kRow + kTok + ln] = l_tot;
      }
    }
    __syncthreads();
    if (tl == 0 && wave_active) {
      float mt[kWaves];
      float mx = st.m;
      mt[0] = st.m;
      for (int t = 1; t < wt; ++t) {
        mt[t] = region(t)[kTok * kRow + ln];
        mx = fmaxf(mx, mt[t]);
      }
      const float mu = (mx == kNegInf) ? 0.f : mx;
      const float f0 = (mt[0] == kNegInf) ? 0.f : __builtin_amdgcn_exp2f(mt[0] - mu);
      l_tot *= f0;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) st.o[dt] *= f0;
      for (int t = 1; t < wt; ++t) {
        const float* ot = region(t);
        const float fct = (mt[t] == kNegInf) ? 0.f : __builtin_amdgcn_exp2f(mt[t] - mu);
        l_tot += ot[kTok * kRow + kTok + ln] * fct;
#pragma unroll
        for (int dt = 0; dt < D / 16; ++dt)
          st.o[dt] += *reinterpret_cast<const f32x4*>(ot + ln * kRow + 16 * dt + 4 * lq) * fct;
      }
      m_fin = mx;
    }
  }
  if (bad) m_fin = __builtin_nanf("");

  // ---- write ---------------------------------------------------------------
  const bool writer = tl == 0 && row_ok;
  if (!p.units && p.paged_nsplit == 1) {
    // Whole sequence in this unit: write the normalised result.
    if (writer) {
      float* orow = p.out + (static_cast<int64_t>(beam) * p.hq + qh) * D;
      const float inv = (l_tot > 0.f) ? 1.f / l_tot : 0.f;
      const bool nan = m_fin != m_fin;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        f32x4 v = st.o[dt] * inv;
        if (nan) v = f32x4{m_fin, m_fin, m_fin, m_fin};
        *reinterpret_cast<f32x4*>(orow + 16 * dt + 4 * lq) = v;
      }
    }
    return;
  }
  if (writer) {
    int64_t prow;
    if (p.units)
      prow = static_cast<int64_t>(p.slot_base[beam] + u.slot) * p.hq + qh;
    else
      prow = (static_cast<int64_t>(beam) * p.paged_nsplit + u.slot) * p.hq + qh;
    float* po = p.part_o + prow * D;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) *reinterpret_cast<f32x4*>(po + 16 * dt + 4 * lq) = st.o[dt];
    if (lq == 0) *reinterpret_cast<f32x2*>(p.part_ml + prow * 2) = f32x2{m_fin, l_tot};
  }
#ifdef TTS_PROFILE_UNITS
  if (threadIdx.x == 0 && blockIdx.x < kProfSlots)
    g_prof[blockIdx.x][3] = (static_cast<uint64_t>(__builtin_amdgcn_s_getreg((3 << 11) | 20)) << 32) |
                            static_cast<uint32_t>(__builtin_amdgcn_s_getreg((31 << 11) | 4));
#endif
  TTS_PROF_MARK(2);
}

// Exact merge of the partial softmax states of each (beam, query head), in
// slot order (segments root to leaf, then tail splits):
//   m = max_k m_k,  l = sum_k l_k 2^(m_k - m),  out = sum_k o_k 2^(m_k - m) / l.
// D/4 threads share a row (4 output dims each) and issue the loads of up to
// kBatch slots at once, so a row costs one round trip to memory per batch.
template <int D>
__global__ __launch_bounds__(kThreads) void merge_kernel(MergeParams p) {
  constexpr int kTpr = D / 4;
  constexpr int kRows = kThreads / kTpr;
  constexpr int kBatch = 16;
  const int r = blockIdx.x * kRows + threadIdx.x / kTpr;
  const int d0 = (threadIdx.x % kTpr) * 4;
  if (r >= p.num_seqs * p.hq) return;
  const int b = r / p.hq;
  const int h = r % p.hq;
  int64_t base;
  int n;
  if (p.slot_base) {
    base = p.slot_base[b];
    n = p.slot_base[b + 1] - p.slot_base[b];
  } else {
    base = static_cast<int64_t>(b) * p.paged_nsplit;
    n = p.paged_nsplit;
  }
  const int L = p.seq_lens[b];
  bool nan = p.tail_lblock && L < p.tail_lblock[b] * kTok;
  float mx = kNegInf, l = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < n; k0 += kBatch) {
    f32x2 ml[kBatch];
    f32x4 o[kBatch];
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const int kk = k0 + k < n ? k0 + k : n - 1;
      const int64_t row = (base + kk) * p.hq + h;
      ml[k] = *reinterpret_cast<const f32x2*>(p.part_ml + row * 2);
      o[k] = *reinterpret_cast<const f32x4*>(p.part_o + row * D + d0);
    }
#pragma unroll
    for (int k = 0; k < kBatch; ++k)
      if (k0 + k >= n) ml[k] = f32x2{kNegInf, 0.f};
    float bm = kNegInf;
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      nan |= ml[k].x != ml[k].x;
      bm = fmaxf(bm, ml[k].x);
    }
    const float mn = fmaxf(mx, bm);
    if (mn == kNegInf) continue;
    const float a = (mx == kNegInf) ? 0.f : __builtin_amdgcn_exp2f(mx - mn);
    l *= a;
    acc *= a;
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const float fct = (ml[k].x == kNegInf) ? 0.f : __builtin_amdgcn_exp2f(ml[k].x - mn);
      l += ml[k].y * fct;
      acc += o[k] * fct;
    }
    mx = mn;
  }
  const float inv = (l > 0.f && L > 0) ? 1.f / l : 0.f;
  f32x4 w = acc * inv;
  if (nan) {
    const float q = __builtin_nanf("");
    w = f32x4{q, q, q, q};
  }
  *reinterpret_cast<f32x4*>(p.out + static_cast<int64_t>(r) * D + d0) = w;
}

template <int D, int KV>
static hipError_t launch_attn_t(const AttnParams& p, int num_units, hipStream_t stream) {
  hipLaunchKernelGGL((attn_units_kernel<D, KV>), dim3(num_units), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_merge(const MergeParams& p, int head_dim, hipStream_t stream) {
  const int rows = p.num_seqs * p.hq;
  if (rows <= 0) return hipSuccess;
  const int per = kThreads / (head_dim / 4);
  const int blocks = (rows + per - 1) / per;
  if (head_dim == 128)
    hipLaunchKernelGGL((merge_kernel<128>), dim3(blocks), dim3(kThreads), 0, stream, p);
  else
    hipLaunchKernelGGL((merge_kernel<64>), dim3(blocks), dim3(kThreads), 0, stream, p);
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

}  // namespace tts

#ifdef TTS_PROFILE_UNITS
extern "C" int tts_prof_read(uint64_t* host, int n) {
  if (n > tts::kProfSlots) n = tts::kProfSlots;
  return static_cast<int>(hipMemcpyFromSymbol(host, HIP_SYMBOL(tts::g_prof), sizeof(uint64_t) * 4 * n, 0,
                                              hipMemcpyDeviceToHost));
}
extern "C" int tts_prof_clear() {
  static uint64_t zeros[tts::kProfSlots][4];
  return static_cast<int>(hipMemcpyToSymbol(HIP_SYMBOL(tts::g_prof), zeros, sizeof(zeros), 0, hipMemcpyHostToDevice));
}
#endif
