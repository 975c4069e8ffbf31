// HIP kernels (gfx950) for prefix-shared beam decode attention.
//
// attn_kernel: one workgroup (4 waves) per compute unit walks a chain of
// work units (tts_work.h), each the query rows of whole beams for one KV
// head against a list of KV blocks (up to 128, in two windows of 64).
//  * Narrow units (up to 64 rows, 4 row tiles of 16): every wave keeps the
//    softmax state of all of the unit's rows in registers and streams its
//    own share of the block pairs (pairs w, w + 4, ...) straight from HBM
//    into registers, one pair ahead of the one it computes; no LDS staging
//    and no barriers until the four waves combine their states.
//  * Wide units (a segment shared by many beams, up to 192 rows): each block
//    pair is loaded once, a quarter per wave, staged in LDS and read by all
//    four waves, each running its own row tiles.
//
// Products on MFMA, two 16-token blocks ("a pair") at a time, per row tile:
//   S^T = K Q^T   : 2 x 4 v_mfma_f32_16x16x32_bf16 (M = 16 tokens, N = 16
//                   rows, K = 128 head dims)
//   O^T += V^T P^T: 8 x v_mfma_f32_16x16x32_bf16 (M = 16 dims, N = 16 rows,
//                   K = the pair's 32 tokens)
// The two S tiles of a pair take their 16 token rows in an interleaved
// order (tile t, row m -> token 8*(m/4) + 4*t + m%4), so after the first
// product every lane holds the scores of 8 consecutive tokens of one row,
// all in one block of the pair: exactly the B operand of the second
// product. Values are stored dim-major inside a block, so the matching A
// operand is one contiguous 16-byte read.
//
// Softmax without a running maximum: probabilities are exp2(s - m_ref) with
// a fixed reference m_ref = 0 (log2 units), so the hot loop has no
// cross-lane reductions, no accumulator rescaling and no data-dependent
// branches. Each lane tracks the largest score it has seen; if a row's
// maximum leaves [-kRefWindow, kRefWindow] (where exp2 could overflow the
// fp32 accumulators or underflow every weight), its pairs are computed again
// with m_ref = that row's exact maximum: per wave in narrow units (no
// barrier inside their loop), by the whole workgroup in wide units (whose
// loop holds barriers, so the decision is taken over all four waves).
// Either way each row ends with a consistent (m_ref, l, o) triple; a state
// that saw no token (l = 0) carries m = -inf, so it never sets the maximum
// of a combine or a merge.
//
// Every unit writes one partial softmax state per row; merge_row_kernel or
// merge_kernel combines each (beam, query head)'s states in a fixed order
// (deterministic, no float atomics).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <type_traits>

#include "tts_work.h"

namespace tts {

#ifdef TTS_PROFILE_UNITS
// Per-unit timestamps for tuning builds only (indexed by record): start,
// end of wave 0's block loop, end, the XCC / HW_ID registers, all waves
// done, next unit issued, combine area written. (bf16 and fp8 kernels only:
// with the marks in the fp32 kernels too, the compiler's AGPR-copy rewrite
// pass crashes on the VGPR-form build.)
constexpr int kProfSlots = 1 << 15;
__device__ uint64_t g_prof[kProfSlots][8];
#define TTS_PROF_MARK(k, i) \
  do { if (KV != kKvF32 && threadIdx.x == 0 && (i) < kProfSlots) g_prof[(i)][k] = wall_clock64(); } while (0)
#else
#define TTS_PROF_MARK(k, i) do {} while (0)
#endif

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kTok = 16;  // tokens per KV block
constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kTiles = kMaxRows / 16;
constexpr int kWideTiles = kMaxWideRows / 16 / 4;  // row tiles per wave in a wide unit
constexpr float kNegInf = -__builtin_inff();
constexpr float kInf = __builtin_inff();
constexpr float kRefWindow = 64.0f;  // |row max| (log2 units) handled with m_ref = 0

enum KvKind : int { kKvF32 = 0, kKvBf16 = 1, kKvFp8 = 2 };

template <int KV>
struct KvBytes {
  static constexpr int value = KV == kKvF32 ? 4 : (KV == kKvBf16 ? 2 : 1);
};

template <int D, int KV>
struct Geo {
  static constexpr int eb = KvBytes<KV>::value;
  static constexpr int row_bytes = D * eb;           // one token of K
  static constexpr int blk_bytes = kTok * row_bytes;  // one (block, head) of K or V
  static constexpr int vrow_bytes = kTok * eb;        // one dim of V (16 tokens)
  // End-of-unit combine: per (wave, tile) 16 rows of D floats padded by 4
  // (bank spread), then m and l.
  static constexpr int comb_row = D + 4;
  static constexpr int comb_floats = kTok * comb_row + 2 * kTok;
};

__device__ __forceinline__ uint32_t f32_bits(float x) { return __builtin_bit_cast(uint32_t, x); }

// Two OCP E4M3 codes (byte pair kHi of w) -> two bf16 in one dword, in one
// conversion instruction with unit scale. Every E4M3 value fits bf16
// exactly, so the conversion is exact.
template <bool kHi>
__device__ __forceinline__ uint32_t fp8x2_to_bf16x2(uint32_t w) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, kHi));
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

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

// A row's partial state: m, l, the output row and its factor z, with
// (stored element) x z = o / l. For bf16 and fp8 caches the elements are o
// scaled by a power of two, 2^-e, in fp16 (z = 2^e / l); for fp32 caches
// they are o / l in fp32 (z = 1). Elements in lane order: lane (ln, lq)
// holds dimensions 16 t + 4 lq + j of row ln in o[t][j]; the four lanes of
// a row call together.
//
// partial_exp: the exponent e with every |o| / 2^e below 1, reduced across
// the row's lanes (every lane of the wave must call it).
template <int D, int KV>
__device__ __forceinline__ int partial_exp(const f32x4 (&o)[D / 16]) {
  int e = 0;
  if constexpr (KV != kKvF32) {
    float amax = 0.f;
#pragma unroll
    for (int t = 0; t < D / 16; ++t)
#pragma unroll
      for (int j = 0; j < 4; ++j) amax = fmaxf(amax, __builtin_fabsf(o[t][j]));
    amax = fmaxf(amax, __shfl_xor(amax, 16));
    amax = fmaxf(amax, __shfl_xor(amax, 32));
    // amax = f 2^e with f in [0.5, 1): every element over 2^e is in [-1, 1].
    if (amax > 0.f && amax <= 3.0e38f) e = __builtin_amdgcn_frexp_expf(amax);
  }
  return e;
}

// store_partial: the row's stores, with inv = 1 / l (0 for l = 0) and e
// from above. (Scaling by 2^-e alone, not by 1 / l as well, takes one
// instruction per element instead of two.)
template <int D, int KV>
__device__ __forceinline__ void store_partial(void* part_o, float* part_ml, int64_t prow, const f32x4 (&o)[D / 16],
                                              float m, float l, float inv, int e, int lq) {
  float z = 1.f;
  if constexpr (KV != kKvF32) {
    uint32_t w[D / 8];
#pragma unroll
    for (int t = 0; t < D / 16; ++t)
#pragma unroll
      for (int j = 0; j < 4; j += 2) {
        const f16x2 h = {static_cast<_Float16>(__builtin_ldexpf(o[t][j], -e)),
                         static_cast<_Float16>(__builtin_ldexpf(o[t][j + 1], -e))};
        w[2 * t + j / 2] = __builtin_bit_cast(uint32_t, h);
      }
    uint4* dst = reinterpret_cast<uint4*>(static_cast<uint16_t*>(part_o) + prow * D + (D / 4) * lq);
#pragma unroll
    for (int c = 0; c < D / 32; ++c) dst[c] = uint4{w[4 * c], w[4 * c + 1], w[4 * c + 2], w[4 * c + 3]};
    z = __builtin_ldexpf(inv, e);
  } else {
    f32x4* dst = reinterpret_cast<f32x4*>(static_cast<float*>(part_o) + prow * D + (D / 4) * lq);
#pragma unroll
    for (int t = 0; t < D / 16; ++t) dst[t] = o[t] * inv;
  }
  // A state without tokens (l = 0) takes no part in the merge's maximum; a
  // NaN m (a bad row) is kept.
  const float m_out = (l > 0.f || m != m) ? m : kNegInf;
  if (lq == 0) *reinterpret_cast<f32x4*>(part_ml + prow * kPartMl) = f32x4{m_out, l, z, 0.f};
}

// Both steps for one row; `active` says whether the row exists.
template <int D, int KV>
__device__ __forceinline__ void write_partial(void* part_o, float* part_ml, int64_t prow, const f32x4 (&o)[D / 16],
                                              float m, float l, int lq, bool active) {
  const float inv = l > 0.f ? 1.f / l : 0.f;
  const int e = partial_exp<D, KV>(o);
  if (active) store_partial<D, KV>(part_o, part_ml, prow, o, m, l, inv, e, lq);
}

__device__ __forceinline__ int rl(int x, int i) { return __builtin_amdgcn_readlane(x, i); }
__device__ __forceinline__ float rlf(float x, int i) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), i));
}

// Token row of S tile t, MFMA row m inside a pair (see the header).
__device__ __forceinline__ int pair_token(int t, int m) { return ((m >> 2) << 3) + (t << 2) + (m & 3); }

// Operands of one block pair in compute form: bf16 bits (bf16 and fp8
// caches) or fp32. Lane (ln, lq):
//   k[t][j]: K of token pair_token(t, ln), dims 32j + 8lq .. + 8 (bf16)
//            or 16j + 4lq .. + 4 (fp32);
//   v[dt]  : V of dim 16dt + ln, tokens 8lq .. 8lq + 7 of the pair.
template <int D, int KV>
struct Ops {
  static constexpr bool f32 = KV == kKvF32;
  static constexpr int kk = f32 ? D / 16 : D / 32;
  typedef typename std::conditional<f32, f32x4, uint4>::type T;
  T k[2][kk];
  T v[D / 16][f32 ? 2 : 1];
};

// fp8 caches load raw codes (half the registers) and convert per pair.
template <int D>
struct Fp8Frags {
  static constexpr int kk = D / 32;
  typedef uint2 T;
  uint2 k[2][kk];
  uint2 v[D / 16][1];
};

template <int D, int KV>
using Frags = typename std::conditional<KV == kKvFp8, Fp8Frags<D>, Ops<D, KV>>::type;

// standin: every load reads the first bytes of kb0 instead (a placeholder
// whose data is never used).
template <int D, int KV>
__device__ __forceinline__ void load_pair(Frags<D, KV>& f, const unsigned char* kb0, const unsigned char* kb1,
                                          const unsigned char* vb0, const unsigned char* vb1, int ln, int lq,
                                          bool standin = false) {
  using G = Geo<D, KV>;
  using F = Frags<D, KV>;
  typedef typename F::T T;
  auto at = [&](const unsigned char* a) { return reinterpret_cast<const T*>(standin ? kb0 : a); };
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int tok = pair_token(t, ln);
    const unsigned char* kr = (tok < 16 ? kb0 : kb1) + (tok & 15) * G::row_bytes;
#pragma unroll
    for (int j = 0; j < F::kk; ++j) {
      if constexpr (KV == kKvFp8)
        f.k[t][j] = *at(kr + 32 * j + 8 * lq);
      else
        f.k[t][j] = *at(kr + (4 * j + lq) * 16);
    }
  }
  const unsigned char* vb = (lq >= 2 ? vb1 : vb0) + (lq & 1) * 8 * G::eb + ln * G::vrow_bytes;
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    const unsigned char* vr = vb + 16 * dt * G::vrow_bytes;
    f.v[dt][0] = *at(vr);
    if constexpr (KV == kKvF32) f.v[dt][1] = *at(vr + 16);
  }
}

template <int D>
__device__ __forceinline__ void fp8_to_ops(const Fp8Frags<D>& f, Ops<D, kKvFp8>& o) {
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int j = 0; j < D / 32; ++j) o.k[t][j] = fp8x8_to_bf16x8(f.k[t][j]);
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) o.v[dt][0] = fp8x8_to_bf16x8(f.v[dt][0]);
}

// Zero the V^T operands of tokens past `valid` in this lane's block, so
// unused slots of a partial block never reach the value product.
template <int D, int KV>
__device__ __forceinline__ void mask_v(Ops<D, KV>& o, int lq, int valid0, int valid1) {
  const int valid = lq >= 2 ? valid1 : valid0;
  const int slot0 = 8 * (lq & 1);
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    if constexpr (KV == kKvF32) {
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (slot0 + 4 * h + e >= valid) o.v[dt][h][e] = 0.f;
    } else {
      uint32_t* a = reinterpret_cast<uint32_t*>(&o.v[dt][0]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t keep =
            (slot0 + 2 * e < valid ? 0x0000FFFFu : 0u) | (slot0 + 2 * e + 1 < valid ? 0xFFFF0000u : 0u);
        a[e] &= keep;
      }
    }
  }
}

// Query rows of the unit in LDS (B operand of S^T = K Q^T): row r is D
// elements (bf16, or fp32 for fp32 caches), its 16-byte columns XOR-swizzled
// by the row so that the 16 lanes of a column read distinct banks.
template <int D, int KV>
struct QLds {
  static constexpr int eb = KV == kKvF32 ? 4 : 2;
  static constexpr int row_bytes = D * eb;
  static constexpr int ncol = row_bytes / 16;
  static constexpr int swz_mask = (ncol < 16 ? ncol : 16) - 1;
  static constexpr int bytes = kMaxRows * row_bytes;
  static __device__ __forceinline__ int offset(int row, int col) {
    return row * row_bytes + ((col ^ (row & swz_mask)) << 4);
  }
};

// Softmax state of one row tile (lane ln = row, lq = token / dim group).
template <int D>
struct RowState {
  f32x4 o[D / 16];
  float m;     // reference (log2 units), uniform over the 4 lanes of a row
  float l;     // per-lane partial sum
  float seen;  // largest exponent argument (scaled score - m) this lane has seen (-inf: none)
};

// Uniform description of one pair: blocks' valid tokens, row ranges and
// (fp8) scales.
struct PairInfo {
  int v0, v1;      // valid tokens (0: no block)
  int a0, e0;      // rows [a0, e0) of block 0
  int a1, e1;      // rows [a1, e1) of block 1
  float ks0, ks1;  // logit scale (softmax scale * log2 e * k_scale)
  float vs0, vs1;  // value scale (fp8) or 1
};

// One pair against one row tile `r`.
// Query operands of one row tile (lane: row 16r + ln, dims as K's).
template <int D, int KV>
struct QFrag {
  typename Ops<D, KV>::T q[Ops<D, KV>::kk];
};

template <int D, int KV>
__device__ __forceinline__ QFrag<D, KV> q_from_lds(const unsigned char* qlds, int r, int ln, int lq) {
  using O = Ops<D, KV>;
  using Q = QLds<D, KV>;
  QFrag<D, KV> qf;
#pragma unroll
  for (int j = 0; j < O::kk; ++j)
    qf.q[j] = *reinterpret_cast<const typename O::T*>(qlds + Q::offset(16 * r + ln, 4 * j + lq));
  return qf;
}

// kWide: the pair applies to every row of the tile (rows past the unit's
// end hold zero queries and are never written) and only a missing second
// block (pi.v1 == 0) is masked, by a reference of +inf for its half of the
// lanes: no branch, so the compiler interleaves consecutive tiles.
template <int D, int KV, bool kWide = false>
__device__ __forceinline__ void tile_step(const Ops<D, KV>& f, const QFrag<D, KV>& qfr, RowState<D>& st,
                                          const PairInfo& pi, int r, int ln, int lq) {
  using O = Ops<D, KV>;
  const auto& qf = qfr.q;
  f32x4 acc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
  if constexpr (O::f32) {
#pragma unroll
    for (int j = 0; j < O::kk; ++j)
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(f.k[t][j].x, qf[j].x, acc[t], 0, 0, 0);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(f.k[t][j].y, qf[j].y, acc[t], 0, 0, 0);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(f.k[t][j].z, qf[j].z, acc[t], 0, 0, 0);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(f.k[t][j].w, qf[j].w, acc[t], 0, 0, 0);
      }
  } else {
#pragma unroll
    for (int j = 0; j < O::kk; ++j)
#pragma unroll
      for (int t = 0; t < 2; ++t)
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, f.k[t][j]),
                                                         __builtin_bit_cast(bf16x8, qf[j]), acc[t], 0, 0, 0);
  }
  // Lane (ln, lq) holds row 16r + ln, tokens 8lq + 4t + i of the pair: all in
  // block lq >> 1, at slots 8(lq & 1) + 4t + i.
  const bool hi = lq >= 2;
  const float sc = hi ? pi.ks1 : pi.ks0;
  // Exponent arguments x = score * scale - m (the fp8 K scale is part of
  // `sc`), masked to -inf past the valid tokens and outside the rows the
  // blocks apply to. `seen` tracks the largest x: it is taken over the fma
  // results, which are canonical, so the maximum needs no NaN quieting.
  float x[8];
  const float mref = (kWide && hi && pi.v1 == 0) ? kInf : st.m;
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) x[4 * t + i] = __builtin_fmaf(acc[t][i], sc, -mref);
  const int row = 16 * r + ln;
  const int valid = hi ? pi.v1 : pi.v0;
  const int ra = hi ? pi.a1 : pi.a0, re = hi ? pi.e1 : pi.e0;
  const bool full = pi.v0 == kTok && pi.v1 == kTok && pi.a0 <= 16 * r && pi.e0 >= 16 * r + 16 &&
                    pi.a1 <= 16 * r && pi.e1 >= 16 * r + 16;
  if (!kWide && !full) {
    const int lim = (row >= ra && row < re) ? valid : 0;
    const int slot0 = 8 * (lq & 1);
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (slot0 + i >= lim) x[i] = kNegInf;
  }
  st.seen = fmaxf(fmaxf(fmaxf(fmaxf(st.seen, x[0]), fmaxf(x[1], x[2])), fmaxf(x[3], x[4])),
                  fmaxf(fmaxf(x[5], x[6]), x[7]));
  float p[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) p[i] = __builtin_amdgcn_exp2f(x[i]);
  st.l += ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
  if constexpr (O::f32) {
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
    const float vs = hi ? pi.vs1 : pi.vs0;
    float pv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) pv[i] = (KV == kKvFp8) ? p[i] * vs : p[i];
    const uint4 pb = {pack_bf16x2(pv[0], pv[1]), pack_bf16x2(pv[2], pv[3]), pack_bf16x2(pv[4], pv[5]),
                      pack_bf16x2(pv[6], pv[7])};
    const bf16x8 pbf = __builtin_bit_cast(bf16x8, pb);
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt)
      st.o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, f.v[dt][0]), pbf, st.o[dt], 0,
                                                        0, 0);
  }
}

// ---- wide units: block pairs shared by the four waves through LDS --------
// A pair's operands are kChunks 16-byte fragments per lane (K: tile t, slice
// j; then V: dim tile dt). Each wave loads a quarter of them (the
// fragments of all 64 lanes, from the addresses load_pair reads) into
// registers ahead of use, stores them to an LDS stage -- chunk c holds
// fragment c of every lane, lane i at byte 16 i -- and after a barrier every
// wave reads all chunks. (Plain loads stream faster than global-to-LDS
// copies here.)
template <int D, int KV>
struct Stage {  // bf16 operands (fp8 caches stage their codes converted)
  static constexpr int kKChunks = 2 * (D / 32);
  static constexpr int kChunks = kKChunks + D / 16;
  static constexpr int kPerWave = kChunks / kWaves;
  static constexpr int bytes = kChunks * 1024;
  static_assert(kChunks % kWaves == 0, "whole chunks per wave");
};

template <int D, int KV>
__device__ __forceinline__ const unsigned char* frag_src(int c, const unsigned char* kb0, const unsigned char* kb1,
                                                         const unsigned char* vb0, const unsigned char* vb1, int ln,
                                                         int lq) {
  using G = Geo<D, KV>;
  using S = Stage<D, KV>;
  if (c < S::kKChunks) {
    const int t = c / (D / 32), j = c % (D / 32);
    const int tok = pair_token(t, ln);
    return (tok < 16 ? kb0 : kb1) + (tok & 15) * G::row_bytes + (KV == kKvFp8 ? 32 * j + 8 * lq : (4 * j + lq) * 16);
  }
  const int dt = c - S::kKChunks;
  return (lq >= 2 ? vb1 : vb0) + (lq & 1) * 8 * G::eb + ln * G::vrow_bytes + 16 * dt * G::vrow_bytes;
}

// (A vector value rather than an array, so that it stays in registers.)
// fp8 caches hold the raw codes (8 bytes per fragment) until the quarter is
// stored, converted, to the stage.
template <int D, int KV>
struct Quarter {
  static constexpr int kWords = KV == kKvFp8 ? 2 : 4;  // dwords per fragment
  typedef unsigned int V __attribute__((ext_vector_type(kWords * Stage<D, KV>::kPerWave)));
  V v;
};

// This wave's quarter of pair (id0, id1).
template <int D, int KV>
__device__ __forceinline__ void load_quarter(Quarter<D, KV>& q, int id0, int id1, const unsigned char* kbase,
                                             const unsigned char* vbase, size_t blk_stride, int wave, int ln, int lq) {
  using S = Stage<D, KV>;
  const unsigned char* kb0 = kbase + id0 * blk_stride;
  const unsigned char* kb1 = kbase + id1 * blk_stride;
  const unsigned char* vb0 = vbase + id0 * blk_stride;
  const unsigned char* vb1 = vbase + id1 * blk_stride;
#pragma unroll
  for (int i = 0; i < S::kPerWave; ++i) {
    const unsigned char* src = frag_src<D, KV>(wave + kWaves * i, kb0, kb1, vb0, vb1, ln, lq);
    if constexpr (KV == kKvFp8) {
      const uint2 t = *reinterpret_cast<const uint2*>(src);
      q.v[2 * i] = t.x;
      q.v[2 * i + 1] = t.y;
    } else {
      const uint4 t = *reinterpret_cast<const uint4*>(src);
      q.v[4 * i] = t.x;
      q.v[4 * i + 1] = t.y;
      q.v[4 * i + 2] = t.z;
      q.v[4 * i + 3] = t.w;
    }
  }
}

template <int D, int KV>
__device__ __forceinline__ void store_quarter(const Quarter<D, KV>& q, unsigned char* stage, int wave, int lane) {
#pragma unroll
  for (int i = 0; i < Stage<D, KV>::kPerWave; ++i) {
    uint4 w;
    if constexpr (KV == kKvFp8)
      w = fp8x8_to_bf16x8(uint2{q.v[2 * i], q.v[2 * i + 1]});
    else
      w = uint4{q.v[4 * i], q.v[4 * i + 1], q.v[4 * i + 2], q.v[4 * i + 3]};
    *reinterpret_cast<uint4*>(stage + (wave + kWaves * i) * 1024 + lane * 16) = w;
  }
}

template <int D, int KV>
__device__ __forceinline__ void read_stage(Ops<D, KV>& o, const unsigned char* stage, int lane) {
  using S = Stage<D, KV>;
#pragma unroll
  for (int c = 0; c < S::kKChunks; ++c)
    o.k[c / (D / 32)][c % (D / 32)] = *reinterpret_cast<const uint4*>(stage + c * 1024 + lane * 16);
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt)
    o.v[dt][0] = *reinterpret_cast<const uint4*>(stage + (S::kKChunks + dt) * 1024 + lane * 16);
}

// Per-lane view of up to 64 block entries of a unit: lane i holds entry i.
struct Window {
  int id;     // physical block id (clamped into the pool)
  int valid;  // valid tokens (0: skip)
  int a, e;   // rows [a, e)
  float ks, vs;
};

__device__ __forceinline__ int ent_r0(uint32_t inf) { return inf & 63; }
__device__ __forceinline__ int ent_r1(uint32_t inf) { return ((inf >> 6) & 63) + 1; }
__device__ __forceinline__ int ent_valid(uint32_t inf) { return ((inf >> 12) & 15) + 1; }

// Loads of pair pp of a window (n entries) into f.
template <int D, int KV>
__device__ __forceinline__ void issue_pair(Frags<D, KV>& f, const Window& win, int n, int pp,
                                           const unsigned char* kbase, const unsigned char* vbase, size_t blk_stride,
                                           int ln, int lq, bool standin = false) {
  const int i0 = 2 * pp, i1 = 2 * pp + 1;
  const int id0 = rl(win.id, i0);
  const int id1 = i1 < n ? rl(win.id, i1) : id0;
  load_pair<D, KV>(f, kbase + id0 * blk_stride, kbase + id1 * blk_stride, vbase + id0 * blk_stride,
                   vbase + id1 * blk_stride, ln, lq, standin);
}

// Runs every pair of a window (n entries) through the unit's row tiles
// (rows outside a block's range are masked); pairs w, w + 4, ... belong to
// wave w. The next pair's loads are issued before the current pair is
// computed; the wave's first pair has been issued into fa by the caller.
template <int D, int KV>
__device__ __forceinline__ void run_window(const Window& win, int n, int nt, const unsigned char* kbase,
                                           const unsigned char* vbase, size_t blk_stride, float sc,
                                           const unsigned char* qlds, RowState<D> (&st)[kTiles],
                                           Frags<D, KV>& fa, int wave, int ln, int lq) {
  const int np = (n + 1) >> 1;
  if (wave >= np) return;
  auto info = [&](int pp) {
    PairInfo pi;
    const int i0 = 2 * pp, i1 = 2 * pp + 1;
    const bool has1 = i1 < n;
    pi.v0 = rl(win.valid, i0);
    pi.v1 = has1 ? rl(win.valid, i1) : 0;
    pi.a0 = rl(win.a, i0);
    pi.e0 = rl(win.e, i0);
    pi.a1 = has1 ? rl(win.a, i1) : 0;
    pi.e1 = has1 ? rl(win.e, i1) : 0;
    pi.ks0 = sc;
    pi.ks1 = sc;
    pi.vs0 = 1.f;
    pi.vs1 = 1.f;
    if constexpr (KV == kKvFp8) {
      pi.ks0 = sc * rlf(win.ks, i0);
      pi.vs0 = rlf(win.vs, i0);
      pi.ks1 = has1 ? sc * rlf(win.ks, i1) : pi.ks0;
      pi.vs1 = has1 ? rlf(win.vs, i1) : pi.vs0;
    }
    return pi;
  };
  auto tiles = [&](Ops<D, KV>& o, const PairInfo& pi) {
    if (pi.v0 < kTok || pi.v1 < kTok) mask_v<D, KV>(o, lq, pi.v0, pi.v1);
    // Row tiles the pair's valid blocks apply to.
    int lo = kMaxRows, hi = 0;
    if (pi.v0 > 0) {
      lo = pi.a0;
      hi = pi.e0;
    }
    if (pi.v1 > 0) {
      lo = lo < pi.a1 ? lo : pi.a1;
      hi = hi > pi.e1 ? hi : pi.e1;
    }
    const int t0 = lo >> 4, t1 = (hi - 1) >> 4;
#pragma unroll
    for (int r = 0; r < kTiles; ++r)
      if (r < nt && r >= t0 && r <= t1) tile_step<D, KV>(o, q_from_lds<D, KV>(qlds, r, ln, lq), st[r], pi, r, ln, lq);
  };
  auto compute = [&](Frags<D, KV>& f, int pp) {
    const PairInfo pi = info(pp);
    if (pi.v0 <= 0 && pi.v1 <= 0) return;
    if constexpr (KV == kKvFp8) {
      Ops<D, KV> o;
      fp8_to_ops<D>(f, o);
      tiles(o, pi);
    } else {
      tiles(f, pi);
    }
  };
  auto issue = [&](Frags<D, KV>& f, int pp, bool standin) {
    issue_pair<D, KV>(f, win, n, pp, kbase, vbase, blk_stride, ln, lq, standin);
  };
  // The next pair's loads are always issued (constant wait counts); past the
  // wave's last pair they are stand-ins that all read the first 16 bytes of
  // the pair just loaded (a cache hit), so later waits on them are short.
  Frags<D, KV> fb;
  int pp = wave;
  for (;;) {
    int pn = pp + kWaves;
    bool more = pn < np;
    issue(fb, more ? pn : pp, !more);
    compute(fa, pp);
    if (!more) break;
    pp = pn;
    pn = pp + kWaves;
    more = pn < np;
    issue(fa, more ? pn : pp, !more);
    compute(fb, pp);
    if (!more) break;
    pp = pn;
  }
}

// A unit's record as held by a wave: header fields (every lane holds the
// same value; made uniform with readfirstlane where used, so that a record
// fetched ahead of time is not waited for early) and, per lane, beam `lane`
// (lane < 16) and entry `lane`.
struct UnitRegs {
  int kvh, nrows, nstatic, nent, prow0, next, mode, nstatic2;
  int beam_l;
  int ent_id;
  uint32_t ent_inf;
};

// The record's second window (lane i: entry 64 + i), read only by units
// that have one, when they start.
__device__ __forceinline__ void load_window2(const UnitRec* recs, int idx, int lane, int* id, uint32_t* inf) {
  *id = recs[idx].ent_id2[lane];
  *inf = recs[idx].ent_info2[lane];
}

__device__ __forceinline__ int rfl(int x) { return __builtin_amdgcn_readfirstlane(x); }

__device__ __forceinline__ UnitRegs load_unit(const UnitRec* recs, int idx, int lane) {
  const UnitRec* r = recs + idx;
  UnitRegs u;
  const int4 h0 = *reinterpret_cast<const int4*>(&r->kvh);
  const int4 h1 = *reinterpret_cast<const int4*>(&r->prow0);
  u.kvh = h0.x;
  u.nrows = h0.y;
  u.nstatic = h0.z;
  u.nent = h0.w;
  u.prow0 = h1.x;
  u.next = h1.y;
  u.mode = h1.z;
  u.nstatic2 = h1.w;
  u.beam_l = r->beams[lane];
  u.ent_id = r->ent_id[lane];
  u.ent_inf = r->ent_info[lane];
  return u;
}

// Live and build-time lengths of the beams whose entries depend on them
// (the partial last block, the extension marker), loaded by those lanes.
// Current length of beam vb: for verification, virtual beam b * q_len + i
// is beam b's first seq_lens[b] - (q_len - 1 - i) tokens.
template <typename P>
__device__ __forceinline__ int beam_len(const P& p, int vb) {
  if (p.q_len <= 1) return p.seq_lens[vb];
  return p.seq_lens[vb / p.q_len] - (p.q_len - 1 - vb % p.q_len);
}

__device__ __forceinline__ void issue_live(const AttnParams& p, const UnitRegs& u, int lane, int* len, int* build) {
  const bool live = lane < u.nent && (u.ent_inf & (kEntLive | kEntExt)) != 0;
  const int slot = (u.ent_inf & kEntExt) ? u.ent_id : static_cast<int>(ent_r0(u.ent_inf)) / p.g;
  const int lb = __shfl(u.beam_l, slot & 15);  // all lanes take part in the shuffle
  *len = 0;
  *build = 0;
  if (live) {
    *len = beam_len(p, lb);
    *build = p.build_len[lb];
  }
}

// The unit's query rows, fetched into registers (thread t holds 16-byte
// chunks t, t + 256, ... of the rows) while the previous unit finishes, then
// stored to LDS in the swizzled layout. Rows past nrows repeat row 0 (their
// scores are always masked).
// (A vector value rather than an array, so that it stays in registers.)
template <int D, int KV>
struct QRegs {
  static constexpr int kPer = QLds<D, KV>::bytes / (kThreads * 16);
  typedef unsigned int V __attribute__((ext_vector_type(4 * kPer)));
  V v;
};

template <int D, int KV>
__device__ __forceinline__ void load_q(const AttnParams& p, const UnitRegs& u, QRegs<D, KV>& qr, int tid) {
  using Q = QLds<D, KV>;
#pragma unroll
  for (int i = 0; i < QRegs<D, KV>::kPer; ++i) {
    const int c = tid + kThreads * i;
    int row = c / Q::ncol;
    const int col = c % Q::ncol;
    row = row < u.nrows ? row : 0;
    const int b = __shfl(u.beam_l, row / p.g);
    const int qh = u.kvh * p.g + row % p.g;
    const uint4 t = *reinterpret_cast<const uint4*>(static_cast<const unsigned char*>(p.q) +
                                                    (static_cast<int64_t>(b) * p.hq + qh) * Q::row_bytes + col * 16);
    qr.v[4 * i] = t.x;
    qr.v[4 * i + 1] = t.y;
    qr.v[4 * i + 2] = t.z;
    qr.v[4 * i + 3] = t.w;
  }
}

template <int D, int KV>
__device__ __forceinline__ void store_q(const QRegs<D, KV>& qr, unsigned char* qbuf, int tid) {
  using Q = QLds<D, KV>;
#pragma unroll
  for (int i = 0; i < QRegs<D, KV>::kPer; ++i) {
    const int c = tid + kThreads * i;
    *reinterpret_cast<uint4*>(qbuf + Q::offset(c / Q::ncol, c % Q::ncol)) =
        uint4{qr.v[4 * i], qr.v[4 * i + 1], qr.v[4 * i + 2], qr.v[4 * i + 3]};
  }
}

template <int D, int KV, bool kWin2>
__global__ __launch_bounds__(kThreads, 1) void attn_kernel(AttnParams p) {
  using G = Geo<D, KV>;
  using Q = QLds<D, KV>;
  // LDS: the current unit's query rows, and the end-of-unit combine area
  // where each wave publishes the states of the row tiles other waves
  // combine (3 x 4 (wave, tile) slots).
  // Wide units (bf16) use the area after the query rows for their pair
  // stages instead.
  constexpr int kCombBytes = kWaves * (kTiles - 1) * G::comb_floats * 4;
  constexpr int kStageBytes = KV != kKvF32 ? 2 * Stage<D, KV>::bytes : 0;
  constexpr int kAreaBytes = kCombBytes > kStageBytes ? kCombBytes : kStageBytes;
  // Narrow units with a second window park its entries (per lane: block id
  // and info word; every wave writes the same values) until the first one
  // is done, instead of holding two more registers through the pair loop.
  constexpr int kWin2Bytes = kWin2 ? 8 * kMaxEntries : 0;
  // Wide units: each wave's "redo" vote (one word per wave).
  constexpr int kVoteBytes = 4 * kWaves;
  __shared__ __attribute__((aligned(16))) unsigned char lds[Q::bytes + kAreaBytes + kWin2Bytes + kVoteBytes];
  unsigned char* qbuf = lds;
  float* comb = reinterpret_cast<float*>(lds + Q::bytes);
  uint2* win2_lds = reinterpret_cast<uint2*>(lds + Q::bytes + kAreaBytes);
  int* votes = reinterpret_cast<int*>(lds + Q::bytes + kAreaBytes + kWin2Bytes);

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int ln = lane & 15;
  const int lq = lane >> 4;
  const size_t blk_stride = static_cast<size_t>(p.hkv) * G::blk_bytes;
  const bool paged = p.recs == nullptr;
  const float sc_w = p.scale_log2;
  const float sc = p.scale_log2;
  auto comb_slot = [&](int w, int r) {  // (wave w, tile r != w)
    return comb + (w * (kTiles - 1) + (r < w ? r : r - 1)) * G::comb_floats;
  };

  // ---- first unit -----------------------------------------------------------
  int rec_idx;
  UnitRegs u;
  int paged_b = 0, paged_split = 0;
  if (!paged) {
    rec_idx = static_cast<int>(blockIdx.x);
    u = load_unit(p.recs, rec_idx, lane);
  } else {
    // Paged path: unit = (beam, KV head, split) from the workgroup id, one
    // beam's g rows against up to 64 of its blocks.
    rec_idx = 0;
    paged_split = blockIdx.x % p.paged_nsplit;
    const int bh = blockIdx.x / p.paged_nsplit;
    paged_b = bh / p.hkv;
    u.kvh = bh % p.hkv;
    u.nrows = p.g;
    u.nstatic = 0;
    u.nent = 0;
    u.prow0 = 0;
    u.next = -1;
    u.mode = kModeNarrow;
    u.beam_l = paged_b;
    u.ent_id = 0;
    u.ent_inf = 0;
    u.nstatic2 = 0;
  }
  if (rfl(u.nrows) <= 0) return;
  QRegs<D, KV> qr;
  load_q<D, KV>(p, u, qr, tid);
  Frags<D, KV> fa;
  bool fa_ready = false;  // the unit's first pair, lengths and next record are in flight
  int ext_len = 0, ext_build = 0;  // live / extension lanes: live and build-time length
  UnitRegs nu;
  // Hand-over to unit n: a narrow unit's query rows, first pair and lengths
  // go out before this unit's combine. Every path assigns the carried
  // registers, so their previous contents are dead while a unit runs.
  auto handover = [&](const UnitRegs& n) {
    if (rfl(n.mode) == kModeNarrow) {
      load_q<D, KV>(p, n, qr, tid);
      const int nn = rfl(n.nstatic), nkvh = rfl(n.kvh);
      Window nw;
      nw.id = n.ent_id;
      issue_pair<D, KV>(fa, nw, nn > 0 ? nn : 1, wave < ((nn + 1) >> 1) ? wave : 0,
                        static_cast<const unsigned char*>(p.k_cache) + nkvh * G::blk_bytes,
                        static_cast<const unsigned char*>(p.v_cache) + nkvh * G::blk_bytes, blk_stride, ln, lq,
                        wave >= ((nn + 1) >> 1));
      issue_live(p, n, lane, &ext_len, &ext_build);
    } else {
      qr = QRegs<D, KV>{};
      fa = Frags<D, KV>{};
      ext_len = 0;
      ext_build = 0;
    }
    fa_ready = true;
  };

  for (;;) {
    TTS_PROF_MARK(0, rec_idx);
    const int kvh = rfl(u.kvh), nrows = rfl(u.nrows), nent = rfl(u.nent), prow0 = rfl(u.prow0),
              unext = rfl(u.next);
    const int nt = (nrows + 15) >> 4;
    const unsigned char* kbase = static_cast<const unsigned char*>(p.k_cache) + kvh * G::blk_bytes;
    const unsigned char* vbase = static_cast<const unsigned char*>(p.v_cache) + kvh * G::blk_bytes;

    if constexpr (KV != kKvF32) {
      if (rfl(u.mode) == kModeWide) {
        // ---- wide unit: wave w owns row tiles w, w + 4, ...; every block
        // pair is copied to an LDS stage once and read by all four waves ---
        using SG = Stage<D, KV>;
        const int nst = rfl(u.nstatic);
        nu.nrows = 0;
        if (unext >= 0) nu = load_unit(p.recs, unext, lane);
        QFrag<D, KV> qw[kWideTiles];
#pragma unroll
        for (int i = 0; i < kWideTiles; ++i) {
          const int row = 16 * (wave + kWaves * i) + ln;
          const bool ok = row < nrows;
          const int b = __shfl(u.beam_l, ok ? row / p.g : 0);
          const int qh = kvh * p.g + (ok ? row % p.g : 0);
          const uint16_t* qrow = static_cast<const uint16_t*>(p.q) + (static_cast<int64_t>(b) * p.hq + qh) * D;
#pragma unroll
          for (int j = 0; j < Ops<D, KV>::kk; ++j)
            qw[i].q[j] = ok ? *reinterpret_cast<const uint4*>(qrow + 32 * j + 8 * lq) : uint4{0u, 0u, 0u, 0u};
        }
        unsigned char* stages = lds + Q::bytes;
        const int np = (nst + 1) >> 1;
        const int tpw = (nt + kWaves - 1) / kWaves;
        // A wide unit has up to kMaxUnitEntries blocks, numbered across its
        // two windows: entry i < 64 in lane i of ent_id, entry 64 + i in lane
        // i of ent_id2. Entries (e0, e1) and block ids of pair pp; a pair
        // never straddles the two windows.
        int ent_id2 = 0;
        uint32_t ent_inf2 = 0;
        if (kWin2 && nst > kMaxEntries) load_window2(p.recs, rec_idx, lane, &ent_id2, &ent_inf2);
        int e0, e1, id0, id1;
        auto pair_ids = [&](int pp) {
          pp = pp < np ? pp : np - 1;  // past the end: a repeat of the last pair (a cache hit, never used)
          e0 = 2 * pp;
          e1 = 2 * pp + 1 < nst ? 2 * pp + 1 : e0;
          const int ids = (!kWin2 || e0 < kMaxEntries) ? u.ent_id : ent_id2;
          id0 = rl(ids, e0 & (kMaxEntries - 1));
          id1 = rl(ids, e1 & (kMaxEntries - 1));
        };
        // fp8: lane i holds the K and V scales of entries i and 64 + i, read
        // once per unit.
        float ksl = 1.f, vsl = 1.f, ksl2 = 1.f, vsl2 = 1.f;
        if constexpr (KV == kKvFp8) {
          if (lane < nst) {
            ksl = p.k_scale[u.ent_id];
            vsl = p.v_scale[u.ent_id];
          }
          if (kWin2 && lane + kMaxEntries < nst) {
            ksl2 = p.k_scale[ent_id2];
            vsl2 = p.v_scale[ent_id2];
          }
        }
        RowState<D> st[kWideTiles];
        float m_exact[kWideTiles];
#pragma unroll
        for (int i = 0; i < kWideTiles; ++i) m_exact[i] = 0.f;
        for (int attempt = 0;; ++attempt) {
#pragma unroll
          for (int i = 0; i < kWideTiles; ++i) {
#pragma unroll
            for (int d = 0; d < D / 16; ++d) st[i].o[d] = f32x4{0.f, 0.f, 0.f, 0.f};
            st[i].m = m_exact[i];
            st[i].l = 0.f;
            st[i].seen = kNegInf;
          }
          // Two quarters. bf16: each step first sends the next pair's loads
          // into the other quarter. fp8 (quarters of half the size): each
          // quarter is refilled with the pair two ahead as soon as it is
          // staged, so its loads are in flight for about two steps (faster
          // for fp8, slower for bf16 as compiled, where the wait counts of
          // alternate steps cover both quarters).
          constexpr bool kRefill = KV == kKvFp8;
          Quarter<D, KV> qa, qb;
          // fp8: the pair's block scales (K of block 0, 1; V of block 0, 1).
          auto scales = [&]() {
            if constexpr (KV == kKvFp8) {
              const float ks = e0 < kMaxEntries ? ksl : ksl2, vs = e0 < kMaxEntries ? vsl : vsl2;
              const int i0 = e0 & (kMaxEntries - 1), i1 = e1 & (kMaxEntries - 1);
              return f32x4{rlf(ks, i0), rlf(ks, i1), rlf(vs, i0), rlf(vs, i1)};
            } else {
              return f32x4{1.f, 1.f, 1.f, 1.f};
            }
          };
          pair_ids(0);
          load_quarter<D, KV>(qa, id0, id1, kbase, vbase, blk_stride, wave, ln, lq);
          if constexpr (kRefill) {
            pair_ids(1);
            load_quarter<D, KV>(qb, id0, id1, kbase, vbase, blk_stride, wave, ln, lq);
          }
          __syncthreads();  // every wave is done with the stage area (previous unit or attempt)
          // tpw_c: the tiles per wave as a constant of this copy of the
          // loop, or 0 for the count read at run time.
          auto step = [&](auto tpw_c, Quarter<D, KV>& cur, Quarter<D, KV>& nxt, int pp) {
            unsigned char* stage = stages + (pp & 1) * SG::bytes;
            if constexpr (kRefill) {
              store_quarter<D, KV>(cur, stage, wave, lane);
              pair_ids(pp + 2);
              load_quarter<D, KV>(cur, id0, id1, kbase, vbase, blk_stride, wave, ln, lq);
            } else {
              pair_ids(pp + 1);
              load_quarter<D, KV>(nxt, id0, id1, kbase, vbase, blk_stride, wave, ln, lq);
              store_quarter<D, KV>(cur, stage, wave, lane);
            }
            pair_ids(pp);
            const f32x4 cs = scales();
            __syncthreads();  // the whole pair is in the stage
            Ops<D, KV> o;
            read_stage<D, KV>(o, stage, lane);
            // fp8: the compiler's interleaving strategy for small matrix
            // products with LDS reads (long chain -1.5%; for bf16 it
            // measured within noise).
            if constexpr (KV == kKvFp8) __builtin_amdgcn_iglp_opt(1);
            PairInfo pi;
            pi.v0 = kTok;
            pi.v1 = 2 * pp + 1 < nst ? kTok : 0;
            pi.a0 = pi.a1 = 0;
            pi.e0 = pi.e1 = nrows;
            pi.ks0 = sc_w * cs.x;
            pi.ks1 = sc_w * cs.y;
            pi.vs0 = cs.z;
            pi.vs1 = cs.w;
            if (pi.v1 == 0) mask_v<D, KV>(o, lq, pi.v0, pi.v1);
            constexpr int kTpw = decltype(tpw_c)::value;
            if constexpr (kTpw > 0) {
#pragma unroll
              for (int i = 0; i < kTpw; ++i) tile_step<D, KV, true>(o, qw[i], st[i], pi, wave + kWaves * i, ln, lq);
            } else if (tpw >= kWideTiles) {
              // The unit's tiles per wave (uniform): one straight-line block
              // per count, so the compiler interleaves the tiles' products.
#pragma unroll
              for (int i = 0; i < kWideTiles; ++i) tile_step<D, KV, true>(o, qw[i], st[i], pi, wave + kWaves * i, ln, lq);
            } else if (tpw == 2) {
#pragma unroll
              for (int i = 0; i < 2; ++i) tile_step<D, KV, true>(o, qw[i], st[i], pi, wave + kWaves * i, ln, lq);
            } else {
              tile_step<D, KV, true>(o, qw[0], st[0], pi, wave, ln, lq);
            }
          };
          auto run = [&](auto tpw_c) {
            for (int pp = 0; pp < np; pp += 2) {
              step(tpw_c, qa, qb, pp);
              if (pp + 1 >= np) break;
              step(tpw_c, qb, qa, pp + 1);
            }
          };
          // fp8: one copy of the loop per tiles-per-wave count. In the single
          // loop the compiler copies the accumulators of the tiles that one
          // branch updates and another does not at every join (~78 64-bit
          // moves per pair at three tiles); the copies go away with the
          // joins (long chain -2%). bf16 keeps the single loop: its per-count
          // copies measured slower (7b64 +0.5 us, straggler +0.6 us).
          if constexpr (KV == kKvFp8) {
            if (tpw >= kWideTiles)
              run(std::integral_constant<int, kWideTiles>{});
            else if (tpw == 2)
              run(std::integral_constant<int, 2>{});
            else
              run(std::integral_constant<int, 1>{});
          } else {
            run(std::integral_constant<int, 0>{});
          }
          if (attempt == 0) TTS_PROF_MARK(1, rec_idx);
          if (attempt > 0) break;
          bool redo = false;
#pragma unroll
          for (int i = 0; i < kWideTiles; ++i) {
            const float mx = xlane_max16(st[i].seen);
            redo |= mx > kRefWindow || (mx < -kRefWindow && mx != kNegInf);
            m_exact[i] = mx == kNegInf ? 0.f : mx;
          }
          // The loop holds barriers, so every wave repeats it or none does:
          // each wave votes, and all four read every vote. (The votes are
          // written again only after the next unit's first barrier.)
          const bool wave_redo = __builtin_amdgcn_ballot_w64(redo) != 0;
          if (lane == 0) votes[wave] = wave_redo ? 1 : 0;
          __syncthreads();
          if ((votes[0] | votes[1] | votes[2] | votes[3]) == 0) break;
        }
        // Each wave writes the partial states of its own rows. The sums and
        // scales of all its tiles first, in straight-line code, so that the
        // tiles' cross-lane reductions overlap (a tile past the unit's rows
        // holds l = 0 and zeros, and is not written).
        float lw_[kWideTiles], inv_[kWideTiles];
        int e_[kWideTiles];
#pragma unroll
        for (int i = 0; i < kWideTiles; ++i) lw_[i] = xlane_sum16(st[i].l);
#pragma unroll
        for (int i = 0; i < kWideTiles; ++i) inv_[i] = lw_[i] > 0.f ? 1.f / lw_[i] : 0.f;
#pragma unroll
        for (int i = 0; i < kWideTiles; ++i) e_[i] = partial_exp<D, KV>(st[i].o);
#pragma unroll
        for (int i = 0; i < kWideTiles; ++i) {
          if (wave + kWaves * i >= nt) continue;  // wave-uniform
          const int row = 16 * (wave + kWaves * i) + ln;
          const int64_t prow = static_cast<int64_t>(kvh) * p.rows_per_head + prow0 + row;
          if (row < nrows) store_partial<D, KV>(p.part_o, p.part_ml, prow, st[i].o, st[i].m, lw_[i], inv_[i], e_[i], lq);
        }
        TTS_PROF_MARK(2, rec_idx);
        const int nu_rows_w = rfl(nu.nrows);
        if (nu_rows_w <= 0) break;
        handover(nu);
        rec_idx = unext;
        u = nu;
        continue;
      }
    }

    // ---- the unit's block window ------------------------------------------
    Window win;
    uint64_t bad_rows = 0;  // rows that met a bad block id or an over-long beam: NaN
    int nstatic = rfl(u.nstatic);
    if (!paged) {
      win.id = u.ent_id;
      win.a = ent_r0(u.ent_inf);
      win.e = ent_r1(u.ent_inf);
      win.valid = lane < nstatic ? ent_valid(u.ent_inf) : 0;
      if (!fa_ready) issue_live(p, u, lane, &ext_len, &ext_build);
    } else {
      const int L = p.seq_lens[paged_b];
      // Split j covers blocks [j * per, (j + 1) * per) of the beam (per <= 64).
      const int per = (p.paged_max_len + kTok * p.paged_nsplit - 1) / (kTok * p.paged_nsplit);
      const int j = paged_split * per + lane;
      int nb = (L + kTok - 1) / kTok;
      bool bad = false;
      if (L < 0 || L > p.paged_max_len || nb > p.max_blocks) {
        bad = true;
        nb = 0;
      }
      nstatic = nb - paged_split * per;
      nstatic = nstatic < 0 ? 0 : (nstatic < per ? nstatic : per);
      int id = 0, v = 0;
      if (lane < nstatic) {
        id = p.block_tables[static_cast<int64_t>(paged_b) * p.max_blocks + j];
        v = L - j * kTok;
        v = v < kTok ? v : kTok;
        if (id < 0 || id >= p.num_blocks) {
          bad = true;
          id = 0;
          v = 0;
        }
      }
      win.id = id;
      win.valid = v;
      win.a = 0;
      win.e = nrows;
      if (__builtin_amdgcn_ballot_w64(bad) != 0) bad_rows = ~0ull;
    }
    win.ks = 1.f;
    win.vs = 1.f;
    if constexpr (KV == kKvFp8) {
      if (win.valid > 0) {
        win.ks = p.k_scale[win.id];
        win.vs = p.v_scale[win.id];
      }
    }
    // The second window (static entries only, validated at build time) is
    // set up when the first one is done.
    const int nstatic2 = (!kWin2 || paged) ? 0 : rfl(u.nstatic2);
    if (kWin2 && nstatic2 > 0) {
      int id2;
      uint32_t inf2;
      load_window2(p.recs, rec_idx, lane, &id2, &inf2);
      win2_lds[lane] = uint2{static_cast<uint32_t>(id2), inf2};
    }
    if (!fa_ready && wave < ((nstatic + 1) >> 1))
      issue_pair<D, KV>(fa, win, nstatic, wave, kbase, vbase, blk_stride, ln, lq);
    // The next unit's record: it has this unit's pair loop to arrive.
    nu.nrows = 0;
    if (unext >= 0) nu = load_unit(p.recs, unext, lane);

    store_q<D, KV>(qr, qbuf, tid);
    __syncthreads();  // query rows in LDS

    // ---- the unit's blocks with m_ref = 0; again with every row's exact
    // maximum in the rare case that a row's maximum left the safe window ----
    RowState<D> st[kTiles];
    float m_exact[kTiles];
#pragma unroll
    for (int r = 0; r < kTiles; ++r) m_exact[r] = 0.f;
    if (!paged && lane < nstatic && (u.ent_inf & kEntLive)) {
      // The beam's partial last block: it fills up as tokens are appended.
      const int v = win.valid + (ext_len - ext_build);
      win.valid = v < 0 ? 0 : (v > kTok ? kTok : v);
    }
    for (int attempt = 0;; ++attempt) {
#pragma unroll
      for (int r = 0; r < kTiles; ++r) {
#pragma unroll
        for (int i = 0; i < D / 16; ++i) st[r].o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
        st[r].m = m_exact[r];
        st[r].l = 0.f;
        st[r].seen = kNegInf;
      }
      if (attempt > 0 && wave < ((nstatic + 1) >> 1))
        issue_pair<D, KV>(fa, win, nstatic, wave, kbase, vbase, blk_stride, ln, lq);
      // Windows of blocks: the unit's own entries first (one or two
      // windows), then (usually none) blocks its beams gained after the
      // metadata was built, read from the live block table 64 at a time. One
      // call site keeps the register allocation of the pair loop in one
      // piece.
      Window cw = win;
      int cn = nstatic;
      bool second = nstatic2 > 0;
      uint64_t ext_left = paged ? 0ull
                                : __builtin_amdgcn_ballot_w64(lane >= nstatic && lane < nent &&
                                                              (u.ent_inf & kEntExt) != 0);
      int xb = 0, xnext = 0, xend = 0, xlen = 0, xa = 0, xe = 0;
      for (;;) {
        run_window<D, KV>(cw, cn, nt, kbase, vbase, blk_stride, sc, qbuf, st, fa, wave, ln, lq);
        if (attempt == 0) TTS_PROF_MARK(1, rec_idx);
        // The next window: the unit's second one, else the next extension
        // window; one issue site below for both.
        int id = 0, v = 0, wa, we;
        if (second) {
          second = false;
          cn = nstatic2;
          const uint2 w2 = win2_lds[lane];
          id = static_cast<int>(w2.x);
          v = lane < cn ? ent_valid(w2.y) : 0;
          wa = ent_r0(w2.y);
          we = ent_r1(w2.y);
        } else {
          while (xnext >= xend && ext_left != 0) {
            const int e = static_cast<int>(__builtin_ctzll(ext_left));
            ext_left &= ext_left - 1;
            xlen = rl(ext_len, e);
            const int B = rl(ext_build, e);
            xb = __shfl(u.beam_l, rl(u.ent_id, e) & 15);
            xa = rl(win.a, e);
            xe = rl(win.e, e);
            xnext = (B + kTok - 1) / kTok;
            xend = (xlen + kTok - 1) / kTok;
            if (xlen < B) {
              xend = xnext;  // shorter than at build time: the merge reports NaN
            } else if (xend > p.max_blocks) {
              xend = xnext;  // longer than its table row: NaN rows
              bad_rows |= (xe >= 64 ? ~0ull : ((1ull << xe) - 1)) & ~((1ull << xa) - 1);
            }
          }
          if (xnext >= xend) break;
          cn = (xend - xnext) < kMaxEntries ? (xend - xnext) : kMaxEntries;
          bool xbad = false;
          if (lane < cn) {
            const int j = xnext + lane;
            id = p.block_tables[static_cast<int64_t>(xb / p.q_len) * p.max_blocks + j];
            v = xlen - j * kTok;
            v = v < kTok ? v : kTok;
            if (id < 0 || id >= p.num_blocks) {
              xbad = true;
              id = 0;
              v = 0;
            }
          }
          if (__builtin_amdgcn_ballot_w64(xbad) != 0)
            bad_rows |= (xe >= 64 ? ~0ull : ((1ull << xe) - 1)) & ~((1ull << xa) - 1);
          wa = xa;
          we = xe;
          xnext += cn;
        }
        cw.id = id;
        cw.valid = v;
        cw.a = wa;
        cw.e = we;
        cw.ks = 1.f;
        cw.vs = 1.f;
        if constexpr (KV == kKvFp8) {
          if (v > 0) {
            cw.ks = p.k_scale[id];
            cw.vs = p.v_scale[id];
          }
        }
        if (wave < ((cn + 1) >> 1)) issue_pair<D, KV>(fa, cw, cn, wave, kbase, vbase, blk_stride, ln, lq);
      }
      if (attempt > 0) break;
      bool redo = false;
#pragma unroll
      for (int r = 0; r < kTiles; ++r) {
        const float mx = xlane_max16(st[r].seen);
        redo |= mx > kRefWindow || (mx < -kRefWindow && mx != kNegInf);
        m_exact[r] = mx == kNegInf ? 0.f : mx;
      }
      if (__builtin_amdgcn_ballot_w64(redo) == 0) break;
    }

    // ---- hand over: the next unit's query copies and first pair go out
    // before this unit's combine ---------------------------------------------
    __syncthreads();  // every wave is done with qbuf
    TTS_PROF_MARK(4, rec_idx);
    const int nu_rows = rfl(nu.nrows);
    if (nu_rows > 0) handover(nu);

    TTS_PROF_MARK(5, rec_idx);
    // ---- combine the four waves' states, tile r by wave r ------------------
    // (Every tile's row sums first, in straight-line code, so that their
    // cross-lane reductions overlap.)
    float lt_[kTiles];
#pragma unroll
    for (int r = 0; r < kTiles; ++r) lt_[r] = xlane_sum16(st[r].l);
#pragma unroll
    for (int r = 0; r < kTiles; ++r) {
      if (r < nt && r != wave) {
        float* c = comb_slot(wave, r);
#pragma unroll
        for (int dt = 0; dt < D / 16; ++dt)
          *reinterpret_cast<f32x4*>(c + ln * G::comb_row + 16 * dt + 4 * lq) = st[r].o[dt];
        if (lq == 0) {
          c[kTok * G::comb_row + ln] = st[r].m;
          c[kTok * G::comb_row + kTok + ln] = lt_[r];
        }
      }
    }
    __syncthreads();
    TTS_PROF_MARK(6, rec_idx);
    // Wave r combines tile r: its own state straight from registers (one
    // code path per tile index, so nothing is copied), the other waves'
    // from LDS, in wave order.
#pragma unroll
    for (int r = 0; r < kTiles; ++r) {
      if (r != wave || r >= nt) continue;
      const int row = 16 * r + ln;
      const float own_l = lt_[r];
      // A wave that saw no token of the row (l = 0: no pair of it, or every
      // score masked) keeps its initial reference; it must not set the
      // maximum, or a row whose scores all lie far below it would lose every
      // weight to underflow.
      float mw[kWaves], lw[kWaves], mx = kNegInf;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        lw[w] = (w == r) ? own_l : comb_slot(w, r)[kTok * G::comb_row + kTok + ln];
        const float m = (w == r) ? st[r].m : comb_slot(w, r)[kTok * G::comb_row + ln];
        mw[w] = lw[w] > 0.f ? m : kNegInf;
        mx = fmaxf(mx, mw[w]);
      }
      float l = 0.f;
      f32x4 o[D / 16];
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float f = mw[w] == kNegInf ? 0.f : __builtin_amdgcn_exp2f(mw[w] - mx);
        if (w == r) {
          l += own_l * f;
#pragma unroll
          for (int dt = 0; dt < D / 16; ++dt) o[dt] += st[r].o[dt] * f;
        } else {
          const float* c = comb_slot(w, r);
          l += lw[w] * f;
          // All of the wave's reads first: read and add one at a time, the
          // compiler waits for each read before issuing the next.
          f32x4 t[D / 16];
#pragma unroll
          for (int dt = 0; dt < D / 16; ++dt)
            t[dt] = *reinterpret_cast<const f32x4*>(c + ln * G::comb_row + 16 * dt + 4 * lq);
#pragma unroll
          for (int dt = 0; dt < D / 16; ++dt) o[dt] += t[dt] * f;
        }
      }
      float m_fin = mx;
      if ((bad_rows >> row) & 1ull) m_fin = __builtin_nanf("");
      if (row < nrows) {
        if (paged && p.paged_nsplit == 1) {
          // Whole sequence in this unit: the normalised result.
          float* orow = p.out + (static_cast<int64_t>(paged_b) * p.hq + kvh * p.g + row) * D;
          const float inv = (l > 0.f) ? 1.f / l : 0.f;
          const bool nan = m_fin != m_fin;
#pragma unroll
          for (int dt = 0; dt < D / 16; ++dt) {
            f32x4 v = o[dt] * inv;
            if (nan) v = f32x4{m_fin, m_fin, m_fin, m_fin};
            *reinterpret_cast<f32x4*>(orow + 16 * dt + 4 * lq) = v;
          }
        } else {
          int64_t prow;
          if (paged)
            prow = (static_cast<int64_t>(paged_b) * p.paged_nsplit + paged_split) * p.hq + kvh * p.g + row;
          else
            prow = static_cast<int64_t>(kvh) * p.rows_per_head + prow0 + row;
          write_partial<D, KV>(p.part_o, p.part_ml, prow, o, m_fin, l, lq, true);
        }
      }
    }
#ifdef TTS_PROFILE_UNITS
    TTS_PROF_MARK(2, rec_idx);
    if (KV != kKvF32 && threadIdx.x == 0 && rec_idx < kProfSlots)
      g_prof[rec_idx][3] = (static_cast<uint64_t>(__builtin_amdgcn_s_getreg((3 << 11) | 20)) << 32) |
                           static_cast<uint32_t>(__builtin_amdgcn_s_getreg((31 << 11) | 4));
#endif
    if (nu_rows <= 0) break;
    rec_idx = unext;
    u = nu;
    fa_ready = true;
  }
}

// kEpl consecutive stored elements of a partial row (fp16 or fp32), loaded
// with one or two vector loads and widened one at a time.
template <int kEpl, bool F16>
struct MergeRaw;
template <>
struct MergeRaw<8, true> {
  typedef uint4 T;
  static __device__ __forceinline__ T load(const void* base, int64_t off) {
    return *reinterpret_cast<const uint4*>(static_cast<const _Float16*>(base) + off);
  }
  static __device__ __forceinline__ float get(const T& t, int i) {
    const uint32_t w = i < 2 ? t.x : (i < 4 ? t.y : (i < 6 ? t.z : t.w));
    const f16x2 hv = __builtin_bit_cast(f16x2, w);
    return static_cast<float>((i & 1) ? hv.y : hv.x);
  }
};
template <>
struct MergeRaw<4, true> {
  typedef uint2 T;
  static __device__ __forceinline__ T load(const void* base, int64_t off) {
    return *reinterpret_cast<const uint2*>(static_cast<const _Float16*>(base) + off);
  }
  static __device__ __forceinline__ float get(const T& t, int i) {
    const f16x2 hv = __builtin_bit_cast(f16x2, i < 2 ? t.x : t.y);
    return static_cast<float>((i & 1) ? hv.y : hv.x);
  }
};
template <>
struct MergeRaw<8, false> {
  struct T {
    f32x4 a, b;
  };
  static __device__ __forceinline__ T load(const void* base, int64_t off) {
    const f32x4* src = reinterpret_cast<const f32x4*>(static_cast<const float*>(base) + off);
    return T{src[0], src[1]};
  }
  static __device__ __forceinline__ float get(const T& t, int i) { return i < 4 ? t.a[i] : t.b[i - 4]; }
};
template <>
struct MergeRaw<4, false> {
  typedef f32x4 T;
  static __device__ __forceinline__ T load(const void* base, int64_t off) {
    return *reinterpret_cast<const f32x4*>(static_cast<const float*>(base) + off);
  }
  static __device__ __forceinline__ float get(const T& t, int i) { return t[i]; }
};

// Exact merge of the partial softmax states of each (beam, query head), in
// the order of the beam's slot list. With M = max_k m_k over the states
// that saw tokens (l_k > 0), w_k = l_k 2^(m_k - M), and e_k the stored
// elements with factor z_k (e_k z_k = o_k / l_k):
//   out = sum_k w_k z_k e_k / sum_k w_k.
// A slot-table row of zeros for the paged path, which has no table (the
// merges read their table entries without a branch).
__device__ const int kZeroTabRow[kSlotTabReadAhead] = {};

// Two kernels compute it; launch_merge picks by the number of rows.
//
// merge_row_kernel: D / 2 lanes per row (2 elements per lane), for batches
// with few rows, where spreading each row over many lanes shortens the
// work after the data arrives. A row's slot count and first kMergeBatch
// slots sit in one row of the slot table and are loaded with the beam's
// lengths; then kMergeBatch states at a time, the table entries of the
// next batch loaded with them: 1 + ceil(n / kMergeBatch) round trips to
// memory for n slots.
template <int D, bool F16>
__global__ __launch_bounds__(kThreads) void merge_row_kernel(MergeParams p) {
  constexpr int kTpr = D / 2;
  constexpr int kRows = kThreads / kTpr;
  constexpr int kBatch = kMergeBatch;
  const int r = blockIdx.x * kRows + threadIdx.x / kTpr;
  // Stored position pos0 (lane order) holds dimension d0, pos0 + 1 holds d0 + 1.
  const int pos0 = (threadIdx.x % kTpr) * 2;
  const int d0 = 16 * ((pos0 % (D / 4)) / 4) + 4 * (pos0 / (D / 4)) + pos0 % 4;
  if (r >= p.num_seqs * p.hq) return;
  const int b = r / p.hq;
  const int h = r % p.hq;
  const int* tab = p.slot_tab ? p.slot_tab + static_cast<int64_t>(b) * p.slot_stride : nullptr;
  // The row's inputs in one round trip: its table row (count and first
  // kBatch entries; the paged path reads a row of zeros), its live length
  // and its build-time length (the paged path, which has none, reads the
  // live one again). No load waits for another.
  const int* tabr = tab ? tab : kZeroTabRow;
  int ent[kBatch];
#pragma unroll
  for (int k = 0; k < kBatch; ++k) ent[k] = tabr[1 + k];
  const int n = tab ? tabr[0] : p.paged_nsplit;
  const int64_t head_base = tab ? static_cast<int64_t>(h / p.g) * p.rows_per_head + h % p.g : 0;
  const int L = beam_len(p, b);
  const int blen = (p.build_len ? p.build_len : p.seq_lens)[b];
  bool nan = p.build_len && L < blen;
  float mx = kNegInf, den = 0.f;
  f32x2 acc = {0.f, 0.f};
  for (int k0 = 0; k0 < n; k0 += kBatch) {
    f32x4 ml[kBatch];
    f32x2 o[kBatch];
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const int kk = k0 + k < n ? k0 + k : n - 1;
      int64_t row;
      if (tab)
        row = head_base + (k0 + k < n ? ent[k] : ent[0]);
      else
        row = (static_cast<int64_t>(b) * p.paged_nsplit + kk) * p.hq + h;
      ml[k] = *reinterpret_cast<const f32x4*>(p.part_ml + row * kPartMl);
      if constexpr (F16) {
        const f16x2 hv = *reinterpret_cast<const f16x2*>(static_cast<const uint16_t*>(p.part_o) + row * D + pos0);
        o[k] = f32x2{static_cast<float>(hv.x), static_cast<float>(hv.y)};
      } else {
        o[k] = *reinterpret_cast<const f32x2*>(static_cast<const float*>(p.part_o) + row * D + pos0);
      }
    }
    // The next batch's table entries travel with this batch's states
    // (stride >= n + 1, so the reads stay inside the beam's table row).
    if (tab && k0 + kBatch < n) {
#pragma unroll
      for (int k = 0; k < kBatch; ++k) ent[k] = k0 + kBatch + k < n ? tab[1 + k0 + kBatch + k] : 0;
    }
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      if (k0 + k >= n) ml[k] = f32x4{kNegInf, 0.f, 0.f, 0.f};
      if (ml[k].y == 0.f && ml[k].x == ml[k].x) ml[k].x = kNegInf;  // a state without tokens
    }
    float bm = kNegInf;
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      nan |= ml[k].x != ml[k].x;
      bm = fmaxf(bm, ml[k].x);
    }
    const float mn = fmaxf(mx, bm);
    if (mn == kNegInf) continue;
    const float a = (mx == kNegInf) ? 0.f : __builtin_amdgcn_exp2f(mx - mn);
    den *= a;
    acc *= a;
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const float w = (ml[k].x == kNegInf) ? 0.f : ml[k].y * __builtin_amdgcn_exp2f(ml[k].x - mn);
      den += w;
      acc += o[k] * (w * ml[k].z);
    }
    mx = mn;
  }
  const float inv = (den > 0.f && L > 0) ? 1.f / den : 0.f;
  f32x2 w = acc * inv;
  if (nan) {
    const float q = __builtin_nanf("");
    w = f32x2{q, q};
  }
  *reinterpret_cast<f32x2*>(p.out + static_cast<int64_t>(r) * D + d0) = w;
}

// merge_kernel: for batches with many rows. One wave per workgroup, sixteen
// lanes per row, each lane holding D / 16 consecutive stored elements (one
// or two 16-byte loads per state). Lane j of a row holds slot table entries
// j, j + 16, ... (the first kMergeTabChunks
// chunks are read in the first round trip to memory, with the beam's
// lengths); for a batch of 16 slots, lane j reads slot j's (m, l, s) and
// every lane reads its elements of every slot of the batch, the slots' rows
// shuffled across the row's lanes: one round trip per batch. The weights
// are added in slot order.
constexpr int kMergeLanes = 16;
// Up to this many rows the one-row-per-wave kernel runs (about the waves
// the GPU keeps resident at its occupancy); above, the sixteen-lane one.
constexpr int kMergeRowKernelMaxRows = 4096;
constexpr int kMergeTabChunks = 4;
static_assert(1 + kMergeTabChunks * kMergeLanes <= kSlotTabReadAhead && 1 + kMergeBatch <= kSlotTabReadAhead,
              "the merges' table read-ahead stays inside the table's padding");
constexpr int kMergeThreads = 64;
template <int D, bool F16>
__global__ __launch_bounds__(kMergeThreads) void merge_kernel(MergeParams p) {
  constexpr int kLpr = kMergeLanes;
  constexpr int kEpl = D / kLpr;              // stored elements per lane
  constexpr int kRows = kMergeThreads / kLpr;  // rows per workgroup
  constexpr int kBatch = kLpr;                // slots whose states are loaded together
  const int lane = threadIdx.x & 63;
  const int j = lane & (kLpr - 1);
  const int gbase = lane & ~(kLpr - 1);  // first lane of this row's group
  const int total = p.num_seqs * p.hq;
  const int r_raw = static_cast<int>(blockIdx.x) * kRows + static_cast<int>(threadIdx.x) / kLpr;
  const bool valid = r_raw < total;
  const int r = valid ? r_raw : total - 1;  // surplus rows repeat the last one and store nothing
  const int b = r / p.hq;
  const int h = r % p.hq;
  const int* tab = p.slot_tab ? p.slot_tab + static_cast<int64_t>(b) * p.slot_stride : nullptr;
  // The row's inputs in one round trip, as in merge_row_kernel: the count,
  // the first kMergeTabChunks x 16 entries (read past the count, which the
  // table's read-ahead zeros keep in bounds; entries past n are not used),
  // the live and the build-time length.
  const int* tabr = tab ? tab : kZeroTabRow;
  int ent[kMergeTabChunks];
#pragma unroll
  for (int c = 0; c < kMergeTabChunks; ++c) ent[c] = tabr[1 + kBatch * c + j];
  const int n = tab ? tabr[0] : p.paged_nsplit;
  const int head_base = tab ? (h / p.g) * p.rows_per_head + h % p.g : 0;
  // Partial row of slot k (k < n).
  auto slot_row = [&](int k, int entry) { return tab ? head_base + entry : (b * p.paged_nsplit + k) * p.hq + h; };
  const int L = beam_len(p, b);
  const int blen = (p.build_len ? p.build_len : p.seq_lens)[b];
  bool nan = p.build_len && L < blen;
  float mx = kNegInf, den = 0.f;
  float acc[kEpl];
#pragma unroll
  for (int e = 0; e < kEpl; ++e) acc[e] = 0.f;
  for (int k0 = 0, c = 0; k0 < n; k0 += kBatch, ++c) {
    // Lane j: slot k0 + j (a repeat of slot k0 past the end).
    const bool has = k0 + j < n;
    const int kk = has ? k0 + j : k0;
    int entry = 0;
    if (tab) {
      if (c < kMergeTabChunks) {
        entry = ent[0];
#pragma unroll
        for (int i = 1; i < kMergeTabChunks; ++i)
          if (c == i) entry = ent[i];
        const int first = __shfl(entry, gbase);  // slot k0's entry (every lane takes part)
        if (!has) entry = first;
      } else {
        entry = tab[1 + kk];
      }
    }
    const int row_j = slot_row(kk, entry);
    f32x4 ml = *reinterpret_cast<const f32x4*>(p.part_ml + static_cast<int64_t>(row_j) * kPartMl);
    typename MergeRaw<kEpl, F16>::T raw[kBatch];
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const int row_k = __shfl(row_j, gbase + k);
      raw[k] = MergeRaw<kEpl, F16>::load(p.part_o, static_cast<int64_t>(row_k) * D + kEpl * j);
    }
    if (!has) ml = f32x4{kNegInf, 0.f, 0.f, 0.f};
    if (ml.y == 0.f && ml.x == ml.x) ml.x = kNegInf;  // a state without tokens
    nan |= ml.x != ml.x;
    float bm = ml.x;
#pragma unroll
    for (int o = 1; o < kLpr; o <<= 1) bm = fmaxf(bm, __shfl_xor(bm, o));
    const float mn = fmaxf(mx, bm);
    if (mn == kNegInf) continue;  // uniform over the row's lanes
    const float a = (mx == kNegInf) ? 0.f : __builtin_amdgcn_exp2f(mx - mn);
    den *= a;
#pragma unroll
    for (int i = 0; i < kEpl; ++i) acc[i] *= a;
    const float w = (ml.x == kNegInf) ? 0.f : ml.y * __builtin_amdgcn_exp2f(ml.x - mn);
    const float ws = w * ml.z;
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const float wk = __shfl(w, gbase + k);
      const float wsk = __shfl(ws, gbase + k);
      if (k0 + k < n) {
        den += wk;
#pragma unroll
        for (int i = 0; i < kEpl; ++i) acc[i] += MergeRaw<kEpl, F16>::get(raw[k], i) * wsk;
      }
    }
    mx = mn;
  }
  // A NaN state in any slot of the row makes the row NaN.
  int any_nan = nan ? 1 : 0;
#pragma unroll
  for (int o = 1; o < kLpr; o <<= 1) any_nan |= __shfl_xor(any_nan, o);
  if (!valid) return;
  const float inv = (den > 0.f && L > 0) ? 1.f / den : 0.f;
  const float q = __builtin_nanf("");
  float* orow = p.out + static_cast<int64_t>(r) * D;
  // Stored position pos holds dimension 16 t + 4 lq + i for pos = (D/4) lq + 4 t + i.
#pragma unroll
  for (int c = 0; c < kEpl / 4; ++c) {
    const int pos = kEpl * j + 4 * c;
    const int dim = 16 * ((pos % (D / 4)) / 4) + 4 * (pos / (D / 4));
    f32x4 v = {acc[4 * c] * inv, acc[4 * c + 1] * inv, acc[4 * c + 2] * inv, acc[4 * c + 3] * inv};
    if (any_nan) v = f32x4{q, q, q, q};
    *reinterpret_cast<f32x4*>(orow + dim) = v;
  }
}

template <int D, int KV>
static hipError_t launch_attn_t(const AttnParams& p, int grid, hipStream_t stream) {
  if (p.two_windows)
    hipLaunchKernelGGL((attn_kernel<D, KV, true>), dim3(grid), dim3(kThreads), 0, stream, p);
  else
    hipLaunchKernelGGL((attn_kernel<D, KV, false>), dim3(grid), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_merge(const MergeParams& p, int head_dim, int kv_kind, hipStream_t stream) {
  const int rows = p.num_seqs * p.hq;
  if (rows <= 0) return hipSuccess;
  const bool f16 = kv_kind != kKvF32;
  if (rows <= kMergeRowKernelMaxRows) {
    const int per = kThreads / (head_dim / 2);
    const int blocks = (rows + per - 1) / per;
    if (head_dim == 128) {
      if (f16)
        hipLaunchKernelGGL((merge_row_kernel<128, true>), dim3(blocks), dim3(kThreads), 0, stream, p);
      else
        hipLaunchKernelGGL((merge_row_kernel<128, false>), dim3(blocks), dim3(kThreads), 0, stream, p);
    } else {
      if (f16)
        hipLaunchKernelGGL((merge_row_kernel<64, true>), dim3(blocks), dim3(kThreads), 0, stream, p);
      else
        hipLaunchKernelGGL((merge_row_kernel<64, false>), dim3(blocks), dim3(kThreads), 0, stream, p);
    }
    return hipGetLastError();
  }
  const int per = kMergeThreads / kMergeLanes;  // rows per workgroup
  const int blocks = (rows + per - 1) / per;
  if (head_dim == 128) {
    if (f16)
      hipLaunchKernelGGL((merge_kernel<128, true>), dim3(blocks), dim3(kMergeThreads), 0, stream, p);
    else
      hipLaunchKernelGGL((merge_kernel<128, false>), dim3(blocks), dim3(kMergeThreads), 0, stream, p);
  } else {
    if (f16)
      hipLaunchKernelGGL((merge_kernel<64, true>), dim3(blocks), dim3(kMergeThreads), 0, stream, p);
    else
      hipLaunchKernelGGL((merge_kernel<64, false>), dim3(blocks), dim3(kMergeThreads), 0, stream, p);
  }
  return hipGetLastError();
}

hipError_t launch_attn(const AttnParams& p, int grid, int head_dim, int kv_kind, hipStream_t stream) {
  if (grid <= 0) return hipSuccess;
  if (head_dim == 128) {
    if (kv_kind == kKvBf16) return launch_attn_t<128, kKvBf16>(p, grid, stream);
    if (kv_kind == kKvFp8) return launch_attn_t<128, kKvFp8>(p, grid, stream);
    return launch_attn_t<128, kKvF32>(p, grid, stream);
  }
  if (kv_kind == kKvBf16) return launch_attn_t<64, kKvBf16>(p, grid, stream);
  if (kv_kind == kKvFp8) return launch_attn_t<64, kKvFp8>(p, grid, stream);
  return launch_attn_t<64, kKvF32>(p, grid, stream);
}

// ---- scratch of the allocation-free entry point ----------------------------
// Partial softmax states of one prefix-attention call for callers that cannot
// allocate device memory. The array is part of the code object: every GPU
// the library runs on holds its own copy, at its own address, until the
// process ends. In host code the name `scratch` is only a stand-in; the
// device address comes from hipGetSymbolAddress, looked up once per device
// with that device current.
constexpr size_t kScratchBytes = size_t{64} << 20;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kScratchMaxDevices = 64;

hipError_t scratch_buffer(void** ptr, size_t* bytes) {
  static std::mutex mu;
  static void* dev_ptr[kScratchMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kScratchMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!dev_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    dev_ptr[dev] = p;
  }
  *ptr = dev_ptr[dev];
  *bytes = kScratchBytes;
  return hipSuccess;
}

}  // namespace tts

#ifdef TTS_PROFILE_UNITS
extern "C" int tts_prof_read(uint64_t* host, int n) {
  if (n > tts::kProfSlots) n = tts::kProfSlots;
  return static_cast<int>(hipMemcpyFromSymbol(host, HIP_SYMBOL(tts::g_prof), sizeof(uint64_t) * 8 * n, 0,
                                              hipMemcpyDeviceToHost));
}
extern "C" int tts_prof_clear() {
  static uint64_t zeros[tts::kProfSlots][8];
  return static_cast<int>(hipMemcpyToSymbol(HIP_SYMBOL(tts::g_prof), zeros, sizeof(zeros), 0, hipMemcpyHostToDevice));
}
#endif
