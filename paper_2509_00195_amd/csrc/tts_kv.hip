// KV-cache maintenance around the decode step: appending each beam's new
// token to its block (with the fp8 block-scale policy) and copying blocks
// for copy-on-write beam duplication.
//
// A decode step of the search writes one token per beam into the paged
// cache before attention reads it (the current token is part of seq_len),
// and a duplicated beam shares its parent's full blocks while its partially
// filled last block is copied (DuplicateThenTruncate, Sec. 3.1 and Alg. 1;
// the duplicates' speculative tokens are truncated, Sec. 4.1).
#include <hip/hip_runtime.h>

#include <cstdint>

namespace tts {
namespace {

constexpr int kKvThreads = 256;
constexpr int kSlots = 16;  // tokens per block

// Round-to-nearest-even OCP E4M3FN encoding of an fp32 value (already
// divided by its block scale), saturating at +-448 (code 0x7E); NaN gives
// 0x7F. Built from the format: subnormals are multiples of 2^-9 below 2^-6,
// normals keep 3 mantissa bits of the fp32 significand.
__device__ __forceinline__ uint32_t e4m3_encode(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const uint32_t sign = (u >> 24) & 0x80u;
  const float a = __builtin_fabsf(x);
  if (a != a) return 0x7Fu;
  if (a >= 448.f) return sign | 0x7Eu;
  if (a < 0.015625f) {  // 2^-6: subnormal codes q * 2^-9, q in [0, 8]
    const uint32_t q = static_cast<uint32_t>(__builtin_rintf(a * 512.f));  // exact scaling, RNE
    return sign | q;
  }
  const uint32_t ua = __builtin_bit_cast(uint32_t, a);
  int e = static_cast<int>(ua >> 23) - 127;  // -6 .. 8
  uint32_t keep = (ua >> 20) & 7u;
  const uint32_t rest = ua & 0xFFFFFu;
  if (rest > 0x80000u || (rest == 0x80000u && (keep & 1u))) ++keep;
  if (keep == 8u) {
    keep = 0;
    ++e;
  }
  return sign | (static_cast<uint32_t>(e + 7) << 3) | keep;
}

__device__ __forceinline__ float e4m3_decode(uint32_t code) {
  return __builtin_amdgcn_cvt_f32_fp8(static_cast<int>(code), 0);  // exact
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __builtin_bit_cast(float, static_cast<uint32_t>(b) << 16);
}

__device__ __forceinline__ float block_max(float v, float* red) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  const int w = threadIdx.x >> 6;
  __syncthreads();  // red is free (a previous reduction is done with it)
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float m = red[0];
  for (int i = 1; i < kKvThreads / 64; ++i) m = fmaxf(m, red[i]);
  return m;
}

struct AppendParams {
  const void* k_new;  // [S][Hkv][D]: bf16 (bf16 and fp8 caches) or fp32
  const void* v_new;
  const int32_t* block_tables;
  const int32_t* seq_lens;
  void* k_cache;  // [NB][Hkv][16][D]
  void* v_cache;  // [NB][Hkv][D][16]
  float* k_scale;
  float* v_scale;
  int32_t max_blocks;
  int32_t num_blocks;
  int32_t hkv;
  int32_t head_dim;
};

// One tensor (K or V) of one beam's new token into an fp8 block. Element
// i = h * D + d of the token goes to `at(h, slot, d)`. The block's scale
// is set from the token when the token opens the block (slot 0); when a
// later token exceeds the range of the current scale the scale grows to
// fit it and the block's earlier codes are re-encoded under the new scale.
template <typename At>
__device__ void append_fp8(const uint16_t* src, int n, int slot, float* scale_p, At at, int D, float* red) {
  const float s_old = *scale_p;  // read ahead of the reduction's barriers, with the token
  float a = 0.f;
  for (int i = threadIdx.x; i < n; i += kKvThreads) a = fmaxf(a, __builtin_fabsf(bf16_to_f32(src[i])));
  a = block_max(a, red);
  float s = s_old;
  bool requant = false;
  if (slot == 0) {
    s = a > 0.f ? a / 448.f : 1.f;
  } else if (a > 448.f * s_old) {
    s = a / 448.f;
    requant = true;
  }
  if (requant) {
    for (int i = threadIdx.x; i < n; i += kKvThreads) {
      const int h = i / D, d = i % D;
      // All of the element's earlier codes are read first, so that their
      // loads are in flight together, then re-encoded and written.
      uint32_t old[kSlots];
#pragma unroll
      for (int j = 0; j < kSlots; ++j) old[j] = j < slot ? *at(h, j, d) : 0u;
#pragma unroll
      for (int j = 0; j < kSlots; ++j)
        if (j < slot) *at(h, j, d) = static_cast<uint8_t>(e4m3_encode(e4m3_decode(old[j]) * s_old / s));
    }
  }
  for (int i = threadIdx.x; i < n; i += kKvThreads) {
    const int h = i / D, d = i % D;
    *at(h, slot, d) = static_cast<uint8_t>(e4m3_encode(bf16_to_f32(src[i]) / s));
  }
  __syncthreads();  // every thread has read s_old
  if (threadIdx.x == 0) *scale_p = s;
}

// Two workgroups per beam, one for K and one for V (their dependent steps
// run side by side): the beam's current token (position seq_len - 1) into
// slot (seq_len - 1) % 16 of its block. Beams with seq_len 0, a block index
// past the table row or a block id outside the pool write nothing.
template <int KV>  // 0 fp32, 1 bf16, 2 fp8
__global__ __launch_bounds__(kKvThreads) void append_kernel(AppendParams p) {
  __shared__ float red[kKvThreads / 64];
  const int b = static_cast<int>(blockIdx.x >> 1);
  const bool is_v = (blockIdx.x & 1) != 0;
  const int L = p.seq_lens[b];
  if (L <= 0) return;
  const int t = L - 1;
  const int lb = t / kSlots, slot = t % kSlots;
  if (lb >= p.max_blocks) return;
  const int blk = p.block_tables[static_cast<int64_t>(b) * p.max_blocks + lb];
  if (blk < 0 || blk >= p.num_blocks) return;
  const int D = p.head_dim, n = p.hkv * D;
  const int64_t base = static_cast<int64_t>(blk) * p.hkv;  // (block, head 0)
  const int64_t src0 = static_cast<int64_t>(b) * n;
  auto k_at = [&](int h, int j, int d) { return ((base + h) * kSlots + j) * D + d; };
  auto v_at = [&](int h, int j, int d) { return ((base + h) * D + d) * kSlots + j; };
  if constexpr (KV == 0) {
    const float* src = static_cast<const float*>(is_v ? p.v_new : p.k_new) + src0;
    float* dst = static_cast<float*>(is_v ? p.v_cache : p.k_cache);
    for (int i = threadIdx.x; i < n; i += kKvThreads)
      dst[is_v ? v_at(i / D, slot, i % D) : k_at(i / D, slot, i % D)] = src[i];
  } else if constexpr (KV == 1) {
    const uint16_t* src = static_cast<const uint16_t*>(is_v ? p.v_new : p.k_new) + src0;
    uint16_t* dst = static_cast<uint16_t*>(is_v ? p.v_cache : p.k_cache);
    for (int i = threadIdx.x; i < n; i += kKvThreads)
      dst[is_v ? v_at(i / D, slot, i % D) : k_at(i / D, slot, i % D)] = src[i];
  } else if (!is_v) {
    uint8_t* kc = static_cast<uint8_t*>(p.k_cache);
    append_fp8(static_cast<const uint16_t*>(p.k_new) + src0, n, slot, p.k_scale + blk,
               [&](int h, int j, int d) { return kc + k_at(h, j, d); }, D, red);
  } else {
    uint8_t* vc = static_cast<uint8_t*>(p.v_cache);
    append_fp8(static_cast<const uint16_t*>(p.v_new) + src0, n, slot, p.v_scale + blk,
               [&](int h, int j, int d) { return vc + v_at(h, j, d); }, D, red);
  }
}

struct CopyParams {
  const int32_t* pairs;  // [n][2]: source, destination block
  void* k_cache;
  void* v_cache;
  float* k_scale;
  float* v_scale;
  int64_t blk_bytes;  // bytes of one block of K (all KV heads), = V's
  int32_t num_blocks;
};

// One workgroup per pair: K and V of every KV head (and the fp8 scales)
// of the source block into the destination block. Pairs naming a block
// outside the pool, or a block onto itself, copy nothing.
__global__ __launch_bounds__(kKvThreads) void copy_kernel(CopyParams p) {
  const int src = p.pairs[2 * blockIdx.x], dst = p.pairs[2 * blockIdx.x + 1];
  if (src < 0 || src >= p.num_blocks || dst < 0 || dst >= p.num_blocks || src == dst) return;
  const int64_t n16 = p.blk_bytes / 16;
  for (int c = 0; c < 2; ++c) {
    const uint4* s = reinterpret_cast<const uint4*>(static_cast<const unsigned char*>(c ? p.v_cache : p.k_cache) +
                                                    src * p.blk_bytes);
    uint4* d = reinterpret_cast<uint4*>(static_cast<unsigned char*>(c ? p.v_cache : p.k_cache) + dst * p.blk_bytes);
    for (int64_t i = threadIdx.x; i < n16; i += kKvThreads) d[i] = s[i];
  }
  if (threadIdx.x == 0 && p.k_scale) {
    p.k_scale[dst] = p.k_scale[src];
    p.v_scale[dst] = p.v_scale[src];
  }
}

}  // namespace

hipError_t launch_append(const void* k_new, const void* v_new, const int32_t* block_tables, const int32_t* seq_lens,
                         void* k_cache, void* v_cache, float* k_scale, float* v_scale, int num_seqs, int max_blocks,
                         int num_blocks, int hkv, int head_dim, int kv_kind, hipStream_t stream) {
  if (num_seqs <= 0) return hipSuccess;
  AppendParams p{k_new, v_new, block_tables, seq_lens, k_cache, v_cache, k_scale, v_scale,
                 max_blocks, num_blocks, hkv, head_dim};
  if (kv_kind == 0)
    hipLaunchKernelGGL(append_kernel<0>, dim3(2 * num_seqs), dim3(kKvThreads), 0, stream, p);
  else if (kv_kind == 1)
    hipLaunchKernelGGL(append_kernel<1>, dim3(2 * num_seqs), dim3(kKvThreads), 0, stream, p);
  else
    hipLaunchKernelGGL(append_kernel<2>, dim3(2 * num_seqs), dim3(kKvThreads), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_copy_blocks(const int32_t* pairs, int num_pairs, void* k_cache, void* v_cache, float* k_scale,
                              float* v_scale, int64_t blk_bytes, int num_blocks, hipStream_t stream) {
  if (num_pairs <= 0) return hipSuccess;
  CopyParams p{pairs, k_cache, v_cache, k_scale, v_scale, blk_bytes, num_blocks};
  hipLaunchKernelGGL(copy_kernel, dim3(num_pairs), dim3(kKvThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace tts
