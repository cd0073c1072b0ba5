// Shared device helpers and the plan structures the host uploads per call.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "plan.h"

namespace via {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x7FFFFFu)) return (uint16_t)((u >> 16) | 0x40);  // NaN
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename T> __device__ __forceinline__ float to_f(T v);
template <> __device__ __forceinline__ float to_f<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f<uint16_t>(uint16_t v) { return bf2f(v); }

template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ uint16_t from_f<uint16_t>(float v) { return f2bf(v); }

// Paged cache addressing (see include/via.h): pool[slot][block][K|V][kvh][...]
struct PoolRef {
  void* base;
  int32_t n_blocks;
  int32_t kvh, hd;
};

__device__ __forceinline__ size_t page_elems(int kvh, int hd) { return (size_t)kvh * kBlock * hd; }

// Pool layout: [layer_slot][kv_head g][block][K page | V page].  A KV
// head's pages of consecutive blocks are adjacent, so attention over a
// sequence whose blocks were allocated in order streams one contiguous
// region per (layer, head).
// Element offset of K token t, dim i.  K pages are dim-group-major,
// [hd/8][16 tokens][8]: the 16-byte pieces of one dim group of a page's 16
// tokens are contiguous, so an MFMA operand load of 16 tokens x 8 dims reads
// 256 contiguous bytes.
__device__ __forceinline__ size_t k_off(int slot, int block, int nblk, int kvh, int hd, int g, int t, int i) {
  return ((((size_t)slot * kvh + g) * nblk + block) * 2 + 0) * (size_t)(kBlock * hd) +
         ((size_t)(i >> 3) * kBlock + t) * 8 + (i & 7);
}
// Element offset of V token t, dim i: the V page is transposed, [hd][16 tokens]
__device__ __forceinline__ size_t v_off(int slot, int block, int nblk, int kvh, int hd, int g, int t, int i) {
  return ((((size_t)slot * kvh + g) * nblk + block) * 2 + 1) * (size_t)(kBlock * hd) + (size_t)i * kBlock + t;
}

// Activation fragments: the GEMM input X [M, K] as the matrix cores read it.
// Rows are padded to Mp (a multiple of 16 per work-group m-block count);
// S = K / 32 steps, MBn = Mp / 16 row blocks.  Each fp32 value is stored as
// NT bf16 terms (hi [, mid], lo: hi and mid truncated, the last rounded to
// nearest) for bf16 models, or as itself (NT = 1) for fp32 models.  The 8
// consecutive columns k0 .. k0+7 (k0 % 8 == 0) of row m form one group:
//   group(q, m, k0) = ((q * S + k0/32) * MBn + m/16) * 64 + ((k0%32)/8) * 16 + m%16
// so the 64 lanes of a wave read one 16-row x 32-column step of one term as
// a single contiguous block.
__device__ __forceinline__ size_t afrag_group(int q, int m, int k0, int S, int MBn) {
  return (((size_t)q * S + (k0 >> 5)) * MBn + (m >> 4)) * 64 + ((k0 & 31) >> 3) * 16 + (m & 15);
}

__device__ __forceinline__ uint32_t pack_bf16x2(uint32_t lo16, uint32_t hi16) {
  return (lo16 & 0xFFFFu) | (hi16 << 16);
}

template <int NT>
__device__ __forceinline__ void store_afrag(uint16_t* base, int m, int k0, const float* v, int S, int MBn) {
  uint32_t t[NT][8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    float r = v[e];
#pragma unroll
    for (int q = 0; q < NT; ++q) {
      const uint32_t b = (q == NT - 1) ? (uint32_t)f2bf(r) : (__float_as_uint(r) >> 16);
      t[q][e] = b;
      r = r - __uint_as_float(b << 16);
    }
  }
#pragma unroll
  for (int q = 0; q < NT; ++q)
    ((uint4*)base)[afrag_group(q, m, k0, S, MBn)] =
        make_uint4(pack_bf16x2(t[q][0], t[q][1]), pack_bf16x2(t[q][2], t[q][3]), pack_bf16x2(t[q][4], t[q][5]),
                   pack_bf16x2(t[q][6], t[q][7]));
}

__device__ __forceinline__ void store_afrag_f32(float* base, int m, int k0, const float* v, int S, int MBn) {
  float4* g = (float4*)(base + afrag_group(0, m, k0, S, MBn) * 8);
  g[0] = make_float4(v[0], v[1], v[2], v[3]);
  g[1] = make_float4(v[4], v[5], v[6], v[7]);
}

// Store 8 activations of row m, columns k0.. in the model's fragment form.
template <bool BF16, int NT>
__device__ __forceinline__ void put_afrag(void* base, int m, int k0, const float* v, int S, int MBn) {
  if constexpr (BF16)
    store_afrag<NT>((uint16_t*)base, m, k0, v, S, MBn);
  else
    store_afrag_f32((float*)base, m, k0, v, S, MBn);
}

// RMSNorm scale of row m, 1/sqrt(mean(x^2) + eps), from the per-chunk sums
// of squares ss[c * stride + m], c < ceil(d / kNormChunk), added in chunk
// order.
__device__ __forceinline__ float row_scale(const float* ss, int stride, int m, int d, float eps) {
  float t = 0.f;
  const int nch = (d + kNormChunk - 1) / kNormChunk;
  for (int c = 0; c < nch; ++c) t += ss[(size_t)c * stride + m];
  return 1.0f / sqrtf(t / (float)d + eps);
}

__device__ __forceinline__ float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace via
