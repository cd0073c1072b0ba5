// Shared device helpers and the plan structures the host uploads per call.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace via {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 16;        // tokens per KV page
constexpr int kMaxChildren = 8;   // drafts verified by one row
constexpr int kAttnChunk = 128;   // keys per attention work-group (split-KV chunk)

// One fed row of a forward (lag row or window row).
struct RowInfo {
  int32_t tok;      // token id
  int32_t pos;      // RoPE position
  int32_t seq;      // index into the SeqInfo array of this forward
  int32_t slot;     // cache slot the row's K/V are written to
  int32_t vis_len;  // slots [0, vis_len) are visible
  int32_t lm;       // index into the head rows, -1 if the row has no head output
  uint64_t mask;    // extra visible slots win_base + bit (tree rows)
};

struct SeqInfo {
  int32_t kv_len;     // slots written after the forward's K/V write
  int32_t row_start;  // first row of this sequence in the forward
  int32_t n_rows;     // rows of this sequence (lag + window)
  int32_t win_base;   // slot of window row 0 (tree masks are relative to it)
  int32_t bt;         // offset of the block table in the uploaded tables
  int32_t n_blocks;   // block-table length
  int32_t pad0, pad1;
};

// One attention work item: a tile of 32 (row, head-in-group) queries of a sequence.
struct AttnItem {
  int32_t seq;
  int32_t q0;       // first query (row * G + g) of the tile, within the sequence
  int32_t n_chunks; // key chunks of this sequence
  int32_t pad;
};

// Head row: which forward row and where its statistics go.
struct LmRow {
  int32_t row;      // forward row
  int32_t out;      // b * max_rows + r in the caller's output arrays
  int32_t n_drafts; // drafts this row verifies (<= kMaxChildren)
  int32_t pad;
  int32_t draft_idx[kMaxChildren];  // b * max_drafts + j
  int32_t draft_tok[kMaxChildren];
};

// Per-sequence data of an open step, read by the tier decision.
struct StepSeq {
  int32_t n;          // committed length before the step
  int32_t n_drafts;
  int32_t full_ran;   // full forward ran this step
  int32_t pad;
};

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

// Element offset of K[layer_slot][block][g][t][i]
__device__ __forceinline__ size_t k_off(int slot, int block, int nblk, int kvh, int hd, int g, int t, int i) {
  return ((((size_t)slot * nblk + block) * 2 + 0) * kvh + g) * (size_t)(kBlock * hd) + (size_t)t * hd + i;
}
// Element offset of V[layer_slot][block][g][i][t] (transposed page)
__device__ __forceinline__ size_t v_off(int slot, int block, int nblk, int kvh, int hd, int g, int t, int i) {
  return ((((size_t)slot * nblk + block) * 2 + 1) * kvh + g) * (size_t)(kBlock * hd) + (size_t)i * kBlock + t;
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
