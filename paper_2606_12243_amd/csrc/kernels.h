// Launch wrappers of the device kernels (host side declarations).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace via {

enum Epi { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_STATS = 3 };

// Y = X W^T over one 64-column tile per work-group, K split across the
// group's four waves and `ksplit` groups; the fused epilogue consumes the
// reduced tile.
struct GemmArgs {
  const void* X;       // [M, ldx] activations (model dtype)
  int ldx;
  const void* W;       // [rows, K] weights (model dtype)
  int M, K, N;         // N: valid output columns of the plain column mapping
  int ntiles;          // 64-column tiles
  int ksplit;          // work-groups per tile along K
  float* part;         // split-K partial tiles [ksplit][M][ntiles * 64]
  int* counters;       // one per (m-group, tile); self-resetting
  // QKV: RoPE, Q store, paged K/V write
  const RowInfo* rows;
  const SeqInfo* seqs;
  const int32_t* btab;
  void* q_out;         // [M, H, hd]
  void* pool;          // cache pool base
  int pool_blocks, layer_slot;
  int H, KVH, hd;
  float theta;
  // RESID: resid[m, col] += y
  float* resid;
  // SWIGLU: h_out[m, f] = silu(gate) * up
  void* h_out;
  int F;
  // STATS: per (tile, head row) partial max / second / sum-exp / argmax
  const LmRow* lm;
  float* lm_part;      // [ntiles][M][4]
  float inv_T;
  float* logits;       // nullable [*, V] fp32, row = LmRow::out
  float* draft_logit;
};

void launch_gemm(int epi, bool bf16, const GemmArgs& a, hipStream_t s);

// Head statistics: combine the per-tile partials of every head row.
void launch_lm_finalize(const LmRow* lm, const float* lm_part, int n_lm, int ntiles, float inv_T,
                        int32_t* row_argmax, float* row_max, float* row_sumexp, float* row_gap,
                        hipStream_t s);

// Embedding gather into the fp32 residual stream.
void launch_embed(bool bf16, const void* E, const RowInfo* rows, int M, int d, float* X, hipStream_t s);
// RMSNorm of rows (optionally gathered through head rows) into the model dtype.
void launch_rmsnorm(bool bf16, const float* X, const void* g, int M, int d, float eps, void* Y,
                    const LmRow* gather, hipStream_t s);

struct AttnArgs {
  const void* q;           // [M, H, hd]
  const void* pool;
  int pool_blocks, layer_slot;
  const RowInfo* rows;
  const SeqInfo* seqs;
  const int32_t* btab;
  const AttnItem* items;
  int n_items, max_chunks;
  int M, H, KVH, hd;
  float scale;             // 1/sqrt(hd)
  float* part_o;           // [max_chunks][M][H][hd]
  float* part_ml;          // [max_chunks][M][H][2]
  void* out;               // [M, H * hd] model dtype
};
void launch_attention(bool bf16, const AttnArgs& a, hipStream_t s);

// Tree compaction: copy K/V of slot src -> dst for every layer slot.
struct KvMove {
  int32_t bt;      // offset of the block table in btab
  int32_t src, dst;
  int32_t pad;
};
void launch_kv_moves(bool bf16, void* pool, int pool_blocks, int n_slots, int KVH, int hd,
                     const int32_t* btab, const KvMove* moves, int n_moves, hipStream_t s);

struct DecideArgs {
  const StepSeq* seqs;
  int batch, max_rows, max_drafts;
  const int32_t* draft_tok;     // [batch * max_drafts]
  const int32_t* draft_row;
  const int32_t* draft_parent;
  const float* s_row_max;
  const int32_t* s_row_argmax;
  const float* s_draft_logit;
  const float* f_row_max;       // null on the first pass
  const int32_t* f_row_argmax;
  const float* f_draft_logit;
  float tau_acc, tau_full, inv_T;
  int forced;
  int8_t* tier;
  float* conf;
  int32_t* packed;
};
void launch_decide(const DecideArgs& a, hipStream_t s);

}  // namespace via
