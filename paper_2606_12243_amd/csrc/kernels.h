// Launch wrappers of the device kernels (host side declarations).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace via {

// P[split] = X W^T (or, with `lm`, the head's per-tile row statistics).
struct GemmArgs {
  const void* X;       // activation fragments (afrag_group), MBn row blocks
  int MBn;
  const void* W;       // [N, K] weights (model dtype)
  int M, K, N;
  int ksplit;          // K slices, each written as its own partial tile
  float* part;         // [ksplit][M][N] fp32 partial products
  // head statistics (split 1)
  const LmRow* lm;
  float* lm_part;      // [tiles][M][4]
  float inv_T;
  float* logits;       // nullable [*, V] fp32, row = LmRow::out
  float* draft_logit;
};

// Projection a GEMM computes.  Each has its own kernel entry point; the QKV
// input carries 3 bf16 terms per fp32 activation, the others 2; the head
// reduces its tiles to row statistics instead of writing partials.
enum class GemmRole { kQkv, kO, kGateUp, kDown, kHead };
// e0/e1 (both or neither): timing events recorded at the kernel's own start
// and end.
void launch_gemm(bool bf16, GemmRole role, const GemmArgs& a, hipStream_t s, hipEvent_t e0 = nullptr,
                 hipEvent_t e1 = nullptr);
// Column tiles (256 wide) of an N-column GEMM.
int gemm_tiles(int N);
// Rows per GEMM work-group for M rows (16, 32, 48 or 64).
int gemm_rows_per_group(int M);
// Rows of the activation fragments for M rows: M padded to a multiple of
// gemm_rows_per_group(M); non-decreasing in M.
int gemm_padded_rows(int M);
// Row-major [rows, cols] -> packed weight tiles (see include/via.h).
void launch_pack(bool bf16, const void* src, void* dst, int rows, int cols, hipStream_t s);

// X[m] += sum_s P[s][m] (split order; P may be null); the RMSNorm of the row
// times g is written as activation fragments (`terms` bf16 terms, or fp32),
// to fragment row rows[m].lm when `rows` is given (rows with lm < 0 skipped).
void launch_resid_norm(bool bf16, int terms, float* X, const float* P, int ksplit, int M, int d, const void* g,
                       float eps, void* Y, int MBn, const RowInfo* rows, hipStream_t s);
// h[m, f] = silu(sum_s P[s][m][f]) * sum_s P[s][m][F + f], as fragments.
void launch_swiglu(bool bf16, const float* P, int ksplit, int M, int F, void* H, int MBn, hipStream_t s);
// Sum QKV partials, rotate-half RoPE at each row's position, Q -> fp32
// buffer, K/V -> the paged cache (model dtype).
struct QkvArgs {
  const float* P;
  int ksplit, M, H, KVH, hd;
  float theta;
  const RowInfo* rows;
  const SeqInfo* seqs;
  const int32_t* btab;
  uint16_t* q_hi;      // [M, H, hd] bf16 hi terms of Q (fp32 models: Q itself, as float)
  uint16_t* q_lo;      // [M, H, hd] bf16 lo terms (unused for fp32 models)
  void* pool;
  int pool_blocks, layer_slot;
};
void launch_qkv_finish(bool bf16, const QkvArgs& a, hipStream_t s);

// Head statistics: combine the per-tile partials of every head row.
void launch_lm_finalize(const LmRow* lm, const float* lm_part, int n_lm, int ntiles, float inv_T,
                        int32_t* row_argmax, float* row_max, float* row_sumexp, float* row_gap,
                        hipStream_t s);

// Embedding gather into the fp32 residual stream.
void launch_embed(bool bf16, const void* E, const RowInfo* rows, int M, int d, float* X, hipStream_t s);

struct AttnArgs {
  const void* q_hi;        // [M, H, hd] bf16 hi terms of Q (fp32 models: fp32 Q)
  const uint16_t* q_lo;    // [M, H, hd] bf16 lo terms
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
  void* out;               // activation fragments of [M, H * hd] (2 bf16 terms, or fp32)
  int MBn;
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
