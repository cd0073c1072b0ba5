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
  // gate/up projection (kGateUp): W packed with gate and up rows interleaved
  // by 8 (N = 2 F); the SwiGLU product is written as 2-term fragments of
  // [M, F] to H.  Each work-group owns `nb` 16-column blocks over all of K.
  void* H;
  int F;
  int nb;
  // RMSNorm of the input rows (gate/up and head): output row m is multiplied
  // by row_scale(ss, ss_stride, m, K, eps)
  const float* ss;
  int ss_stride;
  float eps;
};

// Projection a GEMM computes.  Each has its own kernel entry point; the QKV
// input carries kQkvTerms bf16 terms per fp32 activation, the others 2; the head
// reduces its tiles to row statistics instead of writing partials; the
// gate/up projection runs over all of K and applies SwiGLU itself.
enum class GemmRole { kQkv, kO, kGateUp, kDown, kHead };
// bf16 terms per fp32 activation at the QKV projection's input (the others take 2).
constexpr int kQkvTerms = 2;
// e0/e1 (both or neither): timing events recorded at the kernel's own start
// and end.
void launch_gemm(bool bf16, GemmRole role, const GemmArgs& a, hipStream_t s, hipEvent_t e0 = nullptr,
                 hipEvent_t e1 = nullptr);
// Forwards of more rows than this run their projections (bf16 models) on the
// compute-bound prefill GEMM, which writes one partial (ksplit must be 1).
// Below it the weight-streaming GEMMs, at most 4 passes of 128-row groups
// over the weights, cost less than 256 x 256 tiles too few to fill the GPU.
constexpr int kPrefillMinRows = 512;
bool gemm_is_prefill(bool bf16, int M);
// Plain bf16 product a.part[M, N] = X[M, K] W[N, K]^T (one activation term)
// on the prefill GEMM.
void launch_gemm_bf16(const GemmArgs& a, hipStream_t s);
// Column tiles (256 wide) of an N-column GEMM.
int gemm_tiles(int N);
// QKV, O and down projections of forwards of up to 32 rows (bf16 models, N a
// multiple of 16) run on the K-interleaved split-K kernel, whose work-groups
// own a.nb 16-column blocks of one of a.ksplit K splits; gemm_ki_plan picks
// both for an [N, K] weight (about 256 work-groups).
bool gemm_uses_ki(GemmRole role, int M, int N);
void gemm_ki_plan(int N, int K, int* nb, int* ksplit);
// Rows per GEMM work-group for M rows (16, 32, 48, 64, 96 or 128).
int gemm_rows_per_group(int M);
// Rows of the activation fragments for M rows: M padded to a multiple of
// gemm_rows_per_group(M); non-decreasing in M.
int gemm_padded_rows(int M);
// Row-major [rows, cols] -> packed weight tiles (see include/via.h).  With
// ffn > 0 the source is [2 ffn, cols] (gate rows, then up rows) and packed
// row 16 b + i takes gate row 8 b + i (i < 8) or up row 8 b + i - 8.
void launch_pack(bool bf16, const void* src, void* dst, int rows, int cols, int ffn, hipStream_t s);
// 16-column blocks per gate/up work-group for d_ffn = F (1..8, about one
// work-group per compute unit).
int gate_up_blocks_per_group(int F);

// X[m] += sum_s P[s][m] (split order; P may be null); x * g is written as
// activation fragments (`terms` bf16 terms, or fp32), to fragment row
// rows[m].lm when `rows` is given (rows with lm < 0 skipped), and the sums of
// x^2 over column chunks to ss[chunk * ss_stride + row]: the consumer of the
// next projection multiplies its output row by row_scale() (RMSNorm).
// Xcopy (nullable): the updated rows are also stored there, row m to row
// erows[m].xs when erows is given (skipped where xs < 0), else to row m.
// E (nullable, model dtype [vocab, d]): X[m] is first set to the embedding
// row of token erows[m].tok (P is then ignored).
void launch_resid_add(bool bf16, int terms, float* X, const float* P, int ksplit, int M, int d, const void* g,
                      void* Y, int MBn, const RowInfo* rows, float* ss, int ss_stride, hipStream_t s,
                      float* Xcopy = nullptr, const void* E = nullptr, const RowInfo* erows = nullptr);

struct PrefixArgs {
  const PrefixXfer* xfer;  // [M]
  int M, P, d, KVH, hd;
  const float* xstate;     // [rows][d]: residual streams after layer P - 1
  float* X;                // the forward's residual stream [M, d]
  const void* src_pool;    // K/V of layers 0..P-1 are read here ...
  int src_blocks;
  void* dst_pool;          // ... and written here
  int dst_blocks;
};
// K/V of layers 0..P-1 copied src -> dst cache at every row's position and
// X[m] = xstate[xfer[m].src_row] (a verify step's full forward: slim -> full
// from the state ring; a prefill's slim forward: full -> slim from the full
// forward's saved rows).
void launch_prefix_copy(bool bf16, const PrefixArgs& a, hipStream_t s);

// DIMR routing cost per row (Eq. 11): q = full verifier logits, p = routed
// slim verifier logits, both [rows][ld] fp32 (first `vocab` entries used).
struct DimrArgs {
  const float* q;
  const float* p;
  int rows, vocab, ld;
  float inv_T, log_1m_alpha, log_beta;
  float* cost;  // [rows]
};
void launch_dimr_cost(const DimrArgs& a, hipStream_t s);
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
  const float* ss;     // RMSNorm sums of squares of the input rows (row_scale)
  int ss_stride, d;
  float eps;
};
void launch_qkv_finish(bool bf16, const QkvArgs& a, hipStream_t s);

// Head statistics: combine the per-tile partials of every head row.
void launch_lm_finalize(const LmRow* lm, const float* lm_part, int n_lm, int ntiles, float inv_T,
                        int32_t* row_argmax, float* row_max, float* row_sumexp, float* row_gap,
                        hipStream_t s);

struct AttnArgs {
  const void* q_hi;        // [M, H, hd] bf16 hi terms of Q (fp32 models: fp32 Q)
  const uint16_t* q_lo;    // [M, H, hd] bf16 lo terms
  const void* pool;
  int pool_blocks, layer_slot;
  const RowInfo* rows;
  const SeqInfo* seqs;
  const int32_t* btab;
  const AttnItem* items;
  int n_items, max_chunks; // max_chunks: most splits of any item (grid x)
  int span;                // keys per split (a multiple of 32)
  int M, H, KVH, hd;
  float scale;             // 1/sqrt(hd)
  float* part_o;           // [split][M][H][hd]
  float* part_ml;          // [split][M][H][2]: max (log2 units), sum
  void* out;               // activation fragments of [M, H * hd] (2 bf16 terms, or fp32)
  int MBn;
  int direct;              // set by launch_attention: every item has one split, whose work-group writes `out`
};
void launch_attention(bool bf16, const AttnArgs& a, hipStream_t s);

// Tree compaction: KvMove (plan.h) copies K/V of slot src -> dst for every layer slot.
void launch_kv_moves(bool bf16, void* pool, int pool_blocks, int n_slots, int KVH, int hd,
                     const int32_t* btab, const KvMove* moves, int n_moves, hipStream_t s);

// A sampled token the decision still owes (kind 1: slim-tier rewrite from
// q', kind 2: residual of a rejected escalated draft; 0: none).
// The vocabulary is cut into at most this many slices for the draw.
constexpr int kSampleSlices = 64;
struct SampleReq {
  int32_t kind, out, j;
  float u;
};

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
  // sampling rules (chain drafts; draft_probs null: greedy rules)
  const float* draft_probs;   // [batch * max_drafts * vocab] drafter distributions
  const float* u;             // [batch * max_drafts * 3] uniforms: accept, slim sample, residual sample
  const float* s_logits;      // [batch * max_rows * vocab]
  const float* f_logits;      // same, full verifier (null on the first pass)
  const float* s_row_sumexp;
  const float* f_row_sumexp;
  float alpha, beta;
  int vocab;
  SampleReq* req;             // [batch]
  double* slice_sum;          // [batch * kSampleSlices * 2] per-slice weight sums
  int32_t* tok_out;           // drawn tokens [batch]; null: the decision's emit slots
  int32_t* h_packed;          // nullable: device address of the pinned host mirror of `packed`,
                              // written by the greedy decision itself (system-scope stores)
};
// Decision kernel, then (sampling rules) the sampling kernel that fills the
// emitted tokens it left open.
void launch_decide(const DecideArgs& a, hipStream_t s);
// Draws of the requests in a.req (kind 1 over a.s_logits rows) into
// a.tok_out; with probs, also writes each request row's softmax
// exp((l - max) / T) / s_row_sumexp as probs[i * probs_ld + v].
void launch_sample_rows(const DecideArgs& a, float* probs, int probs_ld, hipStream_t s);
// The same draws with the requests passed as kernel arguments and the
// request array and slice sums in the library's static device scratch
// (n <= kStaticSampleRows); `scratch` is the address static_scratch gave.
constexpr int kStaticSampleRows = 64;
void launch_sample_rows_static(DecideArgs a, const SampleReq* req, int n, void* scratch, float* probs,
                               int probs_ld, hipStream_t s);
// Device address and size of the static scratch on the current device
// (looked up once per device).
hipError_t static_scratch(void** ptr, size_t* bytes);

}  // namespace via
