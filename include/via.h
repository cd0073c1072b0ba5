/*
 * via.h — C ABI of the VIA-SD verification step on gfx950 (MI355X).
 *
 * The verification step of "VIA-SD: Verification via Intra-Model Routing
 * for Speculative Decoding" (arXiv 2606.12243): one batched forward of a
 * decoder-only verifier over a k-token draft window against its KV cache,
 * run as the full verifier q or as the slim-verifier q' = Pi_z(q) (the layers
 * the routing mask z retains, sharing q's weights, embedding and head;
 * Sec. 3.3 and Sec. 3.2), then a per-position confidence and a three-tier
 * decision (accept / slim rewrite / escalate to q; regions B.1-B.3 of
 * App. B.2), the gate walk and longest accepted prefix (Alg. 1, App. B.1,
 * Sec. 3.4 Steps 3-4), and the KV commit/rollback of the accepted positions.
 *
 * Conventions
 *  - Every pointer documented "device" is caller-owned device memory that
 *    must outlive the handle using it; the library never allocates or frees
 *    device memory.  "host" pointers are read (or written) before the call
 *    returns unless stated otherwise; "pinned host" pointers are written by
 *    an asynchronous copy and are valid once the caller has synchronised the
 *    stream.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Calls enqueue work and return; apart from via_step, which drives a
 *    whole step and waits for its decisions, the library never synchronises.
 *  - Handles are single-stream and not thread-safe.
 *  - Every argument is validated before any work is enqueued.  A non-OK
 *    return leaves model and KV state unchanged; via_last_error() gives a
 *    thread-local message.
 *  - Token ids are int32 in [0, vocab).  Weights are row-major
 *    [out_features, in_features] in the model dtype (fp32 or bf16).
 */
#ifndef VIA_H
#define VIA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t via_status;
#define VIA_OK 0
#define VIA_EINVAL (-1)       /* bad argument: null pointer, size, id, ordering */
#define VIA_ENOMEM (-2)       /* KV block pool (or workspace sizing) exhausted */
#define VIA_EDEVICE (-3)      /* a HIP call failed; sticky for the handle */
#define VIA_ESTATE (-4)       /* call out of order or inconsistent with KV state */
#define VIA_EUNSUPPORTED (-5) /* shape/dtype this build does not run */

#define VIA_DTYPE_F32 0
#define VIA_DTYPE_BF16 1

#define VIA_CACHE_FULL 0
#define VIA_CACHE_SLIM 1

#define VIA_TIER_ACCEPT 0 /* region A: c >= tau_acc */
#define VIA_TIER_SLIM 1   /* region B: tau_full <= c < tau_acc */
#define VIA_TIER_FULL 2   /* region C: c < tau_full (also a non-finite c) */

#define VIA_FORCED_NONE (-1)
#define VIA_FORCED_ACCEPT 0
#define VIA_FORCED_SLIM 1
#define VIA_FORCED_FULL 2

/* Largest draft block / tree (rows with a tree mask, drafts per window). */
#define VIA_MAX_TREE_ROWS 64
#define VIA_MAX_DRAFTS 64
#define VIA_MAX_CHILDREN 8

typedef struct via_model via_model; /* opaque, library-owned host object */
typedef struct via_kv via_kv;       /* opaque, library-owned host object */

/* Verifier architecture.  Supported: head_dim 64 or 128, n_heads a multiple
 * of n_kv_heads, d_model and d_ffn multiples of 64, vocab >= 1.  The layer
 * is RMSNorm -> QKV -> rotate-half RoPE (rope_theta) -> GQA attention -> O,
 * RMSNorm -> SwiGLU FFN, each with a residual add; a final RMSNorm precedes
 * the untied output head. */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ffn, vocab;
  float rms_eps, rope_theta;
  int32_t dtype; /* VIA_DTYPE_F32 or VIA_DTYPE_BF16 */
} via_model_desc;

/* Weight pointers (device, caller-owned, model dtype).  Per-layer entries
 * are HOST arrays of n_layers device pointers, copied at via_model_create.
 * Logical shapes, [out_features, in_features]:
 *   embed     [vocab, d]          lm_head [vocab, d]      final_norm [d]
 *   attn_norm [d]                 ffn_norm [d]
 *   w_qkv     [(H + 2 KVH) hd, d]  rows: Q heads, then K heads, then V heads
 *   w_o       [d, H hd]
 *   w_gate_up [2 F, d]            rows: gate (F), then up (F)
 *   w_down    [d, F]
 * embed and the norm gains are plain row-major.  The five projection
 * matrices are in the PACKED layout, which stores each 64-row x 32-column
 * tile as the matrix cores consume it, so that the verify GEMMs stream
 * weights as contiguous memory: lm_head, w_qkv, w_o and w_down as written
 * by via_pack_weight, w_gate_up as written by via_pack_gate_up (gate and up
 * rows interleaved by 8, so that one 16-row block yields both factors of
 * eight SwiGLU outputs).
 * The slim-verifier reads the same pointers for its retained layers: no
 * weight is copied (Sec. 3.3). */
typedef struct {
  const void *embed, *lm_head, *final_norm;
  const void *const *attn_norm, *const *w_qkv, *const *w_o;
  const void *const *ffn_norm, *const *w_gate_up, *const *w_down;
} via_weights;

/* Tier parameters.  Confidence of draft d verified by row r is the ratio
 * c = q'_r(d) / max_u q'_r(u) = exp((l'_r(d) - max_u l'_r(u)) / T)
 * (App. B.2 gates q'(v) against fractions of M' = max_u q'(u));
 * tau_acc and tau_full stand for 1 - alpha_1 and 1 - alpha_2.
 * Requires 0 <= tau_full <= tau_acc (tau_acc may exceed 1) and T > 0. */
typedef struct {
  float tau_acc, tau_full, temperature;
  int32_t forced; /* VIA_FORCED_*: every tier forced (tests, baselines) */
} via_tier_params;

/* KV handle description.  Two paged caches: the full verifier's (n_layers
 * layer slots) and the slim-verifier's (one slot per retained layer, in
 * route order).  Pool layout, element type = model dtype, block_size = 16:
 *   pool[slot][kv_head][block][K|V][...]   (a head's pages of consecutive blocks adjacent)
 *   K page: [head_dim/8][16 tokens][8]    (dim groups of 8, token-major within)
 *   V page: [head_dim][16 tokens]         (transposed)
 * Cache slot p of a sequence lives in block table[p / 16], row p % 16.
 * Sizes: via_pool_bytes() and via_workspace_bytes(). */
typedef struct {
  int32_t block_size;         /* must be 16 */
  int32_t max_seqs;           /* sequence ids are in [0, max_seqs) */
  int32_t max_blocks_per_seq; /* block-table capacity per sequence */
  int32_t blocks_full, blocks_slim;
  void *pool_full, *pool_slim; /* device, 16-byte aligned */
  int32_t max_rows;   /* rows per forward (lag + window, summed over batch) */
  int32_t max_batch;  /* sequences per window */
  int32_t max_drafts; /* drafts per sequence per window, 1..VIA_MAX_DRAFTS */
  void *workspace;    /* device, >= via_workspace_bytes(...), 256-byte aligned */
  size_t workspace_bytes;
  void *pinned_staging; /* pinned host, >= via_staging_bytes(...) */
  size_t staging_bytes;
} via_kv_desc;

/* One draft window for a batch of sequences (HOST arrays, copied).
 * Row 0 of each sequence is its pending token x[n-1] (the last committed
 * token, whose K/V are not cached yet).  Chain: rows are
 * [x[n-1], d_0 .. d_{k-2}] and draft j is verified by row j (App. B.1 runs q'
 * on the prefixes x_<t .. x_<t+gamma-1).  Tree: rows are the root and every
 * draft node that has children, in node order; draft j is verified by its
 * parent's row.
 *   row_depth NULL: row r sits at RoPE position n-1+r.  Else n-1+row_depth[r].
 *   row_mask  NULL: causal over the window.  Else bit r' of row_mask[r] set
 *             iff row r attends row r' (ancestors and itself; r' <= r; at
 *             most VIA_MAX_TREE_ROWS rows).
 *   draft_parent NULL: chain (parent of draft j is j-1).  Else parent draft
 *             index (< j) or -1 for children of the root; at most
 *             VIA_MAX_CHILDREN children per node.
 *   n_lag / lag_tok: committed tokens the full cache is missing
 *             (x[valid_full .. n-2]); required by via_verify_full when the
 *             full cache lags, ignored by via_verify_slim.
 * Strides: 1 <= max_drafts <= the KV handle's max_drafts. */
typedef struct {
  int32_t batch, max_rows, max_drafts, max_lag; /* strides */
  const int32_t *seq_id;       /* [batch] distinct, attached */
  const int32_t *n_rows;       /* [batch] >= 1 */
  const int32_t *row_tok;      /* [batch * max_rows] */
  const int32_t *row_depth;    /* [batch * max_rows] or NULL */
  const uint64_t *row_mask;    /* [batch * max_rows] or NULL */
  const int32_t *n_drafts;     /* [batch] */
  const int32_t *draft_tok;    /* [batch * max_drafts] */
  const int32_t *draft_row;    /* [batch * max_drafts] */
  const int32_t *draft_parent; /* [batch * max_drafts] or NULL */
  const int32_t *n_lag;        /* [batch] or NULL (no lag rows) */
  const int32_t *lag_tok;      /* [batch * max_lag] */
} via_window;

/* Per-row statistics of one forward (device arrays written by the call).
 * Indexed by b * window.max_rows + r (window rows; lag rows produce none)
 * and b * window.max_drafts + j. */
typedef struct {
  int32_t *row_argmax; /* lowest token id among the maxima */
  float *row_max;      /* max_u l(u) */
  float *row_sumexp;   /* sum_u exp((l(u) - max) / T) */
  float *row_gap;      /* max minus the largest other logit (0 on ties); nullable */
  float *draft_logit;  /* l_{draft_row[j]}(draft_tok[j]) */
  float *logits;       /* nullable fp32 [batch * max_rows * vocab] (debug/parity) */
} via_verify_out;

/* Decision of one window.  `packed` (device) and `h_packed` (pinned host)
 * hold, for B = window.batch and D = window.max_drafts:
 *   [0, B)        status  0 resolved, 1 needs the full verifier,
 *                         2 non-finite full logits (sequence not advanced)
 *   [B, 2B)       kappa   accepted draft count
 *   [2B, 3B)      emit    token appended after the accepted drafts, -1 none
 *   [3B, 4B)      new_len committed length n' = n + kappa + (emit >= 0)
 *   [4B, 4B+B*D)  path    accepted draft indices in order (kappa entries)
 * `tier` and `conf` (device [B * D]) give every draft's tier (VIA_TIER_*)
 * and ratio confidence. */
typedef struct {
  int8_t *tier;
  float *conf;
  int32_t *packed;
  int32_t *h_packed;
} via_decision;

/* ---- weight packing ----------------------------------------------------- */
/* Bytes of a packed [rows, cols] matrix: rows rounded up to a multiple of 64
 * (padding rows are zero), cols must be a multiple of 32. 0 if invalid. */
size_t via_packed_bytes(int32_t rows, int32_t cols, int32_t dtype);
/* Pack a row-major [rows, cols] device matrix `src` into `dst` (device,
 * via_packed_bytes) on `stream`.  Element (r, c) goes to the 8-element group
 *   ((((r/64) * (cols/32) + c/32) * 4 + (r%64)/16) * 64 + ((c%32)/8) * 16 + r%16)
 * at offset c%8.  src and dst must not overlap. */
via_status via_pack_weight(const void *src, void *dst, int32_t rows, int32_t cols, int32_t dtype, void *stream);
/* Pack the FFN input projection: `src` is the row-major [2 d_ffn, d_model]
 * device matrix (gate rows, then up rows) and `dst` (device,
 * via_packed_bytes(2 d_ffn, d_model, dtype)) receives the via_pack_weight
 * layout of the row-interleaved matrix whose row 16 b + i is gate row
 * 8 b + i for i < 8 and up row 8 b + i - 8 for i >= 8.  The FFN is
 * h = silu(x W_gate^T) * (x W_up^T) (SwiGLU; the paper does not fix the
 * verifier's layer, this is the architecture reading of this library).
 * d_ffn must be a multiple of 8.  src and dst must not overlap. */
via_status via_pack_gate_up(const void *src, void *dst, int32_t d_ffn, int32_t d_model, int32_t dtype,
                            void *stream);

/* ---- prefill GEMM --------------------------------------------------------
 * C = X W^T for bf16 X [M, K] and W [N, K], fp32 accumulation and output:
 * the compute-bound tile kernel that runs every projection of a forward of
 * more than 512 rows (a prefill), exposed for measurement and tests.  (A
 * forward feeds it its fp32 activations as 2 bf16 terms, one pass each;
 * this call runs one.)
 *   X  device bf16, ceil(M/16)*16 rows, in the activation-fragment layout:
 *      element (m, k) is at 8-element group
 *      ((k/32) * ceil(M/16) + m/16) * 64 + ((k%32)/8) * 16 + m%16, offset k%8
 *      (rows past M may hold anything; they are never stored)
 *   W  device bf16 in the via_pack_weight layout of [N, K]
 *   C  device fp32 [M, N] row-major, written
 * K must be a multiple of 32.  Asynchronous on `stream`. */
via_status via_gemm_bf16(const void *X, const void *W, float *C, int32_t M, int32_t N, int32_t K, void *stream);

/* Routing-mask cost of DIMR (Sec. 3, Eqs. 9-12): for every row r, with
 * l_q = log softmax(q_logits[r] / T) (the full verifier q) and
 * l_p = log softmax(p_logits[r] / T) (the routed slim verifier q'_z),
 *   cost[r] = sum_v p(v) max(0, log(1 - alpha) + l_p(v) - l_q(v))
 *           + sum_v q(v) max(0, log(beta)      + l_p(v) - l_q(v)),
 * the ReLU form of R^KL_{alpha,beta}(q || q'_z) (Eq. 11); summed over a
 * window of positions it is the cost C(z) a routing search minimises
 * (Eq. 12).
 *   q_logits, p_logits  device fp32 [rows][ld], entries [0, vocab) used
 *                       (finite), e.g. the logits dumps of two forwards
 *   cost                device fp32 [rows], written
 * Requires 0 <= alpha < 1, beta > 0, T > 0, ld >= vocab >= 1; rows == 0
 * is a no-op.  Asynchronous on `stream`; EINVAL before any launch. */
via_status via_dimr_cost(const float *q_logits, const float *p_logits, int32_t rows, int32_t vocab, int32_t ld,
                         float temperature, float alpha, float beta, float *cost, void *stream);

/* ---- sizes -------------------------------------------------------------- */
size_t via_pool_bytes(const via_model_desc *desc, int32_t n_layer_slots, int32_t n_blocks, int32_t block_size);
/* The workspace also holds, per sequence id, a ring of VIA_STATE_ROWS fp32
 * rows of d_model (the residual stream after the layers the slim route
 * shares with the full model, saved by the slim forward for each slot it
 * feeds), so it grows with max_seqs. */
#define VIA_STATE_ROWS 128
size_t via_workspace_bytes(const via_model_desc *desc, int32_t max_rows, int32_t max_batch,
                           int32_t max_blocks_per_seq, int32_t max_drafts, int32_t max_seqs);
size_t via_staging_bytes(const via_model_desc *desc, int32_t max_rows, int32_t max_batch, int32_t max_blocks_per_seq,
                         int32_t max_drafts);

/* ---- model -------------------------------------------------------------- */
/* Validates the shapes and copies the pointer tables.  The slim route
 * defaults to all layers. */
via_status via_model_create(const via_model_desc *desc, const via_weights *w, via_model **out);
/* Routing mask z as the sorted list of retained layer ids (Sec. 3.3);
 * 1 <= n <= n_layers.  Must be set before via_kv_create. */
via_status via_model_set_route(via_model *m, const int32_t *layers, int32_t n);
via_status via_model_destroy(via_model *m);

/* ---- KV handle and sequences ------------------------------------------- */
via_status via_kv_create(via_model *m, const via_kv_desc *desc, via_kv **out);
via_status via_kv_destroy(via_kv *kv);
/* Attach sequence `seq_id` with n_ctx already-cached positions in both
 * caches (blocks allocated, lowest ids first, full cache then slim cache;
 * contents are whatever the caller writes at those slots). */
via_status via_kv_seq_reserve(via_kv *kv, int32_t seq_id, int32_t n_ctx);
/* Attach `seq_id` and cache tokens[0..n) in both caches (full forward and
 * slim forward, causal; RoPE positions 0..n-1).  This is the committed
 * prefix x that the verification loop of Alg. 1 starts from (App. B.1
 * "Require"/"Ensure": the decoded sequence x grows from it); the paper does
 * not discuss the cache itself, so both verifiers keeping their own cache of
 * that prefix is this library's reading.  Forwards of more than 512 rows run
 * on the compute-bound tile GEMM; longer prompts are fed in chunks of the
 * handle's max_rows.  When the slim route starts with the full model's own
 * leading layers (route[i] == i for i < P, 0 < P < route length), those
 * layers run once: each chunk's slim forward starts at route index P from
 * the full forward's residual stream, and the K/V of layers 0..P-1 are
 * copied from the full cache (the values the slim forward would compute).
 * ENOMEM (nothing attached) when either pool lacks the blocks. */
via_status via_prefill(via_model *m, via_kv *kv, int32_t seq_id, const int32_t *tokens, int32_t n,
                       void *stream);
/* via_prefill for several sequences at once: sequence seq_ids[i] caches
 * its lens[i] tokens, which follow those of the earlier sequences in the
 * flat host array `tokens`.  The sequences share each forward (up to the
 * handle's max_rows rows and max_batch sequences per forward; longer
 * prompts continue in later forwards), so the projections of a batch of
 * prompts run as one tall GEMM.  All-or-nothing: on any error no sequence
 * is attached (EINVAL for repeated or attached ids, ENOMEM when the pools
 * lack the blocks).  Same results as one via_prefill per sequence when
 * every forward has more than 512 rows either way. */
via_status via_prefill_batch(via_model *m, via_kv *kv, int32_t n_seqs, const int32_t *seq_ids, const int32_t *lens,
                             const int32_t *tokens, void *stream);
/* Route index at which the last full-verifier forward of the current (or
 * last committed) step started: 0 (every layer), P (after the shared
 * layers, see via_verify_full), -1 if none ran since the step's slim
 * forward. */
via_status via_kv_last_full_start(const via_kv *kv, int32_t *route_index);
/* Detach a sequence and free its blocks.  Not during a step. */
via_status via_kv_seq_release(via_kv *kv, int32_t seq_id);
/* Valid lengths and block table of one cache (host outputs; table may be
 * NULL).  *n_blocks receives the table length. */
via_status via_kv_seq_info(const via_kv *kv, int32_t seq_id, int32_t cache, int32_t *valid,
                           int32_t *table, int32_t cap, int32_t *n_blocks);

/* ---- the verification step ---------------------------------------------
 * Order per step: via_verify_slim -> via_tier_decide(full = NULL) ->
 * [synchronise; if any status == 1: via_verify_full (those sequences) ->
 * via_tier_decide(full)] -> synchronise -> via_kv_commit_rollback. */

/* Slim-verifier forward (route of via_model_set_route, slim cache) over the
 * window rows, then the fused head: per-row max/argmax/sum-exp and the
 * logit of every draft token.  This is the step of Alg. 1 (and its full form
 * in App. B.1) that runs q' in parallel on the block's prefixes
 * x_<t, ..., x_<t+gamma-1 to obtain q'_t..q'_{t+gamma-1}; q' = Pi_z(q) is the
 * routed submodel of Sec. 3.3 reading q's own weights.  The per-row maximum
 * is M' of App. B.2 (in logit form), the draft logits give q'(v) for the gate.
 * Allocates cache blocks for the rows (ENOMEM leaves state unchanged) and
 * starts a step.  ESTATE if a step is open. */
via_status via_verify_slim(via_model *m, via_kv *kv, const via_window *win, const via_tier_params *p,
                           via_verify_out *out, void *stream);
/* Full-verifier forward (all layers, full cache) for the sequences with
 * run[b] != 0 (host [batch]; NULL = all), over lag rows + window rows.
 * This is the escalation branch of App. B.1 ("invoke q on prefix x_<t+j"
 * when q' is not confident, region (B.3) of App. B.2): one batched forward
 * serves every escalated position of a sequence's window.  The lag rows
 * (committed tokens the full cache has not seen because q was not invoked
 * on earlier steps) are this library's reading of the silent cache policy.
 * win must be the window of the open step; n_lag[b] must equal the full
 * cache's lag for each run sequence (ESTATE otherwise).
 * When the slim route begins with layers 0..P-1 of the full model, those
 * layers compute the same K/V and residual stream in both forwards; the
 * forward then starts at layer P, taking the K/V of layers < P from the slim
 * cache and the residual stream from the state ring, provided every run
 * sequence has the state of each lag and window slot there (the ring keeps
 * the last VIA_STATE_ROWS slots; a tree commit the full verifier did not see
 * that keeps more than the root clears it).  Otherwise it runs all layers.
 * via_kv_last_full_start reports which. */
via_status via_verify_full(via_model *m, via_kv *kv, const via_window *win, const int32_t *run,
                           const via_tier_params *p, via_verify_out *out, void *stream);
/* Forward of either verifier (cache = VIA_CACHE_*) that leaves the logical
 * KV state untouched: rows are written past the valid length and any block
 * it needs is returned to the pool on exit.  For drafters and probes. */
via_status via_verify_probe(via_model *m, via_kv *kv, int32_t cache, const via_window *win,
                            const via_tier_params *p, via_verify_out *out, void *stream);
/* Confidence, tier, gate walk of the open step (App. B.1).  With full ==
 * NULL, sequences whose walk reaches an escalated position get status 1.
 * With full, sequences that ran the full forward are resolved.  Writes the
 * decision and copies `packed` to `h_packed`. */
via_status via_tier_decide(via_kv *kv, const via_tier_params *p, const via_verify_out *slim,
                           const via_verify_out *full, via_decision *dec, void *stream);
/* Sampling rules (App. A) for chain drafts.  An accept-tier draft is kept;
 * at a slim-tier position the walk stops and emits a sample of the slim
 * verifier q' = softmax(l'/T) (App. B.1, rewrite from q'); an escalated
 * draft x with drafter probability p(x) and verifier probability
 * q(x) = softmax(l/T)(x) is kept iff uniforms[.., 0] < min(1, q(x) /
 * ((1 - alpha) p(x))) (Eq. A.2; p(x) = 0 keeps it), else the walk stops and
 * emits a sample of norm(max(0, q/beta - p)) (Eq. A.3; q itself if that has
 * no mass).  alpha = 0, beta = 1 is the lossless rule.  A sample with
 * uniform u is the first token, in id order, whose running weight exceeds
 * u times the total weight.  When every draft is kept nothing is emitted.
 *   draft_probs  device fp32 [batch * window.max_drafts * vocab]: p of each
 *                draft position (row b * max_drafts + j), caller-owned.
 *   uniforms     host fp32 [batch * window.max_drafts * 3] in [0, 1): per
 *                draft the acceptance, slim-sample and residual-sample
 *                uniforms (b * max_drafts + j) * 3 + {0, 1, 2}; copied
 *                during the call. */
typedef struct {
  float alpha, beta; /* 0 <= alpha < 1, beta >= 1 - alpha (App. A, with Eq. A.3) */
  const float *draft_probs;
  const float *uniforms;
} via_sampling;
/* via_tier_decide under the sampling rules.  Both verify outputs must carry
 * logits (slim->logits, and full->logits when full is given); both decide
 * calls of a step take the same sampling arguments.  EUNSUPPORTED for tree
 * windows, EINVAL for alpha outside [0, 1), beta < 1 - alpha, missing
 * arrays or a uniform outside [0, 1).  Writes the decision as via_tier_decide does, with the
 * sampled token in `emit`. */
via_status via_tier_decide_sampled(via_kv *kv, const via_tier_params *p, const via_verify_out *slim,
                                   const via_verify_out *full, const via_sampling *smp, via_decision *dec,
                                   void *stream);
/* Draw one token per requested row from softmax(l/T) of a forward's logits
 * (the drafter's draw: App. A's p is this distribution).  For i < n the
 * row is out rows row[i] (host, each in [0, out_rows), the row count of the
 * forward that wrote `out`); the token is the first id whose running weight
 * exp((l - max)/T) exceeds uniforms[i] (host, in [0, 1)) times the total,
 * written to tokens[i] (device).  probs (device, nullable) receives each
 * row's probabilities exp((l - max)/T) / row_sumexp at probs[i * probs_ld
 * + v] (probs_ld >= vocab).
 * temperature must be the one the forward's statistics were taken at.
 * Uses the handle's workspace: call it on the handle's stream, between
 * steps or inside one.  EINVAL for n outside [0, max_batch] or bad
 * arguments. */
via_status via_sample_rows(via_kv *kv, const via_verify_out *out, int32_t out_rows, int32_t n, const int32_t *row,
                           float temperature, const float *uniforms, int32_t *tokens, float *probs,
                           int32_t probs_ld, void *stream);
/* via_sample_rows for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same draws and probabilities, without a KV handle.  The requests go to
 * the device as kernel arguments and the kernels' scratch (request array and
 * per-slice sums, 66560 bytes) is a static device array of the library, which
 * each GPU it runs on holds until the process ends; the call allocates and
 * frees nothing.  Every call on a GPU reuses that GPU's scratch and leaves its
 * contents behind: calls that overlap on one GPU (two streams, two threads)
 * race and must be serialised by the caller.  At most
 * VIA_STATIC_SAMPLE_MAX_ROWS draws per call (EINVAL beyond).  out, out_rows,
 * n, row, temperature, uniforms, tokens, probs and probs_ld are as for
 * via_sample_rows; vocab is the logits row length (the model's vocabulary).
 * EDEVICE if the scratch address cannot be obtained. */
#define VIA_STATIC_SAMPLE_MAX_ROWS 64
via_status via_sample_rows_static(const via_verify_out *out, int32_t out_rows, int32_t vocab, int32_t n,
                                  const int32_t *row, float temperature, const float *uniforms, int32_t *tokens,
                                  float *probs, int32_t probs_ld, void *stream);
/* Commit the open step from dec->h_packed (read on the host: synchronise
 * first).  This is the end of a block in Alg. 1 and App. B.1: append the
 * accepted prefix x_t..x_{t+kappa-1} (plus the rewritten token at the
 * earliest rewrite position j*) and discard the remaining suffix (Sec. 3.4,
 * Step 4: the longest accepted prefix kappa is committed and decoding
 * resumes after it).  Appends kappa drafts (+ emit) per sequence: slim valid length
 * becomes n'-1; full valid length becomes n'-1 if the full verifier ran
 * for that sequence this step, else it keeps lagging; blocks wholly past a
 * valid length are freed; tree steps move the accepted nodes' K/V to
 * contiguous slots (kernel on `stream`).  All-or-nothing: ESTATE (nothing
 * changed) if any status is 1 or no step is open. */
via_status via_kv_commit_rollback(via_kv *kv, const via_decision *dec, void *stream);

/* ---- a whole step, driven natively --------------------------------------
 * The loop body of Alg. 1 (App. B.1) in one call: window assembly from the
 * library's record of each sequence's committed tokens and the caller's
 * drafts, via_verify_slim, via_tier_decide, and -- when some sequence's walk
 * escalates -- via_verify_full over those sequences (with the lag rows their
 * full cache is missing) and the second via_tier_decide, then
 * via_kv_commit_rollback, which also appends the committed tokens to the
 * record.  Unlike the calls it composes, via_step synchronises `stream`: once
 * for the first decision, again after an escalation.  On return dec->h_packed
 * holds the committed decision.  Errors are those of the composed calls (a
 * failure after the slim forward leaves the step open, as the individual
 * calls would); ESTATE for a sequence whose committed tokens were never given.
 */
typedef struct {
  int32_t batch, max_drafts;     /* stride of the draft arrays, 1..VIA_MAX_DRAFTS */
  const int32_t *seq_id;         /* [batch] */
  const int32_t *n_drafts;       /* [batch], >= 1 */
  const int32_t *draft_tok;      /* [batch * max_drafts] */
  const int32_t *draft_parent;   /* [batch * max_drafts] tree parents (-1 root, < j), or NULL: chain */
} via_drafts;
/* Give an attached sequence its committed tokens x[0..n-1] (host, copied):
 * n must be its slim valid length + 1 (x[n-1] is the pending token).  From
 * then on every commit appends the sequence's accepted drafts and emitted
 * token.  ESTATE during a step. */
via_status via_kv_seq_set_tokens(via_kv *kv, int32_t seq_id, const int32_t *tokens, int32_t n);
/* Read the committed tokens (host out[0..cap)); *n receives their count.
 * ESTATE if they were never given. */
via_status via_kv_seq_tokens(const via_kv *kv, int32_t seq_id, int32_t *out, int32_t cap, int32_t *n);
via_status via_step(via_model *m, via_kv *kv, const via_drafts *drafts, const via_tier_params *p,
                    via_verify_out *slim, via_verify_out *full, via_decision *dec, void *stream);

/* ---- kernel timing (profiling aid) --------------------------------------
 * When a kind's bit is set, every launch of that kernel kind is bracketed by
 * two HIP events on the call's stream.  via_kv_timer_read waits for the
 * recorded events, returns the launch count and summed milliseconds of one
 * kind since the last read of that kind, and forgets them. */
#define VIA_KERNEL_QKV 0    /* QKV projection + RoPE + paged K/V write */
#define VIA_KERNEL_ATTN 1   /* window attention (+ split-KV combine) */
#define VIA_KERNEL_O 2      /* O projection + residual */
#define VIA_KERNEL_GATEUP 3 /* gate/up projection + SwiGLU */
#define VIA_KERNEL_DOWN 4   /* down projection + residual */
#define VIA_KERNEL_HEAD 5   /* output head + row statistics */
#define VIA_KERNEL_DECIDE 6 /* tier decision (+ the sampling rules' draw) */
#define VIA_KERNEL_COUNT 7
via_status via_kv_timer_enable(via_kv *kv, uint32_t kind_mask);
via_status via_kv_timer_read(via_kv *kv, int32_t kind, int32_t *launches, double *total_ms);

const char *via_last_error(void);
/* Library version string. */
const char *via_version(void);

#ifdef __cplusplus
}
#endif
#endif /* VIA_H */
