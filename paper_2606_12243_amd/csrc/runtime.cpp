// Host runtime of the C ABI (include/via.h): handles, argument validation,
// the paged block allocator, per-call row plans and kernel sequencing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <set>
#include <string>
#include <vector>

#include "../../include/via.h"
#include "host_book.h"
#include "kernels.h"

using namespace via;

namespace {

constexpr size_t kAlign = 256;
constexpr int kRing = 4;

size_t al(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

int esize_of(const via_model_desc* d) { return d->dtype == VIA_DTYPE_BF16 ? 2 : 4; }

// Split-K policy: about two work-groups per CU, at least two 32-wide K steps
// per wave (8 waves) in each slice.  Depends only on the GEMM shape.
// K splits of a GEMM: as many work-groups as fit the 256 compute units in one
// round (a GEMM work-group occupies a whole CU, so a 257th would run alone
// in a second round), with at least 8 steps of 32 per split.
int choose_ksplit(int N, int K) {
  const int tiles = gemm_tiles(N);
  return std::max(1, std::min(256 / std::max(1, tiles), K / 256));
}

struct GemmShape {
  int N, K, ks;
  GemmRole role;
  int nb_ki, ks_ki;  // the K-interleaved kernel's blocks per work-group and splits (forwards of <= 32 rows)
};

struct Dims {
  int L, d, H, KVH, hd, F, V, qkv, G;
  GemmShape g_qkv, g_o, g_gu, g_down;
};

Dims dims_of(const via_model_desc* d) {
  Dims r;
  r.L = d->n_layers;
  r.d = d->d_model;
  r.H = d->n_heads;
  r.KVH = d->n_kv_heads;
  r.hd = d->head_dim;
  r.F = d->d_ffn;
  r.V = d->vocab;
  r.qkv = (r.H + 2 * r.KVH) * r.hd;
  r.G = r.H / std::max(1, r.KVH);
  const bool f32 = d->dtype != VIA_DTYPE_BF16;
  auto shape = [&](int N, int K, GemmRole role) {
    GemmShape g{N, K, choose_ksplit(N, K), role, 1, 1};
    gemm_ki_plan(N, K, &g.nb_ki, &g.ks_ki);
    return g;
  };
  r.g_qkv = shape(r.qkv, r.d, GemmRole::kQkv);
  r.g_o = shape(r.d, r.H * r.hd, GemmRole::kO);
  r.g_gu = GemmShape{2 * r.F, r.d, 1, GemmRole::kGateUp, 1, 1};  // full K per work-group (SwiGLU epilogue)
  r.g_down = shape(r.d, r.F, GemmRole::kDown);
  return r;
}

struct Layout {
  size_t X, Yf, Q, Af, Hf, Ylf, part, att_o, att_ml, lm_part, ss;
  size_t xstate;                       // state ring: [max_seqs][kStateRows][d] residual stream after the shared layers
  size_t rows, seqs, btab, items, lm, xfer;  // plan region
  size_t step_seqs, dtok, drow, dpar, du;  // step region
  size_t sreq, ssum;                   // sampling requests and slice sums of a decision
  size_t c_btab, c_moves;              // commit region
  size_t plan_bytes, step_bytes, commit_bytes;
  size_t total;
  int max_chunks, max_items;
};

Layout layout_of(const via_model_desc* desc, int max_rows, int max_batch, int max_blocks, int max_drafts,
                 int max_seqs) {
  Dims D = dims_of(desc);
  const size_t es = esize_of(desc);
  Layout L{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t r = o;
    o += al(bytes);
    return r;
  };
  const size_t R = max_rows;
  // activation fragments: rows padded to the GEMM row group; bf16 models
  // keep kQkvTerms bf16 terms for the QKV input, 2 elsewhere; fp32 models 1 fp32
  const size_t Rp = (size_t)gemm_padded_rows(max_rows);
  const size_t fq = es == 2 ? 2 * std::max(2, kQkvTerms) : 4, f2 = 4;
  L.X = take(R * D.d * 4);
  L.Yf = take(Rp * D.d * fq);
  L.Q = take(R * D.H * D.hd * 4);
  L.Af = take(Rp * D.H * D.hd * f2);
  L.Hf = take(Rp * D.F * f2);
  L.Ylf = take(Rp * D.d * f2);
  // split-K partials of forwards of up to kPrefillMinRows rows; longer
  // (prefill-sized) forwards write one partial of all their rows.  The
  // gate/up kernels write h directly and need none.
  size_t part = 0;
  for (const GemmShape& g : {D.g_qkv, D.g_o, D.g_down}) {
    part = std::max(part, (size_t)std::max(g.ks, g.ks_ki) * std::min<size_t>(R, kPrefillMinRows) * g.N * 4);
    if (gemm_is_prefill(es == 2, (int)R)) part = std::max(part, R * g.N * 4);
  }
  L.part = take(part);
  L.max_chunks = std::min(kAttnMaxSplits, ceil_div(max_blocks * kBlock, 32));
  L.att_o = take((size_t)L.max_chunks * R * D.H * D.hd * 4);
  L.att_ml = take((size_t)L.max_chunks * R * D.H * 2 * 4);
  L.lm_part = take((size_t)gemm_tiles(D.V) * R * 4 * 4);
  L.ss = take((size_t)ceil_div(D.d, kNormChunk) * R * 4);  // RMSNorm sums of squares [chunk][row]
  L.xstate = take((size_t)max_seqs * kStateRows * D.d * 4);
  L.max_items = ceil_div(max_rows * D.G, kAttnQueries) + max_batch;
  // plan region (one upload per forward)
  size_t p0 = o;
  L.rows = take(R * sizeof(RowInfo));
  L.seqs = take((size_t)max_batch * sizeof(SeqInfo));
  L.btab = take((size_t)max_batch * max_blocks * 4);
  L.items = take((size_t)L.max_items * sizeof(AttnItem));
  L.lm = take(R * sizeof(LmRow));
  L.xfer = take(R * sizeof(PrefixXfer));
  L.plan_bytes = o - p0;
  size_t s0 = o;
  L.step_seqs = take((size_t)max_batch * sizeof(StepSeq));
  L.dtok = take((size_t)max_batch * max_drafts * 4);
  L.drow = take((size_t)max_batch * max_drafts * 4);
  L.dpar = take((size_t)max_batch * max_drafts * 4);
  L.du = take((size_t)max_batch * max_drafts * 3 * 4);
  L.step_bytes = o - s0;
  L.sreq = take((size_t)max_batch * sizeof(SampleReq));
  L.ssum = take((size_t)max_batch * kSampleSlices * 2 * sizeof(double));
  size_t c0 = o;
  L.c_btab = take((size_t)2 * max_batch * max_blocks * 4);
  L.c_moves = take((size_t)2 * max_batch * max_drafts * sizeof(KvMove));
  L.commit_bytes = o - c0;
  L.total = o;
  return L;
}

size_t staging_slot_bytes(const Layout& L) { return std::max({L.plan_bytes, L.step_bytes, L.commit_bytes}); }

}  // namespace

struct via_model {
  via_model_desc d;
  Dims D;
  const void *embed, *lm_head, *final_norm;
  std::vector<const void*> attn_norm, w_qkv, w_o, ffn_norm, w_gate_up, w_down;
  std::vector<int> route;
  bool bf16;
  int n_kv = 0;
};

struct via_kv {
  via_model* m;
  via_kv_desc d;
  Layout L;
  char* ws;
  char* stage;
  size_t slot_bytes;
  KvBook bk;
  bool step_open = false;
  WinCopy win;
  bool xpref_ok = false;      // the open step's slim forward saved its rows' states after the shared layers
  int last_full_start = -1;   // route index the last full forward started at (-1: none in this step)
  // device copy of the open step's decision inputs uploaded with the slim
  // forward's plan (greedy rule, before the full verifier ran), or null
  char* extra_dev = nullptr;
  const char* staged_step = nullptr;
  std::vector<int> step_n;  // committed length n per batch entry at step start
  bool sticky = false;
  int n_cu = 256;  // compute units of the device (attention work-groups of one round)
  // device address of the last decision's pinned host mirror (null: copy it)
  const int32_t* h_packed_host = nullptr;
  int32_t* h_packed_dev = nullptr;
  hipEvent_t ev[kRing];
  bool ev_used[kRing];
  int ring = 0;
  // kernel timing
  uint32_t timer_mask = 0;
  std::vector<hipEvent_t> ev_pool;
  std::vector<std::pair<int, std::pair<hipEvent_t, hipEvent_t>>> timed;
};

namespace {

via_status hip_check(via_kv* kv, hipError_t e, const char* what) {
  if (e == hipSuccess) return VIA_OK;
  if (kv) kv->sticky = true;
  return fail(VIA_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

// Copy host bytes to device through the next pinned staging slot.
via_status upload(via_kv* kv, void* dst, const void* src, size_t bytes, hipStream_t s) {
  if (bytes == 0) return VIA_OK;
  if (bytes > kv->slot_bytes) return fail(VIA_EINVAL, "upload of %zu bytes exceeds staging slot", bytes);
  int r = kv->ring;
  kv->ring = (kv->ring + 1) % kRing;
  if (kv->ev_used[r]) {
    via_status st = hip_check(kv, hipEventSynchronize(kv->ev[r]), "hipEventSynchronize");
    if (st) return st;
  }
  char* slot = kv->stage + (size_t)r * kv->slot_bytes;
  memcpy(slot, src, bytes);
  via_status st = hip_check(kv, hipMemcpyAsync(dst, slot, bytes, hipMemcpyHostToDevice, s), "hipMemcpyAsync");
  if (st) return st;
  st = hip_check(kv, hipEventRecord(kv->ev[r], s), "hipEventRecord");
  kv->ev_used[r] = true;
  return st;
}

hipEvent_t pool_event(via_kv* kv) {
  if (!kv->ev_pool.empty()) {
    hipEvent_t e = kv->ev_pool.back();
    kv->ev_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Run `launch` bracketed by events when its kind is being timed.
template <typename F>
void timed_launch(via_kv* kv, int kind, hipStream_t s, F&& launch) {
  if (!(kv->timer_mask & (1u << kind))) {
    launch();
    return;
  }
  hipEvent_t a = pool_event(kv), b = pool_event(kv);
  if (!a || !b) {
    launch();
    return;
  }
  (void)hipEventRecord(a, s);
  launch();
  (void)hipEventRecord(b, s);
  kv->timed.push_back({kind, {a, b}});
}

// A GEMM of a timed kind carries its events in its own dispatch.
void timed_gemm(via_kv* kv, int kind, bool bf, GemmRole role, const GemmArgs& g, hipStream_t s) {
  hipEvent_t a = nullptr, b = nullptr;
  if (kv->timer_mask & (1u << kind)) {
    a = pool_event(kv);
    b = a ? pool_event(kv) : nullptr;
    if (a && !b) {
      kv->ev_pool.push_back(a);
      a = nullptr;
    }
  }
  launch_gemm(bf, role, g, s, a, b);
  if (a) kv->timed.push_back({kind, {a, b}});
}

template <typename T>
void put(std::vector<char>& blob, size_t off, const std::vector<T>& v) {
  if (!v.empty()) memcpy(blob.data() + off, v.data(), v.size() * sizeof(T));
}

// Forward of one route over the planned rows; optional fused head.
// Leading layers the slim route shares with the full model (route[i] == i):
// the slim forward's state after them is the full model's.
int shared_prefix(const via_model* m) {
  int n = 0;
  while (n < (int)m->route.size() && m->route[n] == n) ++n;
  return n;
}

// start_si > 0: the forward begins at route position start_si (the shared
// layers) from a saved state, with the shared layers' K/V copied from the
// other cache (P.xfer gives each row's source and pages): a step's full
// forward from the slim forward's state ring, a prefill's slim forward from
// its full forward's rows.  save_prefix: store the residual stream after
// the shared layers in the state ring (slim forwards of a step);
// save_rows: store it per row in the head-input region (full forwards of a
// prefill, which run no head).
via_status exec_forward(via_model* m, via_kv* kv, int cache, Plan& P, bool head, const via_verify_out* out,
                        float inv_T, hipStream_t s, int start_si = 0, bool save_prefix = false,
                        bool save_rows = false) {
  const Layout& L = kv->L;
  const Dims& D = m->D;
  const int M = (int)P.rows.size();
  if (M == 0) return VIA_OK;
  if (M > kv->d.max_rows) return fail(VIA_EINVAL, "forward of %d rows exceeds max_rows %d", M, kv->d.max_rows);
  if ((int)P.items.size() > L.max_items) return fail(VIA_EINVAL, "too many attention tiles");
  // key splits of the attention items: about one work-group per compute unit
  AttnArgs at{};
  if (plan_attention(P.items.data(), (int)P.items.size(), D.KVH, L.max_chunks, kAttnTargetGroups, kv->n_cu, &at.span,
                     &at.max_chunks))
    return fail(VIA_EINVAL, "a sequence is too long for %d attention splits", L.max_chunks);
  // one upload of the plan: its parts packed back to back (256-byte aligned)
  // at the start of the plan region, which has room for the largest plan
  const size_t o_rows = 0;
  const size_t o_seqs = al(o_rows + P.rows.size() * sizeof(RowInfo));
  const size_t o_btab = al(o_seqs + P.seqs.size() * sizeof(SeqInfo));
  const size_t o_items = al(o_btab + P.btab.size() * 4);
  const size_t o_lm = al(o_items + P.items.size() * sizeof(AttnItem));
  const size_t o_xfer = al(o_lm + P.lm.size() * sizeof(LmRow));
  const size_t plan_used = al(o_xfer + P.xfer.size() * sizeof(PrefixXfer));
  if (plan_used > L.plan_bytes) return fail(VIA_EINVAL, "plan of %zu bytes exceeds its region", plan_used);
  // extra bytes ride in the same copy when the plan region has room for them
  const bool extra = !P.extra.empty() && plan_used + P.extra.size() <= L.plan_bytes;
  std::vector<char> blob(plan_used + (extra ? P.extra.size() : 0));
  put(blob, o_rows, P.rows);
  put(blob, o_seqs, P.seqs);
  put(blob, o_btab, P.btab);
  put(blob, o_items, P.items);
  put(blob, o_lm, P.lm);
  put(blob, o_xfer, P.xfer);
  if (extra) memcpy(blob.data() + plan_used, P.extra.data(), P.extra.size());
  char* ws = kv->ws;
  char* plan = ws + L.rows;
  via_status st = upload(kv, plan, blob.data(), blob.size(), s);
  if (st) return st;
  kv->extra_dev = extra ? plan + plan_used : nullptr;
  if (!extra) kv->staged_step = nullptr;  // this plan overwrote any staged decision inputs

  const bool bf = m->bf16;
  const RowInfo* d_rows = (const RowInfo*)(plan + o_rows);
  const SeqInfo* d_seqs = (const SeqInfo*)(plan + o_seqs);
  const int32_t* d_btab = (const int32_t*)(plan + o_btab);
  float* X = (float*)(ws + L.X);
  void* Yf = ws + L.Yf;
  void* Q = ws + L.Q;  // bf16 models: hi terms then lo terms; fp32 models: fp32 Q
  uint16_t* Qlo = (uint16_t*)(ws + L.Q) + (size_t)M * D.H * D.hd;
  void* Af = ws + L.Af;
  void* Hf = ws + L.Hf;
  float* part = (float*)(ws + L.part);
  const int MBn = gemm_padded_rows(M) / 16;
  void* pool = cache == VIA_CACHE_FULL ? kv->d.pool_full : kv->d.pool_slim;
  const int pool_blocks = cache == VIA_CACHE_FULL ? kv->d.blocks_full : kv->d.blocks_slim;
  std::vector<int> route;
  if (cache == VIA_CACHE_FULL)
    for (int l = 0; l < D.L; ++l) route.push_back(l);
  else
    route = m->route;
  const float eps = m->d.rms_eps;

  // K splits of each projection's partials (one on the prefill GEMM)
  const bool prefill_gemm = gemm_is_prefill(bf, M);
  auto ki = [&](const GemmShape& sh) { return bf && gemm_uses_ki(sh.role, M, sh.N); };
  auto ks = [&](const GemmShape& sh) { return prefill_gemm ? 1 : ki(sh) ? sh.ks_ki : sh.ks; };
  auto gemm = [&](const void* Xf, const void* W, const GemmShape& sh, GemmRole role, int kind) {
    GemmArgs g{};
    g.X = Xf;
    g.MBn = MBn;
    g.W = W;
    g.M = M;
    g.K = sh.K;
    g.N = sh.N;
    g.ksplit = ks(sh);
    g.nb = ki(sh) ? sh.nb_ki : 0;
    g.part = part;
    timed_gemm(kv, kind, bf, role, g, s);
  };

  float* ss = (float*)(ws + L.ss);
  const int ss_stride = kv->d.max_rows;
  const int n_shared = shared_prefix(m);
  if (save_rows && (head || cache != VIA_CACHE_FULL || save_prefix))
    return fail(VIA_EINVAL, "internal: per-row states are kept by prefill full forwards only");
  if (start_si > 0) {
    if (start_si != n_shared || (int)P.xfer.size() != M || (cache == VIA_CACHE_SLIM && head))
      return fail(VIA_EINVAL, "internal: forward from the shared layers without its row map");
    const bool from_full = cache == VIA_CACHE_SLIM;  // a prefill's slim forward
    PrefixArgs pa{};
    pa.xfer = (const PrefixXfer*)(plan + o_xfer);
    pa.M = M;
    pa.P = start_si;
    pa.d = D.d;
    pa.KVH = D.KVH;
    pa.hd = D.hd;
    pa.xstate = (const float*)(ws + (from_full ? L.Ylf : L.xstate));
    pa.X = X;
    pa.src_pool = from_full ? kv->d.pool_full : kv->d.pool_slim;
    pa.src_blocks = from_full ? kv->d.blocks_full : kv->d.blocks_slim;
    pa.dst_pool = from_full ? kv->d.pool_slim : kv->d.pool_full;
    pa.dst_blocks = from_full ? kv->d.blocks_slim : kv->d.blocks_full;
    launch_prefix_copy(bf, pa, s);
  }
  // first layer's input norm; from layer 0 it also gathers the embedding rows into X
  launch_resid_add(bf, kQkvTerms, X, nullptr, 1, M, D.d, m->attn_norm[route[start_si]], Yf, MBn, nullptr, ss, ss_stride, s,
                   nullptr, start_si > 0 ? nullptr : m->embed, d_rows);
  at.q_hi = Q;
  at.q_lo = Qlo;
  at.pool = pool;
  at.pool_blocks = pool_blocks;
  at.rows = d_rows;
  at.seqs = d_seqs;
  at.btab = d_btab;
  at.items = (const AttnItem*)(plan + o_items);
  at.n_items = (int)P.items.size();
  at.M = M;
  at.H = D.H;
  at.KVH = D.KVH;
  at.hd = D.hd;
  at.scale = (float)(1.0 / std::sqrt((double)D.hd));
  at.part_o = (float*)(ws + L.att_o);
  at.part_ml = (float*)(ws + L.att_ml);
  at.out = Af;
  at.MBn = MBn;
  QkvArgs qa{};
  qa.P = part;
  qa.ksplit = ks(D.g_qkv);
  qa.M = M;
  qa.H = D.H;
  qa.KVH = D.KVH;
  qa.hd = D.hd;
  qa.theta = m->d.rope_theta;
  qa.rows = d_rows;
  qa.seqs = d_seqs;
  qa.btab = d_btab;
  qa.q_hi = (uint16_t*)Q;
  qa.q_lo = Qlo;
  qa.pool = pool;
  qa.pool_blocks = pool_blocks;
  qa.ss = ss;
  qa.ss_stride = ss_stride;
  qa.d = D.d;
  qa.eps = eps;
  for (size_t si = start_si; si < route.size(); ++si) {
    const int l = route[si];
    // Q/K/V from kQkvTerms bf16 terms per activation (the K/V are rounded to the cache's bf16)
    gemm(Yf, m->w_qkv[l], D.g_qkv, GemmRole::kQkv, VIA_KERNEL_QKV);
    qa.layer_slot = (int)si;
    launch_qkv_finish(bf, qa, s);
    at.layer_slot = (int)si;
    timed_launch(kv, VIA_KERNEL_ATTN, s, [&] { launch_attention(bf, at, s); });
    gemm(Af, m->w_o[l], D.g_o, GemmRole::kO, VIA_KERNEL_O);
    launch_resid_add(bf, 2, X, part, ks(D.g_o), M, D.d, m->ffn_norm[l], Yf, MBn, nullptr, ss, ss_stride, s);
    {
      GemmArgs g{};
      g.X = Yf;
      g.MBn = MBn;
      g.W = m->w_gate_up[l];
      g.M = M;
      g.K = D.d;
      g.N = 2 * D.F;
      g.ksplit = 1;
      g.part = part;
      g.H = Hf;
      g.F = D.F;
      g.nb = gate_up_blocks_per_group(D.F);
      g.ss = ss;
      g.ss_stride = ss_stride;
      g.eps = eps;
      timed_gemm(kv, VIA_KERNEL_GATEUP, bf, GemmRole::kGateUp, g, s);
    }
    gemm(Hf, m->w_down[l], D.g_down, GemmRole::kDown, VIA_KERNEL_DOWN);
    if (si + 1 < route.size()) {
      // after the shared layers: the state ring (slot per row via d_rows) or
      // the prefill's per-row copy in the head-input region
      const bool at_shared = (int)si + 1 == n_shared;
      float* xcopy = at_shared && save_prefix ? (float*)(ws + L.xstate)
                     : at_shared && save_rows ? (float*)(ws + L.Ylf)
                                              : nullptr;
      launch_resid_add(bf, kQkvTerms, X, part, ks(D.g_down), M, D.d, m->attn_norm[route[si + 1]], Yf, MBn, nullptr, ss,
                       ss_stride, s, xcopy, nullptr, save_rows ? nullptr : d_rows);
    }
  }
  if (head && !P.lm.empty()) {
    const int nlm = (int)P.lm.size();
    const LmRow* d_lm = (const LmRow*)(plan + o_lm);
    void* Ylf = ws + L.Ylf;
    const int MBl = gemm_padded_rows(nlm) / 16;
    // last residual update, final norm of the head rows only
    launch_resid_add(bf, 2, X, part, ks(D.g_down), M, D.d, m->final_norm, Ylf, MBl, d_rows, ss, ss_stride, s);
    GemmArgs h{};
    h.X = Ylf;
    h.MBn = MBl;
    h.W = m->lm_head;
    h.M = nlm;
    h.K = D.d;
    h.N = D.V;
    h.ksplit = 1;
    h.lm = d_lm;
    h.lm_part = (float*)(ws + L.lm_part);
    h.inv_T = inv_T;
    h.logits = out->logits;
    h.draft_logit = out->draft_logit;
    h.ss = ss;
    h.ss_stride = ss_stride;
    h.eps = eps;
    timed_launch(kv, VIA_KERNEL_HEAD, s, [&] {
      launch_gemm(bf, GemmRole::kHead, h, s);
      launch_lm_finalize(d_lm, h.lm_part, nlm, gemm_tiles(D.V), inv_T, out->row_argmax, out->row_max,
                         out->row_sumexp, out->row_gap, s);
    });
  }
  return hip_check(kv, hipGetLastError(), "kernel launch");
}

// The decision's per-step inputs in the step region's layout: a StepSeq per
// batch entry (committed length n, drafts, whether the full verifier ran),
// the draft tokens, rows and parents, and the sampling uniforms when given.
// Between steps every full_ran flag is false (the commit clears them), so
// the copy staged with a step's slim forward carries 0, which is what the
// decision after that forward needs.
std::vector<char> step_blob(const via_kv* kv, const WinCopy& w, const std::vector<int>& step_n,
                            const float* uniforms) {
  const Layout& L = kv->L;
  const int B = w.batch, Dd = std::max(1, w.max_drafts);
  std::vector<char> blob(uniforms ? L.step_bytes : L.du - L.step_seqs);
  std::vector<StepSeq> ss(B);
  for (int b = 0; b < B; ++b) {
    ss[b].n = step_n[b];
    ss[b].n_drafts = w.n_drafts[b];
    ss[b].full_ran = kv->bk.seqs[w.seq[b]].full_ran ? 1 : 0;
  }
  memcpy(blob.data(), ss.data(), B * sizeof(StepSeq));
  memcpy(blob.data() + (L.dtok - L.step_seqs), w.draft_tok.data(), (size_t)B * Dd * 4);
  memcpy(blob.data() + (L.drow - L.step_seqs), w.draft_row.data(), (size_t)B * Dd * 4);
  memcpy(blob.data() + (L.dpar - L.step_seqs), w.draft_parent.data(), (size_t)B * Dd * 4);
  if (uniforms) memcpy(blob.data() + (L.du - L.step_seqs), uniforms, (size_t)B * Dd * 3 * 4);
  return blob;
}

via_status check_params(const via_tier_params* p) {
  if (!p) return fail(VIA_EINVAL, "null tier params");
  if (!(p->temperature > 0.f) || !std::isfinite(p->temperature)) return fail(VIA_EINVAL, "temperature must be > 0");
  if (!(p->tau_full >= 0.f) || !(p->tau_acc >= p->tau_full))
    return fail(VIA_EINVAL, "thresholds must satisfy 0 <= tau_full <= tau_acc");
  if (p->forced < -1 || p->forced > 2) return fail(VIA_EINVAL, "forced must be -1..2");
  return VIA_OK;
}

via_status check_out(const via_verify_out* o) {
  if (!o || !o->row_argmax || !o->row_max || !o->row_sumexp || !o->draft_logit)
    return fail(VIA_EINVAL, "verify_out: row_argmax, row_max, row_sumexp and draft_logit are required");
  return VIA_OK;
}

via_status common_checks(via_model* m, via_kv* kv) {
  if (!m || !kv) return fail(VIA_EINVAL, "null handle");
  if (kv->m != m) return fail(VIA_EINVAL, "KV handle belongs to another model");
  if (kv->sticky) return fail(VIA_EDEVICE, "handle has a sticky device error");
  return VIA_OK;
}

via_status verify_impl(via_model* m, via_kv* kv, int cache, const via_window* win, const int32_t* run_mask,
                       const via_tier_params* p, via_verify_out* out, hipStream_t s, bool probe) {
  via_status st = common_checks(m, kv);
  if (st) return st;
  if ((st = check_params(p)) || (st = check_out(out))) return st;
  WinCopy w;
  const WinCopy* wp = &w;
  if (probe || cache == VIA_CACHE_SLIM) {
    if ((st = copy_window(kv->bk, win, m->d.vocab, kv->d.max_batch, kv->d.max_drafts, w))) return st;
  } else {
    if (!kv->step_open) return fail(VIA_ESTATE, "via_verify_full needs an open step (call via_verify_slim first)");
    if (!win || win->batch != kv->win.batch) return fail(VIA_EINVAL, "window batch differs from the open step");
    for (int b = 0; b < win->batch; ++b)
      if (win->seq_id[b] != kv->win.seq[b] || win->n_rows[b] != kv->win.n_rows[b])
        return fail(VIA_EINVAL, "window differs from the open step");
    wp = &kv->win;
  }
  if (!probe && cache == VIA_CACHE_SLIM && kv->step_open) return fail(VIA_ESTATE, "a step is already open");
  std::vector<int> run;
  for (int b = 0; b < wp->batch; ++b)
    if (!run_mask || run_mask[b]) run.push_back(b);
  Plan P;
  std::vector<std::pair<int, int>> taken;
  if ((st = build_verify_plan(kv->bk, cache, *wp, run, win, true, m->d.vocab, m->D.G, P, &taken))) return st;
  // The full forward of a step starts after the layers the slim route shares
  // with it when every running sequence has the states after those layers
  // of its lag slots (kept by earlier slim forwards) and window slots (this
  // step's slim forward) in the state ring; the K/V of the shared layers are
  // copied from the slim cache.  Otherwise it runs every layer.
  const int n_shared = shared_prefix(m);
  const bool save = !probe && cache == VIA_CACHE_SLIM && n_shared > 0 && n_shared < (int)m->route.size();
  int start_si = 0;
  if (!probe && cache == VIA_CACHE_FULL && kv->xpref_ok && n_shared > 0 && build_prefix_xfer(kv->bk, *wp, run, P))
    start_si = n_shared;
  // the first decision of the step reads its inputs from the slim forward's
  // plan upload (one host-to-device copy fewer between the forward and it)
  if (!probe && cache == VIA_CACHE_SLIM) {
    std::vector<int> n0(w.batch);
    for (int b = 0; b < w.batch; ++b) n0[b] = kv->bk.seqs[w.seq[b]].valid[VIA_CACHE_SLIM] + 1;
    P.extra = step_blob(kv, w, n0, nullptr);
  }
  st = exec_forward(m, kv, cache, P, true, out, 1.0f / p->temperature, s, start_si, save);
  if (probe) {
    book_release_taken(kv->bk, cache, taken);
    return st;
  }
  if (st) {
    book_release_taken(kv->bk, cache, taken);
    return st;
  }
  if (cache == VIA_CACHE_SLIM) {
    kv->staged_step = kv->extra_dev;
    kv->xpref_ok = save;
    kv->last_full_start = -1;
    note_slim_forward(kv->bk, w, run, save);
    kv->win = w;
    kv->step_open = true;
    kv->step_n.assign(w.batch, 0);
    for (int b = 0; b < w.batch; ++b) {
      kv->step_n[b] = kv->bk.seqs[w.seq[b]].valid[VIA_CACHE_SLIM] + 1;
      kv->bk.seqs[w.seq[b]].full_ran = false;
    }
  } else {
    kv->last_full_start = start_si;
    for (int b : run) kv->bk.seqs[wp->seq[b]].full_ran = true;
  }
  return VIA_OK;
}

}  // namespace

extern "C" {

const char* via_last_error(void) { return last_error(); }
const char* via_version(void) { return "via-gfx950 0.1"; }

size_t via_pool_bytes(const via_model_desc* desc, int32_t n_layer_slots, int32_t n_blocks, int32_t block_size) {
  if (!desc) return 0;
  return (size_t)n_layer_slots * n_blocks * 2 * desc->n_kv_heads * block_size * desc->head_dim * esize_of(desc);
}

size_t via_packed_bytes(int32_t rows, int32_t cols, int32_t dtype) {
  if (rows < 1 || cols < 32 || cols % 32 || (dtype != VIA_DTYPE_F32 && dtype != VIA_DTYPE_BF16)) return 0;
  return (size_t)((rows + 63) / 64) * 64 * cols * (dtype == VIA_DTYPE_BF16 ? 2 : 4);
}

via_status via_pack_weight(const void* src, void* dst, int32_t rows, int32_t cols, int32_t dtype, void* stream) {
  if (!src || !dst) return fail(VIA_EINVAL, "null pointer");
  if (!via_packed_bytes(rows, cols, dtype)) return fail(VIA_EINVAL, "rows >= 1, cols a positive multiple of 32, dtype f32/bf16");
  launch_pack(dtype == VIA_DTYPE_BF16, src, dst, rows, cols, 0, (hipStream_t)stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(VIA_EDEVICE, "pack launch: %s", hipGetErrorString(e));
  return VIA_OK;
}

via_status via_gemm_bf16(const void* X, const void* W, float* C, int32_t M, int32_t N, int32_t K, void* stream) {
  if (!X || !W || !C) return fail(VIA_EINVAL, "null pointer");
  if (M < 1 || N < 1 || K < 32 || K % 32) return fail(VIA_EINVAL, "M, N >= 1 and K a positive multiple of 32");
  GemmArgs g{};
  g.X = X;
  g.MBn = ceil_div(M, 16);
  g.W = W;
  g.M = M;
  g.K = K;
  g.N = N;
  g.ksplit = 1;
  g.part = C;
  launch_gemm_bf16(g, (hipStream_t)stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(VIA_EDEVICE, "gemm launch: %s", hipGetErrorString(e));
  return VIA_OK;
}

via_status via_dimr_cost(const float* q_logits, const float* p_logits, int32_t rows, int32_t vocab, int32_t ld,
                         float temperature, float alpha, float beta, float* cost, void* stream) {
  if (rows < 0 || vocab < 1 || ld < vocab) return fail(VIA_EINVAL, "rows >= 0, vocab >= 1 and ld >= vocab");
  if (!(temperature > 0.f) || !std::isfinite(temperature)) return fail(VIA_EINVAL, "temperature must be > 0");
  if (!(alpha >= 0.f && alpha < 1.f) || !(beta > 0.f) || !std::isfinite(beta))
    return fail(VIA_EINVAL, "need 0 <= alpha < 1 and beta > 0");
  if (rows == 0) return VIA_OK;
  if (!q_logits || !p_logits || !cost) return fail(VIA_EINVAL, "null pointer");
  DimrArgs a{};
  a.q = q_logits;
  a.p = p_logits;
  a.rows = rows;
  a.vocab = vocab;
  a.ld = ld;
  a.inv_T = 1.0f / temperature;
  a.log_1m_alpha = (float)std::log(1.0 - (double)alpha);
  a.log_beta = (float)std::log((double)beta);
  a.cost = cost;
  launch_dimr_cost(a, (hipStream_t)stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(VIA_EDEVICE, "dimr cost launch: %s", hipGetErrorString(e));
  return VIA_OK;
}

via_status via_pack_gate_up(const void* src, void* dst, int32_t d_ffn, int32_t d_model, int32_t dtype, void* stream) {
  if (!src || !dst) return fail(VIA_EINVAL, "null pointer");
  if (d_ffn < 8 || d_ffn % 8) return fail(VIA_EINVAL, "d_ffn must be a positive multiple of 8");
  if (!via_packed_bytes(2 * d_ffn, d_model, dtype))
    return fail(VIA_EINVAL, "d_model a positive multiple of 32, dtype f32/bf16");
  launch_pack(dtype == VIA_DTYPE_BF16, src, dst, 2 * d_ffn, d_model, d_ffn, (hipStream_t)stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(VIA_EDEVICE, "pack launch: %s", hipGetErrorString(e));
  return VIA_OK;
}

size_t via_workspace_bytes(const via_model_desc* desc, int32_t max_rows, int32_t max_batch, int32_t max_blocks_per_seq,
                           int32_t max_drafts, int32_t max_seqs) {
  if (!desc || max_rows < 1 || max_batch < 1 || max_blocks_per_seq < 1 || max_drafts < 1 || max_seqs < 1) return 0;
  return layout_of(desc, max_rows, max_batch, max_blocks_per_seq, max_drafts, max_seqs).total;
}

size_t via_staging_bytes(const via_model_desc* desc, int32_t max_rows, int32_t max_batch, int32_t max_blocks_per_seq,
                         int32_t max_drafts) {
  if (!desc || max_rows < 1 || max_batch < 1 || max_blocks_per_seq < 1 || max_drafts < 1) return 0;
  Layout L = layout_of(desc, max_rows, max_batch, max_blocks_per_seq, max_drafts, 1);
  return staging_slot_bytes(L) * kRing;
}

via_status via_model_create(const via_model_desc* desc, const via_weights* w, via_model** out) {
  if (!desc || !w || !out) return fail(VIA_EINVAL, "null argument");
  *out = nullptr;
  const via_model_desc& d = *desc;
  if (d.n_layers < 1 || d.d_model < 1 || d.n_heads < 1 || d.n_kv_heads < 1 || d.head_dim < 1 || d.d_ffn < 1 ||
      d.vocab < 1)
    return fail(VIA_EINVAL, "model dimensions must be positive");
  if (d.dtype != VIA_DTYPE_F32 && d.dtype != VIA_DTYPE_BF16) return fail(VIA_EINVAL, "dtype must be f32 or bf16");
  if (d.head_dim != 64 && d.head_dim != 128) return fail(VIA_EUNSUPPORTED, "head_dim must be 64 or 128");
  if (d.n_heads % d.n_kv_heads) return fail(VIA_EUNSUPPORTED, "n_heads must be a multiple of n_kv_heads");
  if (d.d_model % 64 || d.d_ffn % 64 || (d.n_heads * d.head_dim) % 64)
    return fail(VIA_EUNSUPPORTED, "d_model, d_ffn and n_heads*head_dim must be multiples of 64");
  if (!(d.rms_eps > 0.f) || !(d.rope_theta > 0.f)) return fail(VIA_EINVAL, "rms_eps and rope_theta must be > 0");
  if (!w->embed || !w->lm_head || !w->final_norm || !w->attn_norm || !w->w_qkv || !w->w_o || !w->ffn_norm ||
      !w->w_gate_up || !w->w_down)
    return fail(VIA_EINVAL, "weight pointer missing");
  via_model* m = new via_model();
  m->d = d;
  m->D = dims_of(&d);
  m->bf16 = d.dtype == VIA_DTYPE_BF16;
  m->embed = w->embed;
  m->lm_head = w->lm_head;
  m->final_norm = w->final_norm;
  for (int l = 0; l < d.n_layers; ++l) {
    const void* ptrs[6] = {w->attn_norm[l], w->w_qkv[l], w->w_o[l], w->ffn_norm[l], w->w_gate_up[l], w->w_down[l]};
    for (const void* p : ptrs)
      if (!p) {
        delete m;
        return fail(VIA_EINVAL, "layer %d weight pointer missing", l);
      }
    m->attn_norm.push_back(w->attn_norm[l]);
    m->w_qkv.push_back(w->w_qkv[l]);
    m->w_o.push_back(w->w_o[l]);
    m->ffn_norm.push_back(w->ffn_norm[l]);
    m->w_gate_up.push_back(w->w_gate_up[l]);
    m->w_down.push_back(w->w_down[l]);
    m->route.push_back(l);
  }
  *out = m;
  return VIA_OK;
}

via_status via_model_set_route(via_model* m, const int32_t* layers, int32_t n) {
  if (!m || !layers) return fail(VIA_EINVAL, "null argument");
  if (m->n_kv > 0) return fail(VIA_ESTATE, "route is fixed while KV handles exist");
  if (n < 1 || n > m->d.n_layers) return fail(VIA_EINVAL, "route length %d not in [1, %d]", n, m->d.n_layers);
  for (int i = 0; i < n; ++i) {
    if (layers[i] < 0 || layers[i] >= m->d.n_layers) return fail(VIA_EINVAL, "route layer %d out of range", layers[i]);
    if (i && layers[i] <= layers[i - 1]) return fail(VIA_EINVAL, "route must be strictly increasing");
  }
  m->route.assign(layers, layers + n);
  return VIA_OK;
}

via_status via_model_destroy(via_model* m) {
  if (!m) return fail(VIA_EINVAL, "null model");
  if (m->n_kv > 0) return fail(VIA_ESTATE, "destroy the KV handles first");
  delete m;
  return VIA_OK;
}

via_status via_kv_create(via_model* m, const via_kv_desc* d, via_kv** out) {
  if (!m || !d || !out) return fail(VIA_EINVAL, "null argument");
  *out = nullptr;
  if (d->block_size != kBlock) return fail(VIA_EUNSUPPORTED, "block_size must be %d", kBlock);
  if (d->max_seqs < 1 || d->max_blocks_per_seq < 1 || d->blocks_full < 1 || d->blocks_slim < 1 || d->max_rows < 1 ||
      d->max_batch < 1 || d->max_drafts < 1 || d->max_drafts > VIA_MAX_DRAFTS)
    return fail(VIA_EINVAL, "KV description sizes out of range");
  if (!d->pool_full || !d->pool_slim || !d->workspace || !d->pinned_staging)
    return fail(VIA_EINVAL, "pools, workspace and staging are required");
  if ((uintptr_t)d->workspace % kAlign || (uintptr_t)d->pool_full % 16 || (uintptr_t)d->pool_slim % 16)
    return fail(VIA_EINVAL, "workspace must be %zu-byte and the pools 16-byte aligned", kAlign);
  Layout L = layout_of(&m->d, d->max_rows, d->max_batch, d->max_blocks_per_seq, std::max(1, (int)d->max_drafts),
                       d->max_seqs);
  if (d->workspace_bytes < L.total)
    return fail(VIA_ENOMEM, "workspace %zu bytes < required %zu", d->workspace_bytes, L.total);
  size_t slot = staging_slot_bytes(L);
  if (d->staging_bytes < slot * kRing)
    return fail(VIA_ENOMEM, "staging %zu bytes < required %zu", d->staging_bytes, slot * kRing);
  via_kv* kv = new via_kv();
  kv->m = m;
  kv->d = *d;
  kv->L = L;
  kv->ws = (char*)d->workspace;
  kv->stage = (char*)d->pinned_staging;
  kv->slot_bytes = slot;
  book_init(kv->bk, d->max_seqs, d->max_blocks_per_seq, d->blocks_full, d->blocks_slim);
  {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
      kv->n_cu = n;
    (void)hipGetLastError();
  }
  for (int r = 0; r < kRing; ++r) {
    kv->ev_used[r] = false;
    if (hipEventCreateWithFlags(&kv->ev[r], hipEventDisableTiming) != hipSuccess) {
      for (int q = 0; q < r; ++q) (void)hipEventDestroy(kv->ev[q]);
      delete kv;
      return fail(VIA_EDEVICE, "hipEventCreate failed");
    }
  }
  m->n_kv++;
  *out = kv;
  return VIA_OK;
}

via_status via_kv_timer_enable(via_kv* kv, uint32_t kind_mask) {
  if (!kv) return fail(VIA_EINVAL, "null KV handle");
  if (kind_mask >> VIA_KERNEL_COUNT) return fail(VIA_EINVAL, "unknown kernel kind in mask");
  kv->timer_mask = kind_mask;
  return VIA_OK;
}

via_status via_kv_timer_read(via_kv* kv, int32_t kind, int32_t* launches, double* total_ms) {
  if (!kv || !launches || !total_ms) return fail(VIA_EINVAL, "null argument");
  if (kind < 0 || kind >= VIA_KERNEL_COUNT) return fail(VIA_EINVAL, "unknown kernel kind");
  int n = 0;
  double ms = 0;
  std::vector<std::pair<int, std::pair<hipEvent_t, hipEvent_t>>> keep;
  for (auto& t : kv->timed) {
    if (t.first != kind) {
      keep.push_back(t);
      continue;
    }
    via_status st = hip_check(kv, hipEventSynchronize(t.second.second), "hipEventSynchronize");
    if (st) return st;
    float e = 0.f;
    if ((st = hip_check(kv, hipEventElapsedTime(&e, t.second.first, t.second.second), "hipEventElapsedTime")))
      return st;
    ms += e;
    ++n;
    kv->ev_pool.push_back(t.second.first);
    kv->ev_pool.push_back(t.second.second);
  }
  kv->timed.swap(keep);
  *launches = n;
  *total_ms = ms;
  return VIA_OK;
}

via_status via_kv_destroy(via_kv* kv) {
  if (!kv) return fail(VIA_EINVAL, "null KV handle");
  for (auto& t : kv->timed) {
    (void)hipEventSynchronize(t.second.second);
    kv->ev_pool.push_back(t.second.first);
    kv->ev_pool.push_back(t.second.second);
  }
  for (hipEvent_t e : kv->ev_pool) (void)hipEventDestroy(e);
  for (int r = 0; r < kRing; ++r) {
    if (kv->ev_used[r]) (void)hipEventSynchronize(kv->ev[r]);
    (void)hipEventDestroy(kv->ev[r]);
  }
  kv->m->n_kv--;
  delete kv;
  return VIA_OK;
}

static via_status attach_checks(via_kv* kv, int32_t seq_id, int32_t n) {
  if (!kv) return fail(VIA_EINVAL, "null KV handle");
  if (kv->sticky) return fail(VIA_EDEVICE, "handle has a sticky device error");
  if (kv->step_open) return fail(VIA_ESTATE, "a step is open");
  if (seq_id < 0 || seq_id >= kv->d.max_seqs) return fail(VIA_EINVAL, "seq_id %d out of range", seq_id);
  if (kv->bk.seqs[seq_id].on) return fail(VIA_ESTATE, "sequence %d already attached", seq_id);
  if (n < 0) return fail(VIA_EINVAL, "negative length");
  return VIA_OK;
}

via_status via_kv_seq_reserve(via_kv* kv, int32_t seq_id, int32_t n_ctx) {
  via_status st = attach_checks(kv, seq_id, n_ctx);
  if (st) return st;
  if (blocks_for(n_ctx) > (int)kv->bk.free_[0].size() || blocks_for(n_ctx) > (int)kv->bk.free_[1].size() ||
      blocks_for(n_ctx) > kv->d.max_blocks_per_seq)
    return fail(VIA_ENOMEM, "not enough KV blocks for %d slots", n_ctx);
  kv->bk.seqs[seq_id] = SeqSt();
  kv->bk.seqs[seq_id].on = true;
  book_alloc(kv->bk, 0, {{seq_id, n_ctx}}, nullptr);
  book_alloc(kv->bk, 1, {{seq_id, n_ctx}}, nullptr);
  kv->bk.seqs[seq_id].valid[0] = kv->bk.seqs[seq_id].valid[1] = n_ctx;
  return VIA_OK;
}

via_status via_prefill_batch(via_model* m, via_kv* kv, int32_t n_seqs, const int32_t* seq_ids, const int32_t* lens,
                             const int32_t* tokens, void* stream) {
  via_status st = common_checks(m, kv);
  if (st) return st;
  if (n_seqs < 1 || !seq_ids || !lens) return fail(VIA_EINVAL, "need n_seqs >= 1, seq_ids and lens");
  std::set<int> ids;
  std::vector<size_t> off(n_seqs + 1, 0);
  size_t need[2] = {0, 0};
  for (int i = 0; i < n_seqs; ++i) {
    if ((st = attach_checks(kv, seq_ids[i], lens[i]))) return st;
    if (!ids.insert(seq_ids[i]).second) return fail(VIA_EINVAL, "sequence %d appears twice", seq_ids[i]);
    if (blocks_for(lens[i]) > kv->d.max_blocks_per_seq)
      return fail(VIA_ENOMEM, "sequence %d needs %d blocks > max_blocks_per_seq", seq_ids[i], blocks_for(lens[i]));
    off[i + 1] = off[i] + lens[i];
    need[0] += blocks_for(lens[i]);
  }
  need[1] = need[0];
  if (off[n_seqs] > 0 && !tokens) return fail(VIA_EINVAL, "null tokens");
  for (size_t i = 0; i < off[n_seqs]; ++i)
    if (tokens[i] < 0 || tokens[i] >= m->d.vocab) return fail(VIA_EINVAL, "token %d out of range", tokens[i]);
  if (need[0] > kv->bk.free_[0].size() || need[1] > kv->bk.free_[1].size())
    return fail(VIA_ENOMEM, "not enough KV blocks for the prompts");
  auto detach_all = [&] {
    for (int i = 0; i < n_seqs; ++i) {
      book_trim(kv->bk, 0, seq_ids[i], 0);
      book_trim(kv->bk, 1, seq_ids[i], 0);
      kv->bk.seqs[seq_ids[i]] = SeqSt();
    }
  };
  for (int i = 0; i < n_seqs; ++i) {
    kv->bk.seqs[seq_ids[i]] = SeqSt();
    kv->bk.seqs[seq_ids[i]].on = true;
  }
  for (int cache = 0; cache < 2; ++cache) {
    std::vector<std::pair<int, int>> want;
    for (int i = 0; i < n_seqs; ++i) want.push_back({seq_ids[i], lens[i]});
    if ((st = book_alloc(kv->bk, cache, want, nullptr))) {
      detach_all();
      return st;
    }
  }
  hipStream_t s = (hipStream_t)stream;
  const int G = m->D.G;
  // With layers shared by both routes (route layer i == i for i < n_shared),
  // each chunk runs the full forward, which keeps every row's residual
  // stream after the shared layers, then the slim forward from there with
  // the shared layers' K/V copied from the full cache: the same values the
  // slim forward would compute for those layers, without running them twice.
  const int n_shared = shared_prefix(m);
  if (n_shared > 0 && n_shared < (int)m->route.size()) {
    std::vector<int> done(n_seqs, 0);
    for (;;) {
      Plan Pf, Ps;
      std::vector<int> seq_of;
      int used = 0;
      for (int i = 0; i < n_seqs && used < kv->d.max_rows && (int)seq_of.size() < kv->d.max_batch; ++i) {
        if (done[i] >= lens[i]) continue;
        const int c0 = done[i], c1 = std::min(lens[i], c0 + (kv->d.max_rows - used));
        build_prefill_plan(kv->bk.seqs[seq_ids[i]], VIA_CACHE_FULL, tokens + off[i], c0, c1, G, Pf);
        build_prefill_plan(kv->bk.seqs[seq_ids[i]], VIA_CACHE_SLIM, tokens + off[i], c0, c1, G, Ps);
        seq_of.push_back(seq_ids[i]);
        used += c1 - c0;
        done[i] = c1;
      }
      if (used == 0) break;
      build_prefill_xfer(kv->bk, seq_of, Ps);
      if ((st = exec_forward(m, kv, VIA_CACHE_FULL, Pf, false, nullptr, 1.f, s, 0, false, true)) ||
          (st = exec_forward(m, kv, VIA_CACHE_SLIM, Ps, false, nullptr, 1.f, s, n_shared))) {
        detach_all();
        return st;
      }
    }
    for (int i = 0; i < n_seqs; ++i)
      for (int cache = 0; cache < 2; ++cache) kv->bk.seqs[seq_ids[i]].valid[cache] = lens[i];
    return VIA_OK;
  }
  // otherwise one pass per cache: forwards of up to max_rows rows and
  // max_batch sequences; a sequence's later chunk goes into a later forward
  // (it attends to the earlier chunk)
  for (int cache = 0; cache < 2; ++cache) {
    std::vector<int> done(n_seqs, 0);
    for (;;) {
      Plan P;
      int used = 0, nseq = 0;
      for (int i = 0; i < n_seqs && used < kv->d.max_rows && nseq < kv->d.max_batch; ++i) {
        if (done[i] >= lens[i]) continue;
        const int c0 = done[i], c1 = std::min(lens[i], c0 + (kv->d.max_rows - used));
        build_prefill_plan(kv->bk.seqs[seq_ids[i]], cache, tokens + off[i], c0, c1, G, P);
        used += c1 - c0;
        done[i] = c1;
        ++nseq;
      }
      if (used == 0) break;
      if ((st = exec_forward(m, kv, cache, P, false, nullptr, 1.f, s))) {
        detach_all();
        return st;
      }
    }
    for (int i = 0; i < n_seqs; ++i) kv->bk.seqs[seq_ids[i]].valid[cache] = lens[i];
  }
  return VIA_OK;
}

via_status via_prefill(via_model* m, via_kv* kv, int32_t seq_id, const int32_t* tokens, int32_t n, void* stream) {
  return via_prefill_batch(m, kv, 1, &seq_id, &n, tokens, stream);
}

via_status via_kv_seq_release(via_kv* kv, int32_t seq_id) {
  if (!kv) return fail(VIA_EINVAL, "null KV handle");
  if (kv->step_open) return fail(VIA_ESTATE, "a step is open");
  if (seq_id < 0 || seq_id >= kv->d.max_seqs || !kv->bk.seqs[seq_id].on) return fail(VIA_EINVAL, "sequence not attached");
  book_trim(kv->bk, 0, seq_id, 0);
  book_trim(kv->bk, 1, seq_id, 0);
  kv->bk.seqs[seq_id] = SeqSt();
  return VIA_OK;
}

via_status via_kv_seq_info(const via_kv* kv, int32_t seq_id, int32_t cache, int32_t* valid, int32_t* table,
                           int32_t cap, int32_t* n_blocks) {
  if (!kv || !valid || !n_blocks) return fail(VIA_EINVAL, "null argument");
  if (cache != 0 && cache != 1) return fail(VIA_EINVAL, "cache must be VIA_CACHE_FULL or VIA_CACHE_SLIM");
  if (seq_id < 0 || seq_id >= kv->d.max_seqs || !kv->bk.seqs[seq_id].on) return fail(VIA_EINVAL, "sequence not attached");
  const SeqSt& S = kv->bk.seqs[seq_id];
  *valid = S.valid[cache];
  *n_blocks = (int)S.table[cache].size();
  if (table) {
    if (cap < *n_blocks) return fail(VIA_EINVAL, "table capacity %d < %d", cap, *n_blocks);
    for (int i = 0; i < *n_blocks; ++i) table[i] = S.table[cache][i];
  }
  return VIA_OK;
}

via_status via_verify_slim(via_model* m, via_kv* kv, const via_window* win, const via_tier_params* p,
                           via_verify_out* out, void* stream) {
  return verify_impl(m, kv, VIA_CACHE_SLIM, win, nullptr, p, out, (hipStream_t)stream, false);
}

via_status via_verify_full(via_model* m, via_kv* kv, const via_window* win, const int32_t* run,
                           const via_tier_params* p, via_verify_out* out, void* stream) {
  return verify_impl(m, kv, VIA_CACHE_FULL, win, run, p, out, (hipStream_t)stream, false);
}

via_status via_verify_probe(via_model* m, via_kv* kv, int32_t cache, const via_window* win,
                            const via_tier_params* p, via_verify_out* out, void* stream) {
  if (cache != 0 && cache != 1) return fail(VIA_EINVAL, "cache must be VIA_CACHE_FULL or VIA_CACHE_SLIM");
  if (kv && kv->step_open) return fail(VIA_ESTATE, "no probe while a step is open (it would overwrite the window rows)");
  return verify_impl(m, kv, cache, win, nullptr, p, out, (hipStream_t)stream, true);
}

via_status decide_impl(via_kv* kv, const via_tier_params* p, const via_verify_out* slim,
                       const via_verify_out* full, const via_sampling* smp, via_decision* dec, void* stream) {
  if (!kv || !dec) return fail(VIA_EINVAL, "null argument");
  if (kv->sticky) return fail(VIA_EDEVICE, "handle has a sticky device error");
  via_status st = check_params(p);
  if (st) return st;
  if ((st = check_out(slim))) return st;
  if (full && (st = check_out(full))) return st;
  if (!dec->tier || !dec->conf || !dec->packed || !dec->h_packed) return fail(VIA_EINVAL, "decision arrays missing");
  if (!kv->step_open) return fail(VIA_ESTATE, "no open step");
  const WinCopy& w = kv->win;
  const Layout& L = kv->L;
  hipStream_t s = (hipStream_t)stream;
  const int B = w.batch, Dd = std::max(1, w.max_drafts);
  if (smp) {
    if (w.tree) return fail(VIA_EUNSUPPORTED, "sampling rules take chain drafts");
    // the residual of Eq. A.3 is defined for beta >= 1 - alpha (App. A)
    if (!(smp->alpha >= 0.f && smp->alpha < 1.f) || !std::isfinite(smp->beta) ||
        !((double)smp->beta >= 1.0 - (double)smp->alpha))
      return fail(VIA_EINVAL, "need 0 <= alpha < 1 and beta >= 1 - alpha");
    if (!smp->draft_probs || !smp->uniforms) return fail(VIA_EINVAL, "draft_probs and uniforms are required");
    if (!slim->logits || (full && !full->logits)) return fail(VIA_EINVAL, "sampling needs the logits outputs");
    for (size_t i = 0; i < (size_t)B * Dd * 3; ++i)
      if (!(smp->uniforms[i] >= 0.f && smp->uniforms[i] < 1.f)) return fail(VIA_EINVAL, "uniforms must lie in [0, 1)");
  }
  // step region: per-sequence state + draft arrays (+ uniforms).  The
  // greedy decision after the slim forward finds them in that forward's
  // plan upload; otherwise (sampling rules, or after the full verifier ran)
  // they are uploaded here.
  const char* base = kv->staged_step;
  if (smp || full || !base) {
    std::vector<char> blob = step_blob(kv, w, kv->step_n, smp ? smp->uniforms : nullptr);
    if ((st = upload(kv, kv->ws + L.step_seqs, blob.data(), blob.size(), s))) return st;
    base = kv->ws + L.step_seqs;
  }
  DecideArgs a{};
  a.seqs = (const StepSeq*)base;
  a.batch = B;
  a.max_rows = w.max_rows;
  a.max_drafts = Dd;
  a.draft_tok = (const int32_t*)(base + (L.dtok - L.step_seqs));
  a.draft_row = (const int32_t*)(base + (L.drow - L.step_seqs));
  a.draft_parent = (const int32_t*)(base + (L.dpar - L.step_seqs));
  a.s_row_max = slim->row_max;
  a.s_row_argmax = slim->row_argmax;
  a.s_draft_logit = slim->draft_logit;
  if (full) {
    a.f_row_max = full->row_max;
    a.f_row_argmax = full->row_argmax;
    a.f_draft_logit = full->draft_logit;
  }
  a.tau_acc = p->tau_acc;
  a.tau_full = p->tau_full;
  a.inv_T = 1.0f / p->temperature;
  a.forced = p->forced;
  a.tier = dec->tier;
  a.conf = dec->conf;
  a.packed = dec->packed;
  if (smp) {
    a.draft_probs = smp->draft_probs;
    a.u = (const float*)(base + (L.du - L.step_seqs));
    a.s_logits = slim->logits;
    a.s_row_sumexp = slim->row_sumexp;
    if (full) {
      a.f_logits = full->logits;
      a.f_row_sumexp = full->row_sumexp;
    }
    a.alpha = smp->alpha;
    a.beta = smp->beta;
    a.vocab = kv->m->d.vocab;
    a.req = (SampleReq*)(kv->ws + L.sreq);
    a.slice_sum = (double*)(kv->ws + L.ssum);
  }
  // greedy rules: the decision kernel writes the pinned host mirror itself
  // when that memory is mapped for the device (no copy on the step's
  // critical path); otherwise, and under the sampling rules (whose draw
  // completes the decision later), the packed block is copied
  if (!smp) {
    if (dec->h_packed != kv->h_packed_host) {
      void* dp = nullptr;
      kv->h_packed_host = dec->h_packed;
      kv->h_packed_dev = hipHostGetDevicePointer(&dp, dec->h_packed, 0) == hipSuccess ? (int32_t*)dp : nullptr;
      (void)hipGetLastError();  // a host pointer that is not mapped leaves no sticky error
    }
    a.h_packed = kv->h_packed_dev;
  }
  timed_launch(kv, VIA_KERNEL_DECIDE, s, [&] { launch_decide(a, s); });
  if ((st = hip_check(kv, hipGetLastError(), "decide launch"))) return st;
  if (a.h_packed) return VIA_OK;
  size_t bytes = (size_t)(4 * B + B * Dd) * 4;
  return hip_check(kv, hipMemcpyAsync(dec->h_packed, dec->packed, bytes, hipMemcpyDeviceToHost, s), "decision copy");
}

via_status via_tier_decide(via_kv* kv, const via_tier_params* p, const via_verify_out* slim,
                           const via_verify_out* full, via_decision* dec, void* stream) {
  return decide_impl(kv, p, slim, full, nullptr, dec, stream);
}

via_status via_tier_decide_sampled(via_kv* kv, const via_tier_params* p, const via_verify_out* slim,
                                   const via_verify_out* full, const via_sampling* smp, via_decision* dec,
                                   void* stream) {
  if (!smp) return fail(VIA_EINVAL, "null sampling parameters");
  return decide_impl(kv, p, slim, full, smp, dec, stream);
}

via_status via_sample_rows(via_kv* kv, const via_verify_out* out, int32_t out_rows, int32_t n, const int32_t* row,
                           float temperature, const float* uniforms, int32_t* tokens, float* probs, int32_t probs_ld,
                           void* stream) {
  if (!kv || !out) return fail(VIA_EINVAL, "null argument");
  if (kv->sticky) return fail(VIA_EDEVICE, "handle has a sticky device error");
  if (n < 0 || n > kv->d.max_batch) return fail(VIA_EINVAL, "need 0 <= n <= max_batch");
  if (!(temperature > 0.f) || !std::isfinite(temperature)) return fail(VIA_EINVAL, "temperature must be > 0");
  if (probs && probs_ld < kv->m->d.vocab) return fail(VIA_EINVAL, "probs_ld must be >= vocab");
  if (n == 0) return VIA_OK;
  if (!out->logits || !out->row_max || !out->row_sumexp || !tokens || !row || !uniforms)
    return fail(VIA_EINVAL, "logits, row statistics, rows, uniforms and tokens are required");
  std::vector<SampleReq> req(n);
  for (int i = 0; i < n; ++i) {
    if (row[i] < 0 || row[i] >= out_rows) return fail(VIA_EINVAL, "row %d outside [0, %d)", row[i], out_rows);
    if (!(uniforms[i] >= 0.f && uniforms[i] < 1.f)) return fail(VIA_EINVAL, "uniforms must lie in [0, 1)");
    req[i] = SampleReq{1, row[i], i, uniforms[i]};
  }
  const Layout& L = kv->L;
  hipStream_t s = (hipStream_t)stream;
  via_status st = upload(kv, kv->ws + L.sreq, req.data(), (size_t)n * sizeof(SampleReq), s);
  if (st) return st;
  DecideArgs a{};
  a.batch = n;
  a.max_drafts = 1;
  a.s_logits = out->logits;
  a.s_row_max = out->row_max;
  a.s_row_sumexp = out->row_sumexp;
  a.inv_T = 1.0f / temperature;
  a.beta = 1.f;
  a.vocab = kv->m->d.vocab;
  a.req = (SampleReq*)(kv->ws + L.sreq);
  a.slice_sum = (double*)(kv->ws + L.ssum);
  a.tok_out = tokens;
  launch_sample_rows(a, probs, probs_ld, s);
  return hip_check(kv, hipGetLastError(), "sample launch");
}

via_status via_kv_seq_set_tokens(via_kv* kv, int32_t seq_id, const int32_t* tokens, int32_t n) {
  if (!kv || (n > 0 && !tokens)) return fail(VIA_EINVAL, "null argument");
  if (kv->step_open) return fail(VIA_ESTATE, "a step is open");
  if (seq_id < 0 || seq_id >= kv->d.max_seqs || !kv->bk.seqs[seq_id].on) return fail(VIA_EINVAL, "sequence not attached");
  SeqSt& S = kv->bk.seqs[seq_id];
  if (n != S.valid[VIA_CACHE_SLIM] + 1)
    return fail(VIA_EINVAL, "n = %d must be the cached length + 1 = %d", n, S.valid[VIA_CACHE_SLIM] + 1);
  for (int i = 0; i < n; ++i)
    if (tokens[i] < 0 || tokens[i] >= kv->m->d.vocab) return fail(VIA_EINVAL, "token %d out of range", tokens[i]);
  S.tokens.assign(tokens, tokens + n);
  S.has_tokens = true;
  return VIA_OK;
}

via_status via_kv_seq_tokens(const via_kv* kv, int32_t seq_id, int32_t* out, int32_t cap, int32_t* n) {
  if (!kv || !n) return fail(VIA_EINVAL, "null argument");
  if (seq_id < 0 || seq_id >= kv->d.max_seqs || !kv->bk.seqs[seq_id].on) return fail(VIA_EINVAL, "sequence not attached");
  const SeqSt& S = kv->bk.seqs[seq_id];
  if (!S.has_tokens) return fail(VIA_ESTATE, "sequence %d has no committed tokens", seq_id);
  *n = (int)S.tokens.size();
  if (out) {
    if (cap < *n) return fail(VIA_EINVAL, "capacity %d < %d", cap, *n);
    std::copy(S.tokens.begin(), S.tokens.end(), out);
  }
  return VIA_OK;
}

via_status via_step(via_model* m, via_kv* kv, const via_drafts* drafts, const via_tier_params* p,
                    via_verify_out* slim, via_verify_out* full, via_decision* dec, void* stream) {
  via_status st = common_checks(m, kv);
  if (st) return st;
  if (!dec || !dec->h_packed || !full) return fail(VIA_EINVAL, "null argument");
  if (kv->step_open) return fail(VIA_ESTATE, "a step is already open");
  hipStream_t s = (hipStream_t)stream;
  StepWin sw;
  if ((st = build_step_window(kv->bk, drafts, false, sw))) return st;
  if ((st = via_verify_slim(m, kv, &sw.win, p, slim, stream))) return st;
  if ((st = via_tier_decide(kv, p, slim, nullptr, dec, stream))) return st;
  if ((st = hip_check(kv, hipStreamSynchronize(s), "hipStreamSynchronize"))) return st;
  const int B = drafts->batch;
  std::vector<int32_t> run(B, 0);
  bool any = false;
  for (int b = 0; b < B; ++b) any |= (run[b] = dec->h_packed[b] == 1) != 0;
  if (any) {
    StepWin lw;
    if ((st = build_step_window(kv->bk, drafts, true, lw))) return st;
    if ((st = via_verify_full(m, kv, &lw.win, run.data(), p, full, stream))) return st;
    if ((st = via_tier_decide(kv, p, slim, full, dec, stream))) return st;
    if ((st = hip_check(kv, hipStreamSynchronize(s), "hipStreamSynchronize"))) return st;
  }
  return via_kv_commit_rollback(kv, dec, stream);
}

static_assert(VIA_STATIC_SAMPLE_MAX_ROWS == kStaticSampleRows, "the header's limit is the scratch's");
static_assert(VIA_STATE_ROWS == kStateRows, "the header's ring size is the runtime's");

via_status via_sample_rows_static(const via_verify_out* out, int32_t out_rows, int32_t vocab, int32_t n,
                                  const int32_t* row, float temperature, const float* uniforms, int32_t* tokens,
                                  float* probs, int32_t probs_ld, void* stream) {
  if (!out) return fail(VIA_EINVAL, "null argument");
  if (vocab < 1) return fail(VIA_EINVAL, "vocab must be >= 1");
  if (n < 0 || n > VIA_STATIC_SAMPLE_MAX_ROWS)
    return fail(VIA_EINVAL, "n = %d outside [0, %d] (the static scratch holds %d requests)", n,
                VIA_STATIC_SAMPLE_MAX_ROWS, VIA_STATIC_SAMPLE_MAX_ROWS);
  if (!(temperature > 0.f) || !std::isfinite(temperature)) return fail(VIA_EINVAL, "temperature must be > 0");
  if (probs && probs_ld < vocab) return fail(VIA_EINVAL, "probs_ld must be >= vocab");
  if (n == 0) return VIA_OK;
  if (!out->logits || !out->row_max || !out->row_sumexp || !tokens || !row || !uniforms)
    return fail(VIA_EINVAL, "logits, row statistics, rows, uniforms and tokens are required");
  std::vector<SampleReq> req(n);
  for (int i = 0; i < n; ++i) {
    if (row[i] < 0 || row[i] >= out_rows) return fail(VIA_EINVAL, "row %d outside [0, %d)", row[i], out_rows);
    if (!(uniforms[i] >= 0.f && uniforms[i] < 1.f)) return fail(VIA_EINVAL, "uniforms must lie in [0, 1)");
    req[i] = SampleReq{1, row[i], i, uniforms[i]};
  }
  void* scr = nullptr;
  size_t scr_bytes = 0;
  hipError_t e = static_scratch(&scr, &scr_bytes);
  if (e != hipSuccess) return fail(VIA_EDEVICE, "static scratch: %s", hipGetErrorString(e));
  DecideArgs a{};
  a.max_drafts = 1;
  a.s_logits = out->logits;
  a.s_row_max = out->row_max;
  a.s_row_sumexp = out->row_sumexp;
  a.inv_T = 1.0f / temperature;
  a.beta = 1.f;
  a.vocab = vocab;
  a.tok_out = tokens;
  launch_sample_rows_static(a, req.data(), n, scr, probs, probs_ld, (hipStream_t)stream);
  e = hipGetLastError();
  if (e != hipSuccess) return fail(VIA_EDEVICE, "sample launch: %s", hipGetErrorString(e));
  return VIA_OK;
}

via_status via_kv_last_full_start(const via_kv* kv, int32_t* route_index) {
  if (!kv || !route_index) return fail(VIA_EINVAL, "null argument");
  *route_index = kv->last_full_start;
  return VIA_OK;
}

via_status via_kv_commit_rollback(via_kv* kv, const via_decision* dec, void* stream) {
  if (!kv || !dec || !dec->h_packed) return fail(VIA_EINVAL, "null argument");
  if (kv->sticky) return fail(VIA_EDEVICE, "handle has a sticky device error");
  if (!kv->step_open) return fail(VIA_ESTATE, "no open step to commit");
  const WinCopy& w = kv->win;
  const int32_t* hp = dec->h_packed;
  // validate everything before touching state
  CommitMoves cm;
  via_status st = plan_commit(kv->bk, w, kv->step_n, hp, kv->m->d.vocab, cm);
  if (st) return st;
  // tree compaction moves (slim cache always, full cache where it ran)
  hipStream_t s = (hipStream_t)stream;
  for (int cache = 0; cache < 2; ++cache) {
    if (cm.moves[cache].empty()) continue;
    const Layout& L = kv->L;
    std::vector<char> blob(L.commit_bytes);
    memcpy(blob.data(), cm.btab[cache].data(), cm.btab[cache].size() * 4);
    memcpy(blob.data() + (L.c_moves - L.c_btab), cm.moves[cache].data(), cm.moves[cache].size() * sizeof(KvMove));
    if ((st = upload(kv, kv->ws + L.c_btab, blob.data(), L.commit_bytes, s))) return st;
    const int slots = cache == VIA_CACHE_FULL ? kv->m->d.n_layers : (int)kv->m->route.size();
    launch_kv_moves(kv->m->bf16, cache == VIA_CACHE_FULL ? kv->d.pool_full : kv->d.pool_slim,
                    cache == VIA_CACHE_FULL ? kv->d.blocks_full : kv->d.blocks_slim, slots, kv->m->d.n_kv_heads,
                    kv->m->d.head_dim, (const int32_t*)(kv->ws + L.c_btab), (const KvMove*)(kv->ws + L.c_moves),
                    (int)cm.moves[cache].size(), s);
    if ((st = hip_check(kv, hipGetLastError(), "compaction launch"))) return st;
  }
  apply_commit(kv->bk, w, hp);
  kv->step_open = false;
  kv->xpref_ok = false;
  kv->staged_step = nullptr;
  return VIA_OK;
}

}  // extern "C"
