// Small kernels of the verification step: embedding gather, the consumers
// of the split-K GEMM partials (residual + RMSNorm, SwiGLU, QKV RoPE + paged
// K/V write), the tier decision with its gate walk, and tree-path K/V
// compaction.
#include <mutex>
#include <vector>

#include "kernels.h"

namespace via {

namespace {

// Split partials of two float4s (offsets o0 and o1): split_load16 issues
// the loads of splits 0..15 (past the last split it re-reads the last one:
// unconditional loads keep the code branch-free), split_reduce16 sums them
// in split order (the re-reads dropped by a select), and split_sum2 does
// both for splits sp0.. with 16 splits of loads in flight per round.
__device__ __forceinline__ void split_load16(const float* P, size_t stride, int ksplit, int sp0, size_t o0, size_t o1,
                                             float4 (&v0)[16], float4 (&v1)[16]) {
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    const size_t base = (size_t)min(sp0 + q, ksplit - 1) * stride;
    v0[q] = *(const float4*)(P + base + o0);
    v1[q] = *(const float4*)(P + base + o1);
  }
}

__device__ __forceinline__ void split_reduce16(int ksplit, int sp0, const float4 (&v0)[16], const float4 (&v1)[16],
                                               float4& s0, float4& s1) {
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    const bool ok = sp0 + q < ksplit;
    s0.x += ok ? v0[q].x : 0.f;
    s0.y += ok ? v0[q].y : 0.f;
    s0.z += ok ? v0[q].z : 0.f;
    s0.w += ok ? v0[q].w : 0.f;
    s1.x += ok ? v1[q].x : 0.f;
    s1.y += ok ? v1[q].y : 0.f;
    s1.z += ok ? v1[q].z : 0.f;
    s1.w += ok ? v1[q].w : 0.f;
  }
}

__device__ __forceinline__ void split_sum2(const float* P, size_t stride, int ksplit, int sp0, size_t o0, size_t o1,
                                           float4& s0, float4& s1) {
  for (int sp = sp0; sp < ksplit; sp += 16) {
    float4 v0[16], v1[16];
    split_load16(P, stride, ksplit, sp, o0, o1, v0, v1);
    split_reduce16(ksplit, sp, v0, v1, s0, s1);
  }
}

// Residual update and RMSNorm gain, elementwise: x = X[m] + sum_s P[s][m]
// (split order; P may be null), X[m] = x, and x * g is written as
// activation fragments (to fragment row rows[m].lm when `rows` is given;
// rows with lm < 0 only update X).  The RMSNorm scale 1/sqrt(mean(x^2)+eps)
// is a per-row factor that commutes with the next projection, so its
// consumer applies it (row_scale) after the GEMM; here each work-group adds
// the sum of x^2 over its kNormChunk columns to ss[chunk][out].
// Grid (ceil(d / kNormChunk), M), 64 threads of 8 columns each.
template <typename G, bool BF16, int NT, int KS>
__global__ __launch_bounds__(64) void resid_add_kernel(float* X, const float* P, int ksplit, int M, int d,
                                                       const G* g, void* Y, int MBn, const RowInfo* rows,
                                                       float* ss, int ss_stride, float* Xcopy, const G* E,
                                                       const RowInfo* erows) {
  const int m = blockIdx.y, chunk = blockIdx.x;
  const int k0 = chunk * kNormChunk + threadIdx.x * 8;
  const int out = rows ? rows[m].lm : m;
  float* x = X + (size_t)m * d;
  if (Xcopy) {  // uniform per work-group
    const int xr = erows ? erows[m].xs : m;
    Xcopy = xr < 0 ? nullptr : Xcopy + (size_t)xr * d;
  }
  const size_t stride = (size_t)M * d;
  float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float sq = 0.f;
  if (k0 < d && E) {
    // embedding rows: X[m] = E[tok]
    const G* e = E + (size_t)erows[m].tok * d + k0;
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = to_f<G>(e[i]);
    *(float4*)(x + k0) = make_float4(v[0], v[1], v[2], v[3]);
    *(float4*)(x + k0 + 4) = make_float4(v[4], v[5], v[6], v[7]);
    if (Xcopy) {
      *(float4*)(Xcopy + k0) = make_float4(v[0], v[1], v[2], v[3]);
      *(float4*)(Xcopy + k0 + 4) = make_float4(v[4], v[5], v[6], v[7]);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) sq += v[i] * v[i];
  } else if (k0 < d) {
    float4 acc[2] = {make_float4(0.f, 0.f, 0.f, 0.f), make_float4(0.f, 0.f, 0.f, 0.f)};
    if constexpr (KS > 0) {
      // exactly KS splits: all loads in flight, then summed in split order
      if (P) {
        float4 v0[KS], v1[KS];
#pragma unroll
        for (int q = 0; q < KS; ++q) {
          v0[q] = *(const float4*)(P + (size_t)q * stride + (size_t)m * d + k0);
          v1[q] = *(const float4*)(P + (size_t)q * stride + (size_t)m * d + k0 + 4);
        }
#pragma unroll
        for (int q = 0; q < KS; ++q) {
          acc[0].x += v0[q].x;
          acc[0].y += v0[q].y;
          acc[0].z += v0[q].z;
          acc[0].w += v0[q].w;
          acc[1].x += v1[q].x;
          acc[1].y += v1[q].y;
          acc[1].z += v1[q].z;
          acc[1].w += v1[q].w;
        }
      }
    } else {
      if (P) split_sum2(P, stride, ksplit, 0, (size_t)m * d + k0, (size_t)m * d + k0 + 4, acc[0], acc[1]);
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      float4 u = *(float4*)(x + k0 + 4 * h);
      if (P) {
        u.x = u.x + acc[h].x;
        u.y = u.y + acc[h].y;
        u.z = u.z + acc[h].z;
        u.w = u.w + acc[h].w;
        *(float4*)(x + k0 + 4 * h) = u;
      }
      if (Xcopy) *(float4*)(Xcopy + k0 + 4 * h) = u;
      v[4 * h + 0] = u.x;
      v[4 * h + 1] = u.y;
      v[4 * h + 2] = u.z;
      v[4 * h + 3] = u.w;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) sq += v[e] * v[e];
  }
  if (out < 0) return;  // uniform per work-group
  sq = wave_sum(sq);
  if (threadIdx.x == 0) ss[(size_t)chunk * ss_stride + out] = sq;
  if (k0 >= d) return;
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = v[e] * to_f<G>(g[k0 + e]);
  put_afrag<BF16, NT>(Y, out, k0, v, d >> 5, MBn);
}

// Many-row form of the residual update (forwards of more than
// kPrefillMinRows rows, one partial P, no head rows or embedding gather):
// a work-group of 64 threads owns one 16-row block of the fragment layout and
// one kNormChunk of columns.  Thread t takes row t % 16 and, in each of the
// chunk's K32 steps s, the 8-column group t / 16, so every fragment store of
// the wave writes one contiguous 1 KB block (the one-row form writes 16 bytes
// every 256).  The values are those of resid_add_kernel: the 8-column group
// 4 s + t / 16 is that kernel's thread, and its partial sums of squares are
// added in that kernel's wave_sum order (three levels within the thread, two
// across lanes).
template <int NT>
__global__ __launch_bounds__(64) void resid_add_rows_kernel(float* X, const float* P, int M, int d, const uint16_t* g,
                                                            void* Y, int MBn, float* ss, int ss_stride, float* Xcopy) {
  constexpr int kSteps = kNormChunk / 32;
  const int chunk = blockIdx.x, t = threadIdx.x, r = t & 15, j = t >> 4;
  const int m = blockIdx.y * 16 + r;
  const bool live = m < M;
  float p[kSteps];
#pragma unroll
  for (int st = 0; st < kSteps; ++st) {
    const int k0 = chunk * kNormChunk + st * 32 + j * 8;
    p[st] = 0.f;
    if (!live || k0 >= d) continue;
    float* x = X + (size_t)m * d + k0;
    const float* a = P + (size_t)m * d + k0;
    float v[8];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      float4 u = *(float4*)(x + 4 * h);
      const float4 b = *(const float4*)(a + 4 * h);
      u.x = u.x + (0.f + b.x);
      u.y = u.y + (0.f + b.y);
      u.z = u.z + (0.f + b.z);
      u.w = u.w + (0.f + b.w);
      *(float4*)(x + 4 * h) = u;
      if (Xcopy) *(float4*)(Xcopy + (size_t)m * d + k0 + 4 * h) = u;
      v[4 * h + 0] = u.x;
      v[4 * h + 1] = u.y;
      v[4 * h + 2] = u.z;
      v[4 * h + 3] = u.w;
    }
    float sq = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) sq += v[e] * v[e];
    p[st] = sq;
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = v[e] * to_f<uint16_t>(g[k0 + e]);
    put_afrag<true, NT>(Y, m, k0, v, d >> 5, MBn);
  }
  // wave_sum over the one-row form's threads T = 4 s + j: lane xor 32, 16, 8
  // and 4 pair steps s ^ 8, s ^ 4, s ^ 2, s ^ 1 (this thread), xor 2 and 1
  // pair groups j ^ 2 and j ^ 1 (lanes t ^ 32 and t ^ 16)
#pragma unroll
  for (int o = kSteps / 2; o > 0; o >>= 1)
#pragma unroll
    for (int st = 0; st < o; ++st) p[st] = p[st] + p[st + o];
  float sq = p[0];
  sq += __shfl_xor(sq, 32, 64);
  sq += __shfl_xor(sq, 16, 64);
  if (j == 0 && live) ss[(size_t)chunk * ss_stride + m] = sq;
}

// Rotate-half RoPE of the pair (j, j + hd/2) of head hh of row m (Q and K
// heads; V passes through) with the angle's cosine and sine, then the store:
// Q as bf16 hi/lo terms (fp32 models: fp32), K and V into the row's paged
// cache slot in the model dtype.
template <typename T>
__device__ __forceinline__ void qkv_store(const QkvArgs& a, const RowInfo& ri, int m, int hh, int j, float x1,
                                          float x2, double cs, double sn) {
  const int half = a.hd >> 1;
  float y1 = x1, y2 = x2;
  if (hh < a.H + a.KVH) {
    y1 = (float)((double)x1 * cs - (double)x2 * sn);
    y2 = (float)((double)x2 * cs + (double)x1 * sn);
  }
  if (hh < a.H) {
    const size_t o = ((size_t)m * a.H + hh) * a.hd + j;
    if constexpr (sizeof(T) == 2) {
      // Q as bf16 hi (truncated) + lo (rounded) terms for the attention MFMAs
      const uint32_t u1 = __float_as_uint(y1) >> 16, u2 = __float_as_uint(y2) >> 16;
      a.q_hi[o] = (uint16_t)u1;
      a.q_hi[o + half] = (uint16_t)u2;
      a.q_lo[o] = f2bf(y1 - __uint_as_float(u1 << 16));
      a.q_lo[o + half] = f2bf(y2 - __uint_as_float(u2 << 16));
    } else {
      float* q = (float*)a.q_hi;
      q[o] = y1;
      q[o + half] = y2;
    }
    return;
  }
  const int blk = ri.blk, t = ri.slot % kBlock;
  T* pool = (T*)a.pool;
  if (hh < a.H + a.KVH) {
    const int gk = hh - a.H;
    pool[k_off(a.layer_slot, blk, a.pool_blocks, a.KVH, a.hd, gk, t, j)] = from_f<T>(y1);
    pool[k_off(a.layer_slot, blk, a.pool_blocks, a.KVH, a.hd, gk, t, j + half)] = from_f<T>(y2);
  } else {
    const int gv = hh - a.H - a.KVH;
    pool[v_off(a.layer_slot, blk, a.pool_blocks, a.KVH, a.hd, gv, t, j)] = from_f<T>(y1);
    pool[v_off(a.layer_slot, blk, a.pool_blocks, a.KVH, a.hd, gv, t, j + half)] = from_f<T>(y2);
  }
}

// The rotation angle of pair j at position pos, pos * theta^(-2j/hd), in fp64.
__device__ __forceinline__ void rope_angle(int pos, int j, const QkvArgs& a, double* sn, double* cs) {
  sincos((double)pos * pow((double)a.theta, -2.0 * (double)j / (double)a.hd), sn, cs);
}

// QKV partial sums -> RMSNorm scale of the input row -> rotate-half RoPE at
// the row's position -> Q (bf16 hi/lo terms, or fp32) and paged K/V (model
// dtype).  A work-group of 256 threads takes four (row, head of Q, K or V)
// pairs, 64 threads each; thread j owns the rotation pair (j, j + hd/2) and
// its angle pos * theta^(-2j/hd), computed in fp64 while the loads of the
// pair's KS split partials (all in flight at once, summed in split order)
// are outstanding.  KS = 0: the split count is taken from the arguments.
template <typename T, int KS>
__global__ __launch_bounds__(256) void qkv_finish_kernel(QkvArgs a) {
  const int m = blockIdx.x, hh = blockIdx.y * 4 + (threadIdx.x >> 6), j = threadIdx.x & 63;
  const int half = a.hd >> 1;
  if (j >= half || hh >= a.H + 2 * a.KVH) return;
  const size_t N = (size_t)(a.H + 2 * a.KVH) * a.hd, stride = (size_t)a.M * N;
  const size_t c = (size_t)m * N + (size_t)hh * a.hd + j;
  float x1 = 0.f, x2 = 0.f;
  double cs = 1.0, sn = 0.0;
  const RowInfo ri = a.rows[m];
  if constexpr (KS > 0) {
    float v1[KS], v2[KS];
#pragma unroll
    for (int q = 0; q < KS; ++q) {
      v1[q] = a.P[(size_t)q * stride + c];
      v2[q] = a.P[(size_t)q * stride + c + half];
    }
    if (hh < a.H + a.KVH) rope_angle(ri.pos, j, a, &sn, &cs);
#pragma unroll
    for (int q = 0; q < KS; ++q) {
      x1 += v1[q];
      x2 += v2[q];
    }
  } else {
    if (hh < a.H + a.KVH) rope_angle(ri.pos, j, a, &sn, &cs);
    for (int q = 0; q < a.ksplit; ++q) {
      x1 += a.P[(size_t)q * stride + c];
      x2 += a.P[(size_t)q * stride + c + half];
    }
  }
  const float sc = row_scale(a.ss, a.ss_stride, m, a.d, a.eps);  // RMSNorm of the input row
  qkv_store<T>(a, ri, m, hh, j, x1 * sc, x2 * sc, cs, sn);
}

// The same for many-row forwards (prefill): one work-group per row.  The
// row's hd/2 angles are computed once and shared through LDS by all its Q and
// K heads (the per-pair form recomputes each one H + KVH times, which makes
// the fp64 transcendentals the cost at thousands of rows); consecutive
// threads then take consecutive pairs of the row's heads.  Same arithmetic,
// same results.
template <typename T>
__global__ __launch_bounds__(256) void qkv_finish_rows_kernel(QkvArgs a) {
  __shared__ double s_cs[64], s_sn[64];  // hd <= 128
  const int m = blockIdx.x, half = a.hd >> 1;
  const RowInfo ri = a.rows[m];
  for (int j = threadIdx.x; j < half; j += 256) rope_angle(ri.pos, j, a, &s_sn[j], &s_cs[j]);
  const float sc = row_scale(a.ss, a.ss_stride, m, a.d, a.eps);  // RMSNorm of the input row
  __syncthreads();
  const int nh = a.H + 2 * a.KVH;
  const size_t N = (size_t)nh * a.hd, stride = (size_t)a.M * N;
  for (int e = threadIdx.x; e < nh * half; e += 256) {
    const int hh = e / half, j = e - hh * half;
    const size_t c = (size_t)m * N + (size_t)hh * a.hd + j;
    float x1 = 0.f, x2 = 0.f;
    for (int q = 0; q < a.ksplit; ++q) {
      x1 += a.P[(size_t)q * stride + c];
      x2 += a.P[(size_t)q * stride + c + half];
    }
    qkv_store<T>(a, ri, m, hh, j, x1 * sc, x2 * sc, s_cs[j], s_sn[j]);
  }
}

// Tier decision and gate walk for one sequence (App. B.1): every draft gets
// its ratio confidence and tier; one lane then walks the draft chain/tree.
__global__ __launch_bounds__(64) void decide_kernel(DecideArgs a) {
  const int b = blockIdx.x;
  const StepSeq ss = a.seqs[b];
  const int D = a.max_drafts, B = a.batch;
  const int base = b * D;
  const bool have_full = a.f_row_max != nullptr && ss.full_ran;
  for (int j = threadIdx.x; j < ss.n_drafts; j += 64) {
    int out = b * a.max_rows + a.draft_row[base + j];
    float c = expf((a.s_draft_logit[base + j] - a.s_row_max[out]) * a.inv_T);
    int t;
    if (a.forced >= 0)
      t = a.forced;
    else if (c >= a.tau_acc)
      t = 0;
    else if (c >= a.tau_full)
      t = 1;
    else
      t = 2;  // also a NaN confidence
    a.conf[base + j] = c;
    a.tier[base + j] = (int8_t)t;
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
  int* status = a.packed;
  int* kappa = a.packed + B;
  int* emit = a.packed + 2 * B;
  int* new_len = a.packed + 3 * B;
  int* path = a.packed + 4 * B + base;
  if (a.draft_probs) {
    // sampling rules (App. A), chain drafts in order: an accept-tier draft is
    // kept; a slim-tier position owes a sample of q'; an escalated draft x is
    // kept with probability min(1, q(x) / ((1 - alpha) p(x))) (Eq. A.2),
    // accepted iff its uniform is below that, else it owes a sample of the
    // A.3 residual.  The owed sample is drawn by the sampling kernels.
    int k = 0, st = 0;
    SampleReq rq{0, 0, 0, 0.f};
    for (int j = 0; j < ss.n_drafts; ++j) {
      const int t = a.tier[base + j];
      const int out = b * a.max_rows + a.draft_row[base + j];
      if (t == 0) {
        path[k++] = j;
        continue;
      }
      if (t == 1) {
        rq = SampleReq{1, out, j, a.u[(size_t)(base + j) * 3 + 1]};
        break;
      }
      if (!have_full) {
        st = 1;
        break;
      }
      const float fm = a.f_row_max[out];
      if (!isfinite(fm)) {
        st = 2;
        break;
      }
      const float qx = expf((a.f_draft_logit[base + j] - fm) * a.inv_T) / a.f_row_sumexp[out];
      const float px = a.draft_probs[(size_t)(base + j) * a.vocab + a.draft_tok[base + j]];
      const float keep = px <= 0.f ? 1.f : fminf(1.f, qx / ((1.f - a.alpha) * px));
      if (a.u[(size_t)(base + j) * 3] < keep) {
        path[k++] = j;
        continue;
      }
      rq = SampleReq{2, out, j, a.u[(size_t)(base + j) * 3 + 2]};
      break;
    }
    if (st != 0) rq.kind = 0;
    a.req[b] = rq;
    status[b] = st;
    kappa[b] = k;
    emit[b] = -1;  // a sample owed is written by sample_pick_kernel
    new_len[b] = st == 2 ? ss.n : ss.n + k + (rq.kind ? 1 : 0);
    for (int q = k; q < D; ++q) path[q] = -1;
    return;
  }
  int u = -1, k = 0, em = -1, st = 0;
  for (;;) {
    // children of u, in draft order
    int best_acc = -1, any_slim = 0, first_kid = -1, nk = 0;
    float best_c = 0.f;
    int kids[kMaxChildren * 8];
    for (int j = 0; j < ss.n_drafts; ++j) {
      if (a.draft_parent[base + j] != u) continue;
      if (first_kid < 0) first_kid = j;
      if (nk < kMaxChildren * 8) kids[nk++] = j;
      int t = a.tier[base + j];
      float c = a.conf[base + j];
      if (t == 0 && (best_acc < 0 || c > best_c)) {
        best_acc = j;
        best_c = c;
      }
      if (t == 1) any_slim = 1;
    }
    if (first_kid < 0) break;  // leaf: whole path accepted, no emit
    const int out = b * a.max_rows + a.draft_row[base + first_kid];
    if (best_acc >= 0) {
      path[k++] = best_acc;
      u = best_acc;
      continue;
    }
    if (any_slim) {
      em = a.s_row_argmax[out];
      break;
    }
    if (!have_full) {
      st = 1;
      break;
    }
    float fm = a.f_row_max[out];
    if (!isfinite(fm)) {  // non-finite logits of q
      st = 2;
      break;
    }
    int gtok = a.f_row_argmax[out], take = -1;
    for (int q = 0; q < nk; ++q)
      if (a.draft_tok[base + kids[q]] == gtok) {
        take = kids[q];
        break;
      }
    if (take >= 0) {
      path[k++] = take;
      u = take;
      continue;
    }
    em = gtok;
    break;
  }
  const int ev = st == 0 ? em : -1;
  const int nv = st == 2 ? ss.n : ss.n + k + (st == 0 && em >= 0 ? 1 : 0);
  status[b] = st;
  kappa[b] = k;
  emit[b] = ev;
  new_len[b] = nv;
  for (int q = k; q < D; ++q) path[q] = -1;
  if (a.h_packed) {
    // the host mirror, written past the caches so that it is in host memory
    // once the stream has been synchronised.  Values come from registers
    // (the path in rounds of 8 loads, then 8 stores): a value re-read from
    // device memory after each store would make every system-scope store
    // wait for a load, one host round trip per value.
    auto put = [&](int i, int v) { __hip_atomic_store(a.h_packed + i, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM); };
    put(b, st);
    put(B + b, k);
    put(2 * B + b, ev);
    put(3 * B + b, nv);
    for (int q0 = 0; q0 < D; q0 += 8) {
      int pv[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) pv[j] = q0 + j < D ? path[q0 + j] : 0;
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (q0 + j < D) put(4 * B + base + q0 + j, pv[j]);
    }
  }
}

// Tree compaction: copy the K/V of slot src to slot dst in every layer slot.
template <typename T>
__global__ __launch_bounds__(128) void kv_move_kernel(T* pool, int nblk, int KVH, int hd, const int32_t* btab,
                                                      const KvMove* moves, int n_moves) {
  const int l = blockIdx.y;  // layer slot
  for (int mv = 0; mv < n_moves; ++mv) {  // in order: destinations never overtake later sources
    const KvMove m = moves[mv];
    int sb = btab[m.bt + m.src / kBlock], st = m.src % kBlock;
    int db = btab[m.bt + m.dst / kBlock], dt = m.dst % kBlock;
    for (int e = threadIdx.x; e < KVH * hd; e += 128) {
      int g = e / hd, i = e % hd;
      pool[k_off(l, db, nblk, KVH, hd, g, dt, i)] = pool[k_off(l, sb, nblk, KVH, hd, g, st, i)];
      pool[v_off(l, db, nblk, KVH, hd, g, dt, i)] = pool[v_off(l, sb, nblk, KVH, hd, g, st, i)];
    }
    __syncthreads();
  }
}

}  // namespace

void launch_resid_add(bool bf16, int terms, float* X, const float* P, int ksplit, int M, int d, const void* g,
                      void* Y, int MBn, const RowInfo* rows, float* ss, int ss_stride, hipStream_t s, float* Xcopy,
                      const void* E, const RowInfo* erows) {
  const dim3 grid((d + kNormChunk - 1) / kNormChunk, M);
  if (bf16 && P && ksplit == 1 && !rows && !E && !erows && M > kPrefillMinRows && (terms == 2 || terms == 3)) {
    const dim3 rgrid((d + kNormChunk - 1) / kNormChunk, (M + 15) / 16);
    if (terms == 3)
      hipLaunchKernelGGL(resid_add_rows_kernel<3>, rgrid, dim3(64), 0, s, X, P, M, d, (const uint16_t*)g, Y, MBn, ss,
                         ss_stride, Xcopy);
    else
      hipLaunchKernelGGL(resid_add_rows_kernel<2>, rgrid, dim3(64), 0, s, X, P, M, d, (const uint16_t*)g, Y, MBn, ss,
                         ss_stride, Xcopy);
    return;
  }
  if (!bf16) {
    hipLaunchKernelGGL((resid_add_kernel<float, false, 1, 0>), grid, dim3(64), 0, s, X, P, ksplit, M, d,
                       (const float*)g, Y, MBn, rows, ss, ss_stride, Xcopy, (const float*)E, erows);
    return;
  }
  auto go = [&](auto kernel) {
    hipLaunchKernelGGL(kernel, grid, dim3(64), 0, s, X, P, ksplit, M, d, (const uint16_t*)g, Y, MBn, rows, ss,
                       ss_stride, Xcopy, (const uint16_t*)E, erows);
  };
  // the split counts of the projections that feed it get their exact loads
  if (terms >= 3) {
    switch (P ? ksplit : 0) {
      case 4: go(resid_add_kernel<uint16_t, true, 3, 4>); break;
      case 8: go(resid_add_kernel<uint16_t, true, 3, 8>); break;
      default: go(resid_add_kernel<uint16_t, true, 3, 0>); break;
    }
  } else {
    switch (P ? ksplit : 0) {
      case 4: go(resid_add_kernel<uint16_t, true, 2, 4>); break;
      case 8: go(resid_add_kernel<uint16_t, true, 2, 8>); break;
      default: go(resid_add_kernel<uint16_t, true, 2, 0>); break;
    }
  }
}

void launch_qkv_finish(bool bf16, const QkvArgs& a, hipStream_t s) {
  if (a.M > kPrefillMinRows && a.hd <= 128) {  // many rows: angles shared per row
    if (bf16)
      hipLaunchKernelGGL(qkv_finish_rows_kernel<uint16_t>, dim3(a.M), dim3(256), 0, s, a);
    else
      hipLaunchKernelGGL(qkv_finish_rows_kernel<float>, dim3(a.M), dim3(256), 0, s, a);
    return;
  }
  const dim3 grid(a.M, (a.H + 2 * a.KVH + 3) / 4);
  auto go = [&](auto kernel) { hipLaunchKernelGGL(kernel, grid, dim3(256), 0, s, a); };
  if (bf16) {
    switch (a.ksplit) {
      case 1: go(qkv_finish_kernel<uint16_t, 1>); break;
      case 2: go(qkv_finish_kernel<uint16_t, 2>); break;
      case 4: go(qkv_finish_kernel<uint16_t, 4>); break;
      default: go(qkv_finish_kernel<uint16_t, 0>); break;
    }
  } else {
    go(qkv_finish_kernel<float, 0>);
  }
}

namespace {

// Owed samples (App. A): the token a uniform u draws from weights w(v),
// v < V, is the first v in id order whose running sum exceeds u * sum(w)
// (the last token with weight when rounding leaves no crossing).  Weights:
// kind 1 the slim row's exp((l - max) / T); kind 2 the A.3 residual
// max(0, q / beta - p), q = exp((l - max) / T) / sum, or q itself when the
// residual has no mass.
//
// The vocabulary is cut into slices of kSampleThreads * E ids; thread t of a
// slice owns the E consecutive ids starting at t * E.  Sums are fp64 in one
// fixed grouping, shared by both kernels: a thread's ids in order; four
// consecutive threads in order per lane of wave 0; a 64-lane inclusive scan.
// sample_sums_kernel (one work-group per slice and sequence) writes each
// slice's residual and q sums; sample_pick_kernel (one per sequence) finds
// the crossing slice from them, rescans that slice with the same grouping,
// and walks the crossing lane, thread and id.
constexpr int kSampleThreads = 256;

struct SampleGeom {
  int E, slice, G;
};
__host__ __device__ inline SampleGeom sample_geom(int V) {
  int E = (V + kSampleSlices * kSampleThreads - 1) / (kSampleSlices * kSampleThreads);
  if (E < 1) E = 1;
  const int slice = E * kSampleThreads;
  return SampleGeom{E, slice, (V + slice - 1) / slice};
}

struct SampleRow {
  const float* lg;
  const float* p;
  float mx, inv_z, inv_T, inv_beta;
};
__device__ inline SampleRow sample_row(const DecideArgs& a, const SampleReq& r, int b) {
  const size_t V = (size_t)a.vocab;
  SampleRow w;
  w.lg = (r.kind == 1 ? a.s_logits : a.f_logits) + (size_t)r.out * V;
  w.p = a.draft_probs + (size_t)(b * a.max_drafts + r.j) * V;
  w.mx = r.kind == 1 ? a.s_row_max[r.out] : a.f_row_max[r.out];
  w.inv_z = r.kind == 2 ? 1.f / a.f_row_sumexp[r.out] : 1.f;
  w.inv_T = a.inv_T;
  w.inv_beta = 1.f / a.beta;
  return w;
}
// q-weight of id v (kind 1: unnormalised q', kind 2: q)
__device__ inline float q_weight(const SampleRow& w, int v) { return expf((w.lg[v] - w.mx) * w.inv_T) * w.inv_z; }
__device__ inline float r_weight(const SampleRow& w, int v, float q) { return fmaxf(0.f, q * w.inv_beta - w.p[v]); }

// Inclusive scan of one fp64 value over the 64 lanes of a wave.
__device__ inline double wave_scan(double x, int lane) {
  for (int d = 1; d < 64; d <<= 1) {
    const double y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  return x;
}

// Thread sums of one slice (both weight kinds) into LDS.
__device__ inline void slice_thread_sums(const SampleRow& w, int kind, int V, const SampleGeom& g, int slice_id,
                                         double* tq, double* tr) {
  const int t = threadIdx.x;
  const int lo = slice_id * g.slice + t * g.E;
  double sq = 0.0, sr = 0.0;
  for (int e = 0; e < g.E; ++e) {
    const int v = lo + e;
    if (v >= V) break;
    const float q = q_weight(w, v);
    sq += (double)q;
    if (kind == 2) sr += (double)r_weight(w, v, q);
  }
  tq[t] = sq;
  tr[t] = sr;
}

// Lane sums (four threads in order) and their inclusive scan, wave 0.
__device__ inline double lane_scan(const double* ts, int lane, double* lane_sum) {
  const double x = ((ts[4 * lane] + ts[4 * lane + 1]) + ts[4 * lane + 2]) + ts[4 * lane + 3];
  *lane_sum = x;
  return wave_scan(x, lane);
}

__global__ __launch_bounds__(kSampleThreads) void sample_sums_kernel(DecideArgs a) {
  const int b = blockIdx.y, g = blockIdx.x;
  const SampleReq r = a.req[b];
  if (r.kind == 0) return;  // uniform per work-group
  const SampleGeom geo = sample_geom(a.vocab);
  __shared__ double tq[kSampleThreads], tr[kSampleThreads];
  const SampleRow w = sample_row(a, r, b);
  slice_thread_sums(w, r.kind, a.vocab, geo, g, tq, tr);
  __syncthreads();
  if (threadIdx.x >= 64) return;
  const int lane = threadIdx.x;
  double ls;
  const double iq = lane_scan(tq, lane, &ls);
  const double ir = lane_scan(tr, lane, &ls);
  if (lane == 63) {
    double* out = a.slice_sum + ((size_t)b * kSampleSlices + g) * 2;
    out[0] = iq;
    out[1] = ir;
  }
}

__global__ __launch_bounds__(kSampleThreads) void sample_pick_kernel(DecideArgs a) {
  const int b = blockIdx.x;
  const SampleReq r = a.req[b];
  if (r.kind == 0) return;  // uniform per work-group
  const int V = a.vocab;
  const SampleGeom geo = sample_geom(V);
  const SampleRow w = sample_row(a, r, b);
  const int t = threadIdx.x, lane = t & 63;
  __shared__ double tq[kSampleThreads], tr[kSampleThreads];
  __shared__ int s_slice, s_last, s_resid;
  __shared__ double s_acc, s_target;
  if (t < 64) {
    // slice level: totals, the weights in use, the crossing slice
    const double* ssum = a.slice_sum + (size_t)b * kSampleSlices * 2;
    const double xq = lane < geo.G ? ssum[lane * 2] : 0.0, xr = lane < geo.G ? ssum[lane * 2 + 1] : 0.0;
    const double iq = wave_scan(xq, lane), ir = wave_scan(xr, lane);
    const double tot_r = __shfl(ir, 63, 64);
    const bool resid = r.kind == 2 && tot_r > 0.0;
    const double x = resid ? xr : xq, inc = resid ? ir : iq;
    const double tot = __shfl(inc, 63, 64);
    const double target = (double)r.u * tot;
    // crossings only at slices with weight (sums of zeros may round apart)
    const unsigned long long cross = __ballot(lane < geo.G && x > 0.0 && inc > target);
    const unsigned long long pos = __ballot(x > 0.0);
    if (lane == 0) {
      int c, last = 0;
      if (cross) {
        c = __ffsll((long long)cross) - 1;
      } else {
        c = pos ? 63 - __clzll((long long)pos) : 0;
        last = 1;
      }
      s_slice = c;
      s_last = last;
      s_resid = resid ? 1 : 0;
      s_target = target;
    }
    // running sum before the crossing slice: the previous lane's prefix
    const int c = cross ? __ffsll((long long)cross) - 1 : 0;
    const double before = __shfl(inc, c > 0 ? c - 1 : 0, 64);
    if (lane == 0) s_acc = c > 0 ? before : 0.0;
  }
  __syncthreads();
  const int c = s_slice;
  const bool resid = s_resid != 0;
  slice_thread_sums(w, resid ? 2 : 1, V, geo, c, tq, tr);
  __syncthreads();
  if (t >= 64) return;
  const double* ts = resid ? tr : tq;
  double ls;
  const double inc = lane_scan(ts, lane, &ls);
  const double target = s_target;
  const double run0 = s_acc;
  bool last = s_last != 0;
  unsigned long long cross = last ? 0ull : __ballot(ls > 0.0 && run0 + inc > target);
  if (!cross) last = true;
  const unsigned long long pos = __ballot(ls > 0.0);
  int L;
  if (!last)
    L = __ffsll((long long)cross) - 1;
  else
    L = pos ? 63 - __clzll((long long)pos) : 0;
  if (lane != L) return;
  // the chosen lane: its four threads in order, then the chosen thread's ids
  double run = run0 + (inc - ls);
  int th = -1;
  if (!last) {
    for (int i = 0; i < 4; ++i) {
      const double v = ts[4 * L + i];
      if (v > 0.0 && run + v > target) {
        th = 4 * L + i;
        break;
      }
      run += v;
    }
  }
  bool take_last = th < 0;
  if (take_last) {
    th = 4 * L;
    for (int i = 3; i >= 0; --i)
      if (ts[4 * L + i] > 0.0) {
        th = 4 * L + i;
        break;
      }
  }
  const int lo = c * geo.slice + th * geo.E;
  int tok = -1, lastpos = lo < V ? lo : V - 1;
  for (int e = 0; e < geo.E; ++e) {
    const int v = lo + e;
    if (v >= V) break;
    const float q = q_weight(w, v);
    const float wt = resid ? r_weight(w, v, q) : q;
    if (wt > 0.f) {
      lastpos = v;
      run += (double)wt;
      if (!take_last && run > target) {
        tok = v;
        break;
      }
    }
  }
  const int drawn = tok >= 0 ? tok : lastpos;
  if (a.tok_out)
    a.tok_out[b] = drawn;
  else
    a.packed[2 * a.batch + b] = drawn;
}

// probs[i * ld + v] = exp((l - max) / T) / sum for request i's row.
__global__ __launch_bounds__(kSampleThreads) void sample_probs_kernel(DecideArgs a, float* probs, int ld) {
  const int i = blockIdx.y;
  const SampleReq r = a.req[i];
  const SampleGeom geo = sample_geom(a.vocab);
  const float* lg = a.s_logits + (size_t)r.out * a.vocab;
  const float mx = a.s_row_max[r.out], inv_z = 1.f / a.s_row_sumexp[r.out];
  float* o = probs + (size_t)i * ld;
  const int lo = blockIdx.x * geo.slice;
  const int hi = min(a.vocab, lo + geo.slice);
  for (int v = lo + threadIdx.x; v < hi; v += kSampleThreads) o[v] = expf((lg[v] - mx) * a.inv_T) * inv_z;
}

}  // namespace

void launch_decide(const DecideArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(decide_kernel, dim3(a.batch), dim3(64), 0, s, a);
  if (a.draft_probs) {
    const SampleGeom g = sample_geom(a.vocab);
    hipLaunchKernelGGL(sample_sums_kernel, dim3(g.G, a.batch), dim3(kSampleThreads), 0, s, a);
    hipLaunchKernelGGL(sample_pick_kernel, dim3(a.batch), dim3(kSampleThreads), 0, s, a);
  }
}

void launch_sample_rows(const DecideArgs& a, float* probs, int probs_ld, hipStream_t s) {
  const SampleGeom g = sample_geom(a.vocab);
  hipLaunchKernelGGL(sample_sums_kernel, dim3(g.G, a.batch), dim3(kSampleThreads), 0, s, a);
  hipLaunchKernelGGL(sample_pick_kernel, dim3(a.batch), dim3(kSampleThreads), 0, s, a);
  if (probs) hipLaunchKernelGGL(sample_probs_kernel, dim3(g.G, a.batch), dim3(kSampleThreads), 0, s, a, probs, probs_ld);
}

// ---------------------------------------------------------------- draws without allocation
// Scratch of the draw entry point that allocates nothing (via_sample_rows_static):
// the request array, then the per-slice sums [request][slice][2].  Each GPU
// holds its own copy until the process ends; every call on a GPU reuses it.
namespace {
constexpr size_t kStaticReqBytes = (size_t)kStaticSampleRows * sizeof(SampleReq);
constexpr size_t kStaticScratchBytes = kStaticReqBytes + (size_t)kStaticSampleRows * kSampleSlices * 2 * sizeof(double);
static_assert(kStaticScratchBytes == 66560, "the size include/via.h states");
static __device__ __align__(256) char scratch[kStaticScratchBytes];

// Requests travel as kernel arguments (no host buffer, no copy).
struct StaticReqs {
  SampleReq r[kStaticSampleRows];
  int n;
};
__global__ __launch_bounds__(kStaticSampleRows) void put_reqs_kernel(StaticReqs q, SampleReq* dst) {
  const int i = threadIdx.x;
  if (i < q.n) dst[i] = q.r[i];
}
}  // namespace

hipError_t static_scratch(void** ptr, size_t* bytes) {
  // the array's device address, looked up once per device with that device current
  static std::mutex mu;
  static std::vector<void*> addr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  if ((size_t)dev >= addr.size()) addr.resize(dev + 1, nullptr);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  *bytes = kStaticScratchBytes;
  return hipSuccess;
}

void launch_sample_rows_static(DecideArgs a, const SampleReq* req, int n, void* scratch_ptr, float* probs,
                               int probs_ld, hipStream_t s) {
  StaticReqs q{};
  for (int i = 0; i < n; ++i) q.r[i] = req[i];
  q.n = n;
  char* base = (char*)scratch_ptr;
  a.req = (SampleReq*)base;
  a.slice_sum = (double*)(base + kStaticReqBytes);
  a.batch = n;
  hipLaunchKernelGGL(put_reqs_kernel, dim3(1), dim3(kStaticSampleRows), 0, s, q, a.req);
  launch_sample_rows(a, probs, probs_ld, s);
}

void launch_kv_moves(bool bf16, void* pool, int pool_blocks, int n_slots, int KVH, int hd, const int32_t* btab,
                     const KvMove* moves, int n_moves, hipStream_t s) {
  if (n_moves <= 0) return;
  if (bf16)
    hipLaunchKernelGGL(kv_move_kernel<uint16_t>, dim3(1, n_slots), dim3(128), 0, s, (uint16_t*)pool, pool_blocks,
                       KVH, hd, btab, moves, n_moves);
  else
    hipLaunchKernelGGL(kv_move_kernel<float>, dim3(1, n_slots), dim3(128), 0, s, (float*)pool, pool_blocks, KVH,
                       hd, btab, moves, n_moves);
}


namespace {

// Forward that starts after the layers the two routes share (route layer
// i == i for i < a.P): grid (M, P + 1).  y < P: the row's K and V of layer
// y, copied from the source cache (slot y) to the destination cache (slot y)
// at the row's position; y == P: the row's residual stream after layer
// P - 1.  A verify step's full forward copies slim -> full and takes the
// state from the state ring (saved there by the slim forward that fed the
// slot: this step's for window rows, an earlier one for lag rows); a
// prefill's slim forward copies full -> slim and takes the state its full
// forward saved for the same rows.
template <typename T>
__global__ __launch_bounds__(256) void prefix_copy_kernel(PrefixArgs a) {
  const int m = blockIdx.x, y = blockIdx.y;
  const PrefixXfer x = a.xfer[m];
  if (y == a.P) {
    const float* src = a.xstate + (size_t)x.src_row * a.d;
    float* dst = a.X + (size_t)m * a.d;
    for (int i = threadIdx.x; i < a.d; i += 256) dst[i] = src[i];
    return;
  }
  const T* sp = (const T*)a.src_pool;
  T* dp = (T*)a.dst_pool;
  const int n = a.KVH * a.hd;
  for (int e = threadIdx.x; e < 2 * n; e += 256) {
    const int g = (e % n) / a.hd, i = e % a.hd;
    if (e < n)
      dp[k_off(y, x.dst_blk, a.dst_blocks, a.KVH, a.hd, g, x.t, i)] =
          sp[k_off(y, x.src_blk, a.src_blocks, a.KVH, a.hd, g, x.t, i)];
    else
      dp[v_off(y, x.dst_blk, a.dst_blocks, a.KVH, a.hd, g, x.t, i)] =
          sp[v_off(y, x.src_blk, a.src_blocks, a.KVH, a.hd, g, x.t, i)];
  }
}

}  // namespace

void launch_prefix_copy(bool bf16, const PrefixArgs& a, hipStream_t s) {
  const dim3 grid(a.M, a.P + 1);
  if (bf16)
    hipLaunchKernelGGL(prefix_copy_kernel<uint16_t>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(prefix_copy_kernel<float>, grid, dim3(256), 0, s, a);
}

}  // namespace via
