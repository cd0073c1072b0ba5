// Small kernels of the verification step: embedding gather, the consumers
// of the split-K GEMM partials (residual + RMSNorm, SwiGLU, QKV RoPE + paged
// K/V write), the tier decision with its gate walk, and tree-path K/V
// compaction.
#include "kernels.h"

namespace via {

namespace {

template <typename T>
__global__ __launch_bounds__(256) void embed_kernel(const T* E, const RowInfo* rows, int d, float* X) {
  const int m = blockIdx.x;
  const T* e = E + (size_t)rows[m].tok * d;
  for (int i = threadIdx.x; i < d; i += 256) X[(size_t)m * d + i] = to_f<T>(e[i]);
}

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
template <typename G, bool BF16, int NT>
__global__ __launch_bounds__(64) void resid_add_kernel(float* X, const float* P, int ksplit, int M, int d,
                                                       const G* g, void* Y, int MBn, const RowInfo* rows,
                                                       float* ss, int ss_stride, float* Xcopy) {
  const int m = blockIdx.y, chunk = blockIdx.x;
  const int k0 = chunk * kNormChunk + threadIdx.x * 8;
  const int out = rows ? rows[m].lm : m;
  float* x = X + (size_t)m * d;
  const size_t stride = (size_t)M * d;
  float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float sq = 0.f;
  if (k0 < d) {
    float4 acc[2] = {make_float4(0.f, 0.f, 0.f, 0.f), make_float4(0.f, 0.f, 0.f, 0.f)};
    if (P) split_sum2(P, stride, ksplit, 0, (size_t)m * d + k0, (size_t)m * d + k0 + 4, acc[0], acc[1]);
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
      if (Xcopy) *(float4*)(Xcopy + (size_t)m * d + k0 + 4 * h) = u;
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

// QKV partial sums -> RMSNorm scale of the input row -> rotate-half RoPE at
// the row's position -> Q (bf16 hi/lo terms, or fp32) and paged K/V (model
// dtype).  One work-group of 64 threads per (row, head of Q, K or V); thread
// j owns the rotation pair (j, j + hd/2) and its angle pos * theta^(-2j/hd),
// computed in fp64 while the loads of the pair's split partials (all in
// flight at once, summed in split order) are outstanding.
template <typename T>
__global__ __launch_bounds__(64) void qkv_finish_kernel(QkvArgs a) {
  const int m = blockIdx.x, hh = blockIdx.y, j = threadIdx.x;
  const int half = a.hd >> 1;
  if (j >= half) return;
  const size_t N = (size_t)(a.H + 2 * a.KVH) * a.hd, stride = (size_t)a.M * N;
  const size_t c = (size_t)m * N + (size_t)hh * a.hd + j;
  float v1[16], v2[16];
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    const size_t base = (size_t)min(q, a.ksplit - 1) * stride;
    v1[q] = a.P[base + c];
    v2[q] = a.P[base + c + half];
  }
  const RowInfo ri = a.rows[m];
  double cs = 1.0, sn = 0.0;
  if (hh < a.H + a.KVH) sincos((double)ri.pos * pow((double)a.theta, -2.0 * (double)j / (double)a.hd), &sn, &cs);
  const float sc = row_scale(a.ss, a.ss_stride, m, a.d, a.eps);  // RMSNorm of the input row
  float x1 = 0.f, x2 = 0.f;
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    x1 += q < a.ksplit ? v1[q] : 0.f;
    x2 += q < a.ksplit ? v2[q] : 0.f;
  }
  for (int sp = 16; sp < a.ksplit; ++sp) {
    x1 += a.P[(size_t)sp * stride + c];
    x2 += a.P[(size_t)sp * stride + c + half];
  }
  x1 *= sc;
  x2 *= sc;
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
  const SeqInfo si = a.seqs[ri.seq];
  const int blk = a.btab[si.bt + ri.slot / kBlock], t = ri.slot % kBlock;
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
  status[b] = st;
  kappa[b] = k;
  emit[b] = st == 0 ? em : -1;
  new_len[b] = st == 2 ? ss.n : ss.n + k + (st == 0 && em >= 0 ? 1 : 0);
  for (int q = k; q < D; ++q) path[q] = -1;
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

void launch_embed(bool bf16, const void* E, const RowInfo* rows, int M, int d, float* X, hipStream_t s) {
  if (bf16)
    hipLaunchKernelGGL(embed_kernel<uint16_t>, dim3(M), dim3(256), 0, s, (const uint16_t*)E, rows, d, X);
  else
    hipLaunchKernelGGL(embed_kernel<float>, dim3(M), dim3(256), 0, s, (const float*)E, rows, d, X);
}

void launch_resid_add(bool bf16, int terms, float* X, const float* P, int ksplit, int M, int d, const void* g,
                      void* Y, int MBn, const RowInfo* rows, float* ss, int ss_stride, hipStream_t s, float* Xcopy) {
  const dim3 grid((d + kNormChunk - 1) / kNormChunk, M);
  if (!bf16)
    hipLaunchKernelGGL((resid_add_kernel<float, false, 1>), grid, dim3(64), 0, s, X, P, ksplit, M, d,
                       (const float*)g, Y, MBn, rows, ss, ss_stride, Xcopy);
  else if (terms >= 3)
    hipLaunchKernelGGL((resid_add_kernel<uint16_t, true, 3>), grid, dim3(64), 0, s, X, P, ksplit, M, d,
                       (const uint16_t*)g, Y, MBn, rows, ss, ss_stride, Xcopy);
  else
    hipLaunchKernelGGL((resid_add_kernel<uint16_t, true, 2>), grid, dim3(64), 0, s, X, P, ksplit, M, d,
                       (const uint16_t*)g, Y, MBn, rows, ss, ss_stride, Xcopy);
}

void launch_qkv_finish(bool bf16, const QkvArgs& a, hipStream_t s) {
  const dim3 grid(a.M, a.H + 2 * a.KVH);
  if (bf16)
    hipLaunchKernelGGL(qkv_finish_kernel<uint16_t>, grid, dim3(64), 0, s, a);
  else
    hipLaunchKernelGGL(qkv_finish_kernel<float>, grid, dim3(64), 0, s, a);
}

void launch_decide(const DecideArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(decide_kernel, dim3(a.batch), dim3(64), 0, s, a);
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

// Full forward that starts after the layers it shares with the slim route
// (route layer i == i for i < a.P): grid (M, P + 1).  y < P: the row's K and
// V of layer y, copied from the slim cache (slot y) to the full cache (slot
// y) at the row's position; y == P: the row's residual stream after layer
// P - 1, taken from the slim forward of the same step.
template <typename T>
__global__ __launch_bounds__(256) void prefix_copy_kernel(PrefixArgs a) {
  const int m = blockIdx.x, y = blockIdx.y;
  const PrefixXfer x = a.xfer[m];
  if (y == a.P) {
    const float* src = a.Xpref + (size_t)x.src_row * a.d;
    float* dst = a.X + (size_t)m * a.d;
    for (int i = threadIdx.x; i < a.d; i += 256) dst[i] = src[i];
    return;
  }
  const T* sp = (const T*)a.slim_pool;
  T* dp = (T*)a.full_pool;
  const int n = a.KVH * a.hd;
  for (int e = threadIdx.x; e < 2 * n; e += 256) {
    const int g = (e % n) / a.hd, i = e % a.hd;
    if (e < n)
      dp[k_off(y, x.dst_blk, a.full_blocks, a.KVH, a.hd, g, x.t, i)] =
          sp[k_off(y, x.src_blk, a.slim_blocks, a.KVH, a.hd, g, x.t, i)];
    else
      dp[v_off(y, x.dst_blk, a.full_blocks, a.KVH, a.hd, g, x.t, i)] =
          sp[v_off(y, x.src_blk, a.slim_blocks, a.KVH, a.hd, g, x.t, i)];
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
