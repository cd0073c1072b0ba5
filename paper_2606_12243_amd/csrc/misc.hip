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

// Sum of the split partials of one float4, in split order (4 loads in flight).
__device__ __forceinline__ float4 split_sum4(const float* P, size_t stride, int ksplit, size_t off) {
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  int sp = 0;
  for (; sp + 4 <= ksplit; sp += 4) {
    float4 v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = *(const float4*)(P + (size_t)(sp + q) * stride + off);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      acc.x += v[q].x;
      acc.y += v[q].y;
      acc.z += v[q].z;
      acc.w += v[q].w;
    }
  }
  for (; sp < ksplit; ++sp) {
    const float4 v = *(const float4*)(P + (size_t)sp * stride + off);
    acc.x += v.x;
    acc.y += v.y;
    acc.z += v.z;
    acc.w += v.w;
  }
  return acc;
}

// x = X[m] + sum_s P[s][m] (split order); X[m] = x; y = x / sqrt(mean(x^2) + eps) * g,
// written as activation fragments (row rows[m].lm when `rows` is given).
// One work-group per row; d is a multiple of 64, each thread owns float4s.
template <typename G, bool BF16, int NT>
__global__ __launch_bounds__(1024) void resid_norm_kernel(float* X, const float* P, int ksplit, int M, int d,
                                                          const G* g, float eps, void* Y, int MBn,
                                                          const RowInfo* rows) {
  __shared__ float red[1024];
  const int m = blockIdx.x;
  float* x = X + (size_t)m * d;
  const size_t stride = (size_t)M * d;
  float ss = 0.f;
  for (int i = threadIdx.x * 4; i < d; i += 4096) {
    float4 v = *(float4*)(x + i);
    if (P) {
      const float4 acc = split_sum4(P, stride, ksplit, (size_t)m * d + i);
      v.x = v.x + acc.x;
      v.y = v.y + acc.y;
      v.z = v.z + acc.z;
      v.w = v.w + acc.w;
      *(float4*)(x + i) = v;
    }
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  red[threadIdx.x] = ss;
  __syncthreads();
  for (int o = 512; o > 0; o >>= 1) {
    if (threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  const int out = rows ? rows[m].lm : m;
  if (out < 0) return;
  const float inv = 1.0f / sqrtf(red[0] / (float)d + eps);
  for (int k0 = threadIdx.x * 8; k0 < d; k0 += 8192) {
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = x[k0 + e] * inv * to_f<G>(g[k0 + e]);
    put_afrag<BF16, NT>(Y, out, k0, v, d >> 5, MBn);
  }
}

// h = silu(gate) * up from the gate/up partial sums, as fragments; grid (M, F / 2048).
template <bool BF16, int NT>
__global__ __launch_bounds__(256) void swiglu_kernel(const float* P, int ksplit, int M, int F, void* H, int MBn) {
  const int m = blockIdx.x;
  const int f = blockIdx.y * 2048 + threadIdx.x * 8;
  if (f >= F) return;
  const size_t N = 2 * (size_t)F, stride = (size_t)M * N;
  float v[8];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const float4 gt = split_sum4(P, stride, ksplit, (size_t)m * N + f + 4 * h);
    const float4 up = split_sum4(P, stride, ksplit, (size_t)m * N + F + f + 4 * h);
    v[4 * h + 0] = gt.x / (1.0f + expf(-gt.x)) * up.x;
    v[4 * h + 1] = gt.y / (1.0f + expf(-gt.y)) * up.y;
    v[4 * h + 2] = gt.z / (1.0f + expf(-gt.z)) * up.z;
    v[4 * h + 3] = gt.w / (1.0f + expf(-gt.w)) * up.w;
  }
  put_afrag<BF16, NT>(H, m, f, v, F >> 5, MBn);
}

// QKV partial sums -> rotate-half RoPE -> Q (fp32) and paged K/V (model
// dtype); grid (M, H + 2 KVH), thread i owns the pair (i, i + hd/2).
template <typename T>
__global__ __launch_bounds__(64) void qkv_finish_kernel(QkvArgs a) {
  const int m = blockIdx.x, hh = blockIdx.y, i = threadIdx.x;
  const int half = a.hd >> 1;
  if (i >= half) return;
  const RowInfo ri = a.rows[m];
  const size_t N = (size_t)(a.H + 2 * a.KVH) * a.hd, stride = (size_t)a.M * N;
  const size_t c = (size_t)m * N + (size_t)hh * a.hd + i;
  float x1 = 0.f, x2 = 0.f;
  for (int sp = 0; sp < a.ksplit; ++sp) {
    x1 += a.P[sp * stride + c];
    x2 += a.P[sp * stride + c + half];
  }
  float y1 = x1, y2 = x2;
  if (hh < a.H + a.KVH) {
    // angle pos * theta^(-2i/hd) and the rotation in fp64
    const double inv = pow((double)a.theta, -2.0 * (double)i / (double)a.hd);
    const double ang = (double)ri.pos * inv;
    const double cs = cos(ang), sn = sin(ang);
    y1 = (float)((double)x1 * cs - (double)x2 * sn);
    y2 = (float)((double)x2 * cs + (double)x1 * sn);
  }
  if (hh < a.H) {
    const size_t o = ((size_t)m * a.H + hh) * a.hd + i;
    if constexpr (sizeof(T) == 2) {
      // Q as bf16 hi (truncated) + lo (rounded) terms for the attention MFMAs
      const uint32_t h1 = __float_as_uint(y1) >> 16, h2 = __float_as_uint(y2) >> 16;
      a.q_hi[o] = (uint16_t)h1;
      a.q_hi[o + half] = (uint16_t)h2;
      a.q_lo[o] = f2bf(y1 - __uint_as_float(h1 << 16));
      a.q_lo[o + half] = f2bf(y2 - __uint_as_float(h2 << 16));
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
    pool[k_off(a.layer_slot, blk, a.pool_blocks, a.KVH, a.hd, gk, t, i)] = from_f<T>(y1);
    pool[k_off(a.layer_slot, blk, a.pool_blocks, a.KVH, a.hd, gk, t, i + half)] = from_f<T>(y2);
  } else {
    const int gv = hh - a.H - a.KVH;
    pool[v_off(a.layer_slot, blk, a.pool_blocks, a.KVH, a.hd, gv, t, i)] = from_f<T>(y1);
    pool[v_off(a.layer_slot, blk, a.pool_blocks, a.KVH, a.hd, gv, t, i + half)] = from_f<T>(y2);
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

void launch_resid_norm(bool bf16, int terms, float* X, const float* P, int ksplit, int M, int d, const void* g,
                       float eps, void* Y, int MBn, const RowInfo* rows, hipStream_t s) {
  if (!bf16)
    hipLaunchKernelGGL((resid_norm_kernel<float, false, 1>), dim3(M), dim3(1024), 0, s, X, P, ksplit, M, d,
                       (const float*)g, eps, Y, MBn, rows);
  else if (terms >= 3)
    hipLaunchKernelGGL((resid_norm_kernel<uint16_t, true, 3>), dim3(M), dim3(1024), 0, s, X, P, ksplit, M, d,
                       (const uint16_t*)g, eps, Y, MBn, rows);
  else
    hipLaunchKernelGGL((resid_norm_kernel<uint16_t, true, 2>), dim3(M), dim3(1024), 0, s, X, P, ksplit, M, d,
                       (const uint16_t*)g, eps, Y, MBn, rows);
}

void launch_swiglu(bool bf16, const float* P, int ksplit, int M, int F, void* H, int MBn, hipStream_t s) {
  const dim3 grid(M, (F + 2047) / 2048);
  if (bf16)
    hipLaunchKernelGGL((swiglu_kernel<true, 2>), grid, dim3(256), 0, s, P, ksplit, M, F, H, MBn);
  else
    hipLaunchKernelGGL((swiglu_kernel<false, 1>), grid, dim3(256), 0, s, P, ksplit, M, F, H, MBn);
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

}  // namespace via
