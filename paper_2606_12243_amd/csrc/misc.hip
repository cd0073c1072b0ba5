// Small kernels of the verification step: embedding gather, RMSNorm, the
// tier decision with its gate walk, and tree-path K/V compaction.
#include "kernels.h"

namespace via {

namespace {

template <typename T>
__global__ __launch_bounds__(256) void embed_kernel(const T* E, const RowInfo* rows, int d, float* X) {
  const int m = blockIdx.x;
  const T* e = E + (size_t)rows[m].tok * d;
  for (int i = threadIdx.x; i < d; i += 256) X[(size_t)m * d + i] = to_f<T>(e[i]);
}

// y = x / sqrt(mean(x^2) + eps) * g; fixed-order block reduction.
template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float* X, const T* g, int d, float eps, T* Y,
                                                      const LmRow* gather) {
  __shared__ float red[256];
  const int m = blockIdx.x;
  const int src = gather ? gather[m].row : m;
  const float* x = X + (size_t)src * d;
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) ss += x[i] * x[i];
  red[threadIdx.x] = ss;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  const float inv = 1.0f / sqrtf(red[0] / (float)d + eps);
  for (int i = threadIdx.x; i < d; i += 256) Y[(size_t)m * d + i] = from_f<T>(x[i] * inv * to_f<T>(g[i]));
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
    if (!(fabsf(fm) <= 3.0e38f)) {  // non-finite logits of q
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

void launch_rmsnorm(bool bf16, const float* X, const void* g, int M, int d, float eps, void* Y, const LmRow* gather,
                    hipStream_t s) {
  if (bf16)
    hipLaunchKernelGGL(rmsnorm_kernel<uint16_t>, dim3(M), dim3(256), 0, s, X, (const uint16_t*)g, d, eps,
                       (uint16_t*)Y, gather);
  else
    hipLaunchKernelGGL(rmsnorm_kernel<float>, dim3(M), dim3(256), 0, s, X, (const float*)g, d, eps, (float*)Y,
                       gather);
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
