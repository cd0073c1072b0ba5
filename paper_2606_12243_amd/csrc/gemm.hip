// Tall-skinny GEMMs of the verification forward with fused epilogues.
//
// Y[M, cols] = X[M, K] * W[cols, K]^T, M = fed rows (a few to a few hundred),
// W streamed once from HBM.  One work-group = 4 waves = one 64-column tile
// (two 32-column blocks) by up to 32*MB rows; the waves interleave 64-wide
// K steps and their partial tiles are summed in LDS in wave order; when
// `ksplit` > 1 the groups of a tile write partial tiles to the workspace and
// the last group to arrive (integer counter) sums them in split order.  All
// reductions have a fixed order, so results are bitwise reproducible.
//
// bf16 path: v_mfma_f32_32x32x16_bf16.  Lane l holds row/column l%32 and the
// K sub-range (l/32)*32 .. +31 of each 64-wide step: four 8-element slices,
// one per MFMA (A and B use the same K permutation, so the contraction is
// unchanged).  fp32 path: plain FMA on the vector ALUs.
#include "kernels.h"

namespace via {

namespace {

constexpr int kTileN = 64;
constexpr int kThreads = 256;
constexpr int kLdsStride = 65;

// Column blocks of a tile in W-row space.
__device__ __forceinline__ void tile_cols(int epi, const GemmArgs& a, int t, int& c0, int& c1) {
  if (epi == EPI_QKV) {
    // 32-wide blocks paired for rotate-half RoPE: dims i and i + hd/2 of one head
    int half = a.hd >> 1, per_head = half >> 5;
    int h = t / per_head, j = t - h * per_head;
    c0 = h * a.hd + j * 32;
    c1 = c0 + half;
  } else if (epi == EPI_SWIGLU) {
    c0 = t * 32;          // gate rows
    c1 = a.F + t * 32;    // matching up rows
  } else {
    c0 = t * kTileN;
    c1 = c0 + 32;
  }
}

__device__ __forceinline__ int valid_cols(int epi, const GemmArgs& a) {
  // rows of W that exist for the plain mapping; QKV/SWIGLU tiles are always full
  return (epi == EPI_RESID || epi == EPI_STATS) ? a.N : 0x7fffffff;
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// bf16 MFMA tile: lds[32*MB][64] = X[m0.., K-range] * W[cols, K-range]^T
template <int MB>
__device__ void tile_bf16(int epi, const GemmArgs& a, int tile, int split, int m0, float (*lds)[kLdsStride]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 31, h = lane >> 5;
  int c0, c1;
  tile_cols(epi, a, tile, c0, c1);
  const int ncol = valid_cols(epi, a);
  const int ksteps = a.K >> 6;
  const int per = (ksteps + a.ksplit - 1) / a.ksplit;
  const int s_beg = split * per;
  const int s_end = min(ksteps, s_beg + per);
  const uint16_t* W = (const uint16_t*)a.W;
  const uint16_t* X = (const uint16_t*)a.X;
  const bool v0 = (c0 + n) < ncol, v1 = (c1 + n) < ncol;
  const uint4* w0 = (const uint4*)(W + (size_t)(v0 ? c0 + n : 0) * a.K + h * 32);
  const uint4* w1 = (const uint4*)(W + (size_t)(v1 ? c1 + n : 0) * a.K + h * 32);
  const uint4* xr[MB];
  bool xv[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    int m = m0 + mb * 32 + n;
    xv[mb] = m < a.M;
    xr[mb] = (const uint4*)(X + (size_t)(xv[mb] ? m : 0) * a.ldx + h * 32);
  }
  f32x16 acc[MB][2];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.f;

  const uint4 z = make_uint4(0, 0, 0, 0);
  uint4 bw0[4], bw1[4], bx[MB][4];
  auto load = [&](int s) {
    const int o = s * 8;  // 64 bf16 = 8 uint4 per step; this lane's 32 start at h*32
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      bw0[i] = v0 ? w0[o + i] : z;
      bw1[i] = v1 ? w1[o + i] : z;
    }
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int i = 0; i < 4; ++i) bx[mb][i] = xv[mb] ? xr[mb][o + i] : z;
  };
  int s = s_beg + wave;
  if (s < s_end) load(s);
  while (s < s_end) {
    uint4 cw0[4], cw1[4], cx[MB][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      cw0[i] = bw0[i];
      cw1[i] = bw1[i];
    }
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int i = 0; i < 4; ++i) cx[mb][i] = bx[mb][i];
    const int sn = s + 4;
    if (sn < s_end) load(sn);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        acc[mb][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(cx[mb][i]), as_bf16x8(cw0[i]), acc[mb][0], 0, 0, 0);
        acc[mb][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(cx[mb][i]), as_bf16x8(cw1[i]), acc[mb][1], 0, 0, 0);
      }
    }
    s = sn;
  }
  // C layout: lane l, register r -> row (r/4)*8 + (l/32)*4 + r%4, column l%32
  for (int w = 0; w < 4; ++w) {
    if (wave == w) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            int row = mb * 32 + (r >> 2) * 8 + h * 4 + (r & 3);
            int col = nb * 32 + n;
            if (w == 0)
              lds[row][col] = acc[mb][nb][r];
            else
              lds[row][col] += acc[mb][nb][r];
          }
    }
    __syncthreads();
  }
}

// fp32 tile on the vector ALUs: thread (row t/8, columns (t%8)*8 .. +7).
template <int MB>
__device__ void tile_f32(int epi, const GemmArgs& a, int tile, int split, int m0, float (*lds)[kLdsStride]) {
  const int t = threadIdx.x;
  const int r = t >> 3, cg = (t & 7) * 8;
  int c0, c1;
  tile_cols(epi, a, tile, c0, c1);
  const int ncol = valid_cols(epi, a);
  const int ksteps = a.K >> 6;
  const int per = (ksteps + a.ksplit - 1) / a.ksplit;
  const int k_beg = split * per * 64;
  const int k_end = min(a.K, k_beg + per * 64);
  const float* W = (const float*)a.W;
  const float* X = (const float*)a.X;
  for (int mb = 0; mb < MB; ++mb) {
    int m = m0 + mb * 32 + r;
    float acc[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] = 0.f;
    if (m < a.M) {
      const float* x = X + (size_t)m * a.ldx;
      for (int k = k_beg; k < k_end; ++k) {
        float xv = x[k];
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          int cc = cg + c;
          int col = cc < 32 ? c0 + cc : c1 + cc - 32;
          if (col < ncol) acc[c] = fmaf(xv, W[(size_t)col * a.K + k], acc[c]);
        }
      }
    }
#pragma unroll
    for (int c = 0; c < 8; ++c) lds[mb * 32 + r][cg + c] = acc[c];
  }
  __syncthreads();
}

__device__ __forceinline__ float load_acquire(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Split-K: returns false for groups that are not the last of their tile.
template <int MB>
__device__ bool reduce_splits(const GemmArgs& a, int tile, int split, int mg, int m0, float (*lds)[kLdsStride]) {
  if (a.ksplit == 1) return true;
  __shared__ int s_last;
  const size_t ld = (size_t)a.ntiles * kTileN;
  float* P = a.part + (size_t)split * a.M * ld;
  for (int idx = threadIdx.x; idx < 32 * MB * kTileN; idx += kThreads) {
    int r = idx >> 6, c = idx & 63, m = m0 + r;
    if (m < a.M) P[(size_t)m * ld + tile * kTileN + c] = lds[r][c];
  }
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    int ci = mg * a.ntiles + tile;
    int prev = atomicAdd(&a.counters[ci], 1);
    s_last = (prev == a.ksplit - 1);
    if (s_last) a.counters[ci] = 0;
  }
  __syncthreads();
  if (!s_last) return false;
  __threadfence();
  for (int idx = threadIdx.x; idx < 32 * MB * kTileN; idx += kThreads) {
    int r = idx >> 6, c = idx & 63, m = m0 + r;
    float sum = 0.f;
    if (m < a.M)
      for (int sp = 0; sp < a.ksplit; ++sp)
        sum += load_acquire(a.part + ((size_t)sp * a.M + m) * ld + tile * kTileN + c);
    lds[r][c] = sum;
  }
  __syncthreads();
  return true;
}

template <typename T, int MB>
__device__ void epi_qkv(const GemmArgs& a, int tile, int m0, float (*lds)[kLdsStride]) {
  const int half = a.hd >> 1, per_head = half >> 5;
  const int hh = tile / per_head, j = tile - hh * per_head;
  T* Q = (T*)a.q_out;
  T* pool = (T*)a.pool;
  for (int idx = threadIdx.x; idx < 32 * MB * 32; idx += kThreads) {
    int r = idx >> 5, c = idx & 31, m = m0 + r;
    if (m >= a.M) continue;
    int i = j * 32 + c;
    float x1 = lds[r][c], x2 = lds[r][32 + c];
    const RowInfo ri = a.rows[m];
    float y1 = x1, y2 = x2;
    if (hh < a.H + a.KVH) {
      // rotate-half RoPE at the row's position; angle and rotation in fp64
      double inv = pow((double)a.theta, -2.0 * (double)i / (double)a.hd);
      double ang = (double)ri.pos * inv;
      double cs = cos(ang), sn = sin(ang);
      y1 = (float)((double)x1 * cs - (double)x2 * sn);
      y2 = (float)((double)x2 * cs + (double)x1 * sn);
    }
    if (hh < a.H) {
      size_t o = ((size_t)m * a.H + hh) * a.hd;
      Q[o + i] = from_f<T>(y1);
      Q[o + i + half] = from_f<T>(y2);
    } else {
      const SeqInfo si = a.seqs[ri.seq];
      int blk = a.btab[si.bt + ri.slot / kBlock], t = ri.slot % kBlock;
      if (hh < a.H + a.KVH) {
        int g = hh - a.H;
        pool[k_off(a.layer_slot, blk, a.pool_blocks, a.KVH, a.hd, g, t, i)] = from_f<T>(y1);
        pool[k_off(a.layer_slot, blk, a.pool_blocks, a.KVH, a.hd, g, t, i + half)] = from_f<T>(y2);
      } else {
        int g = hh - a.H - a.KVH;
        pool[v_off(a.layer_slot, blk, a.pool_blocks, a.KVH, a.hd, g, t, i)] = from_f<T>(y1);
        pool[v_off(a.layer_slot, blk, a.pool_blocks, a.KVH, a.hd, g, t, i + half)] = from_f<T>(y2);
      }
    }
  }
}

template <int MB>
__device__ void epi_resid(const GemmArgs& a, int tile, int m0, float (*lds)[kLdsStride]) {
  for (int idx = threadIdx.x; idx < 32 * MB * kTileN; idx += kThreads) {
    int r = idx >> 6, c = idx & 63, m = m0 + r, col = tile * kTileN + c;
    if (m < a.M && col < a.N) a.resid[(size_t)m * a.N + col] += lds[r][c];
  }
}

template <typename T, int MB>
__device__ void epi_swiglu(const GemmArgs& a, int tile, int m0, float (*lds)[kLdsStride]) {
  T* Hb = (T*)a.h_out;
  for (int idx = threadIdx.x; idx < 32 * MB * 32; idx += kThreads) {
    int r = idx >> 5, c = idx & 31, m = m0 + r;
    if (m >= a.M) continue;
    float g = lds[r][c], u = lds[r][32 + c];
    float hv = g / (1.0f + expf(-g)) * u;
    Hb[(size_t)m * a.F + tile * 32 + c] = from_f<T>(hv);
  }
}

// (max, argmax, second) merge with lowest-index tie break
__device__ __forceinline__ void merge3(float& mx, int& am, float& sc, float mx2, int am2, float sc2) {
  if (mx2 > mx || (mx2 == mx && am2 < am)) {
    sc = fmaxf(sc2, mx);
    mx = mx2;
    am = am2;
  } else {
    sc = fmaxf(sc, mx2);
  }
}

template <int MB>
__device__ void epi_stats(const GemmArgs& a, int tile, int m0, float (*lds)[kLdsStride]) {
  const int grp = threadIdx.x >> 3, gl = threadIdx.x & 7;  // 32 groups of 8 threads
  const int c0 = tile * kTileN;
  for (int r = grp; r < 32 * MB; r += 32) {
    int m = m0 + r;
    if (m >= a.M) continue;  // uniform within the group
    float mx = -INFINITY, sc = -INFINITY;
    int am = 0x7fffffff;
    for (int c = gl * 8; c < gl * 8 + 8; ++c) {
      int col = c0 + c;
      if (col < a.N) merge3(mx, am, sc, lds[r][c], col, -INFINITY);
    }
    for (int o = 1; o < 8; o <<= 1) {
      float mx2 = __shfl_xor(mx, o, 64), sc2 = __shfl_xor(sc, o, 64);
      int am2 = __shfl_xor(am, o, 64);
      merge3(mx, am, sc, mx2, am2, sc2);
    }
    float se = 0.f;
    for (int c = gl * 8; c < gl * 8 + 8; ++c) {
      int col = c0 + c;
      if (col < a.N) se += expf((lds[r][c] - mx) * a.inv_T);
    }
    for (int o = 1; o < 8; o <<= 1) se += __shfl_xor(se, o, 64);
    const LmRow lr = a.lm[m];
    if (gl == 0) {
      float* p = a.lm_part + ((size_t)tile * a.M + m) * 4;
      p[0] = mx;
      p[1] = sc;
      p[2] = se;
      p[3] = __int_as_float(am);
      for (int q = 0; q < lr.n_drafts; ++q) {
        int tk = lr.draft_tok[q];
        if (tk >= c0 && tk < c0 + kTileN) a.draft_logit[lr.draft_idx[q]] = lds[r][tk - c0];
      }
    }
    if (a.logits) {
      for (int c = gl * 8; c < gl * 8 + 8; ++c) {
        int col = c0 + c;
        if (col < a.N) a.logits[(size_t)lr.out * a.N + col] = lds[r][c];
      }
    }
  }
}

template <typename T, int MB, int EPI>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmArgs a) {
  __shared__ float lds[32 * MB][kLdsStride];
  const int tile = blockIdx.x % a.ntiles;
  const int split = blockIdx.x / a.ntiles;
  const int mg = blockIdx.y;
  const int m0 = mg * 32 * MB;
  if constexpr (sizeof(T) == 2)
    tile_bf16<MB>(EPI, a, tile, split, m0, lds);
  else
    tile_f32<MB>(EPI, a, tile, split, m0, lds);
  if (!reduce_splits<MB>(a, tile, split, mg, m0, lds)) return;
  if constexpr (EPI == EPI_QKV) epi_qkv<T, MB>(a, tile, m0, lds);
  if constexpr (EPI == EPI_RESID) epi_resid<MB>(a, tile, m0, lds);
  if constexpr (EPI == EPI_SWIGLU) epi_swiglu<T, MB>(a, tile, m0, lds);
  if constexpr (EPI == EPI_STATS) epi_stats<MB>(a, tile, m0, lds);
}

template <typename T, int MB>
void launch_mb(int epi, const GemmArgs& a, dim3 grid, hipStream_t s) {
  switch (epi) {
    case EPI_QKV: hipLaunchKernelGGL((gemm_kernel<T, MB, EPI_QKV>), grid, dim3(kThreads), 0, s, a); break;
    case EPI_RESID: hipLaunchKernelGGL((gemm_kernel<T, MB, EPI_RESID>), grid, dim3(kThreads), 0, s, a); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((gemm_kernel<T, MB, EPI_SWIGLU>), grid, dim3(kThreads), 0, s, a); break;
    default: hipLaunchKernelGGL((gemm_kernel<T, MB, EPI_STATS>), grid, dim3(kThreads), 0, s, a); break;
  }
}

template <typename T>
void launch_t(int epi, const GemmArgs& a, hipStream_t s) {
  // rows per group: up to 128; groups cover M
  int mb = (a.M + 31) / 32;
  if (mb > 4) mb = 4;
  dim3 grid(a.ntiles * a.ksplit, (a.M + 32 * mb - 1) / (32 * mb));
  switch (mb) {
    case 1: launch_mb<T, 1>(epi, a, grid, s); break;
    case 2: launch_mb<T, 2>(epi, a, grid, s); break;
    case 3: launch_mb<T, 3>(epi, a, grid, s); break;
    default: launch_mb<T, 4>(epi, a, grid, s); break;
  }
}

// ---------------------------------------------------------------- head stats
__global__ __launch_bounds__(256) void lm_finalize_kernel(const LmRow* lm, const float* part, int M, int ntiles,
                                                          float inv_T, int32_t* row_argmax, float* row_max,
                                                          float* row_sumexp, float* row_gap) {
  __shared__ float s_mx[256], s_sc[256], s_se[256];
  __shared__ int s_am[256];
  const int m = blockIdx.x, t = threadIdx.x;
  float mx = -INFINITY, sc = -INFINITY;
  int am = 0x7fffffff;
  for (int tl = t; tl < ntiles; tl += 256) {
    const float* p = part + ((size_t)tl * M + m) * 4;
    merge3(mx, am, sc, p[0], __float_as_int(p[3]), p[1]);
  }
  s_mx[t] = mx;
  s_sc[t] = sc;
  s_am[t] = am;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (t < o) {
      float a_mx = s_mx[t], a_sc = s_sc[t];
      int a_am = s_am[t];
      merge3(a_mx, a_am, a_sc, s_mx[t + o], s_am[t + o], s_sc[t + o]);
      s_mx[t] = a_mx;
      s_sc[t] = a_sc;
      s_am[t] = a_am;
    }
    __syncthreads();
  }
  const float gmx = s_mx[0];
  float se = 0.f;
  for (int tl = t; tl < ntiles; tl += 256) {
    const float* p = part + ((size_t)tl * M + m) * 4;
    se += p[2] * expf((p[0] - gmx) * inv_T);
  }
  s_se[t] = se;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (t < o) s_se[t] += s_se[t + o];
    __syncthreads();
  }
  if (t == 0) {
    const int out = lm[m].out;
    row_max[out] = gmx;
    row_argmax[out] = s_am[0];
    row_sumexp[out] = s_se[0];
    if (row_gap) row_gap[out] = gmx - s_sc[0];
  }
}

}  // namespace

void launch_gemm(int epi, bool bf16, const GemmArgs& a, hipStream_t s) {
  if (bf16)
    launch_t<uint16_t>(epi, a, s);
  else
    launch_t<float>(epi, a, s);
}

void launch_lm_finalize(const LmRow* lm, const float* lm_part, int n_lm, int ntiles, float inv_T, int32_t* row_argmax,
                        float* row_max, float* row_sumexp, float* row_gap, hipStream_t s) {
  hipLaunchKernelGGL(lm_finalize_kernel, dim3(n_lm), dim3(256), 0, s, lm, lm_part, n_lm, ntiles, inv_T, row_argmax,
                     row_max, row_sumexp, row_gap);
}

}  // namespace via
