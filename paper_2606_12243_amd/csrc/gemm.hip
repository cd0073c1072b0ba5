// Tall-skinny GEMMs of the verification forward.
//
// P[split][M][N] = X[M, K-slice] * W[N, K-slice]^T with M = fed rows (tens),
// W (bf16) streamed once from HBM, X (fp32 activations) read from L2.
// A work-group (8 waves) owns a 64-column tile and one K slice; its waves
// split the slice further, keep two batches of loads in flight and sum their
// partial tiles in LDS in wave order.  The K slices of a tile ("splits") are
// written as separate fp32 partial tiles and summed, in split order, by the
// consumer kernel after the kernel boundary: handing partial sums between
// work-groups inside one kernel would need a device-scope release, which
// costs an L2 writeback on this GPU.  Every reduction has a fixed order, so
// results are bitwise reproducible and independent of M.
//
// bf16 path: v_mfma_f32_16x16x32_bf16.  Lane l holds row/column l%16 and
// K sub-block (l/16)*8 .. +7 of each 32-wide step (a load instruction reads
// 64 contiguous bytes of each of 16 weight rows).  The fp32 activations enter
// the matrix cores as NT bf16 terms: x = hi + (mid) + lo, hi and mid
// truncated, the last rounded to nearest, so NT = 3 keeps ~24 significant
// bits and NT = 2 ~16.  Output register r of lane l is row (l/16)*4 + r,
// column l%16.  The head GEMM (split 1) reduces its tile to per-row
// (max, second, sum-exp, argmax) partials and draft-token logits in place.
// fp32 path: plain FMA on the vector ALUs (small models only).
#include "kernels.h"

namespace via {

namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;
constexpr int kTileN = 64;   // columns per work-group: 4 blocks of 16
constexpr int kNB = 4;
constexpr int kBatch = 2;    // 32-wide K steps per load batch

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ uint4 zero_if(uint4 v, bool ok) {
  v.x = ok ? v.x : 0u;
  v.y = ok ? v.y : 0u;
  v.z = ok ? v.z : 0u;
  v.w = ok ? v.w : 0u;
  return v;
}

__device__ __forceinline__ uint32_t pack2(uint32_t lo16, uint32_t hi16) { return (lo16 & 0xFFFFu) | (hi16 << 16); }

// Split 8 fp32 values into NT bf16x8 terms (hi, [mid,] lo).
template <int NT>
__device__ __forceinline__ void split_terms(const float* x, uint4* out) {
  uint32_t t[NT][8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    float r = x[e];
#pragma unroll
    for (int q = 0; q < NT; ++q) {
      uint32_t u = __float_as_uint(r);
      uint32_t b = (q == NT - 1) ? (uint32_t)f2bf(r) : (u >> 16);  // last term rounded, others truncated
      t[q][e] = b;
      r = r - __uint_as_float(b << 16);
    }
  }
#pragma unroll
  for (int q = 0; q < NT; ++q)
    out[q] = make_uint4(pack2(t[q][0], t[q][1]), pack2(t[q][2], t[q][3]), pack2(t[q][4], t[q][5]),
                        pack2(t[q][6], t[q][7]));
}

// lds[16*MB][64] = X[m0 .., K slice] * W[c0 .. c0+64, K slice]^T
template <int MB, int NT>
__device__ void tile_bf16(const GemmArgs& a, int c0, int m0, int k_beg, int k_end, float* lds) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 15, g = lane >> 4;
  const uint16_t* W = (const uint16_t*)a.W;
  const float* X = (const float*)a.X;
  const int st_beg = k_beg >> 5, st_all = (k_end - k_beg) >> 5;
  const int per = (st_all + kWaves - 1) / kWaves;
  const int s0 = st_beg + wave * per, s1 = min(st_beg + st_all, s0 + per);

  const uint4* wp[kNB];
  bool wv[kNB];
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    const int col = c0 + nb * 16 + n;
    wv[nb] = col < a.N;
    wp[nb] = (const uint4*)(W + (size_t)(wv[nb] ? col : 0) * a.K + g * 8);
  }
  const uint4* xp[MB];
  bool xv[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int m = m0 + mb * 16 + n;
    xv[mb] = m < a.M;
    xp[mb] = (const uint4*)(X + (size_t)(xv[mb] ? m : 0) * a.ldx + g * 8);
  }
  f32x4 acc[MB][kNB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  // two batches in flight; loads are unconditional (rows past the end read
  // row 0, steps past the slice re-read its last step) and masked afterwards
  uint4 wb[2][kBatch][kNB], xb[2][kBatch][MB][2];
  auto issue = [&](int buf, int s) {
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int st = min(s + u, s1 - 1);
#pragma unroll
      for (int nb = 0; nb < kNB; ++nb) wb[buf][u][nb] = wp[nb][st * 4];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        xb[buf][u][mb][0] = xp[mb][st * 8];
        xb[buf][u][mb][1] = xp[mb][st * 8 + 1];
      }
    }
  };
  auto compute = [&](int buf, int s) {
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const bool live = (s + u) < s1;
      bf16x8 bw[kNB];
#pragma unroll
      for (int nb = 0; nb < kNB; ++nb) bw[nb] = as_bf16x8(zero_if(wb[buf][u][nb], wv[nb] && live));
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        float xf[8];
        __builtin_memcpy(xf, &xb[buf][u][mb][0], 32);
        uint4 terms[NT];
        split_terms<NT>(xf, terms);
#pragma unroll
        for (int q = 0; q < NT; ++q) {
          const bf16x8 av = as_bf16x8(zero_if(terms[q], xv[mb]));
#pragma unroll
          for (int nb = 0; nb < kNB; ++nb)
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bw[nb], acc[mb][nb], 0, 0, 0);
        }
      }
    }
  };
  // buffer indices are compile-time constants (a runtime index would put
  // the buffers in scratch memory)
  if (s0 < s1) {
    issue(0, s0);
    for (int s = s0; s < s1; s += 2 * kBatch) {
      if (s + kBatch < s1) issue(1, s + kBatch);
      compute(0, s);
      if (s + kBatch >= s1) break;
      if (s + 2 * kBatch < s1) issue(0, s + 2 * kBatch);
      compute(1, s + kBatch);
    }
  }
  for (int w = 0; w < kWaves; ++w) {
    if (wave == w) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            float* p = lds + (mb * 16 + g * 4 + r) * kTileN + nb * 16 + n;
            *p = (w == 0) ? acc[mb][nb][r] : *p + acc[mb][nb][r];
          }
    }
    __syncthreads();
  }
}

// fp32 tile on the vector ALUs.
template <int MB>
__device__ void tile_f32(const GemmArgs& a, int c0, int m0, int k_beg, int k_end, float* lds) {
  const float* W = (const float*)a.W;
  const float* X = (const float*)a.X;
  for (int e = threadIdx.x; e < 16 * MB * kTileN; e += kThreads) {
    const int r = e / kTileN, c = e - r * kTileN;
    const int m = m0 + r, col = c0 + c;
    float acc = 0.f;
    if (m < a.M && col < a.N) {
      const float* x = X + (size_t)m * a.ldx;
      const float* w = W + (size_t)col * a.K;
      for (int k = k_beg; k < k_end; ++k) acc = fmaf(x[k], w[k], acc);
    }
    lds[e] = acc;
  }
  __syncthreads();
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

// Head tile epilogue, per head row: partial (max, second, sum-exp at the tile
// max, argmax), the logit of each draft token inside the tile, and the
// optional fp32 logits dump.  8 threads per row, 8 columns each.
template <int MB>
__device__ void epi_stats(const GemmArgs& a, int tile, int m0, const float* lds) {
  const int grp = threadIdx.x >> 3, gl = threadIdx.x & 7;  // 64 groups of 8 threads
  const int c0 = tile * kTileN;
  for (int r = grp; r < 16 * MB; r += kThreads / 8) {
    const int m = m0 + r;
    if (m >= a.M) continue;  // uniform within the group
    float mx = -INFINITY, sc = -INFINITY;
    int am = 0x7fffffff;
    for (int c = gl * 8; c < gl * 8 + 8; ++c)
      if (c0 + c < a.N) merge3(mx, am, sc, lds[r * kTileN + c], c0 + c, -INFINITY);
    for (int o = 1; o < 8; o <<= 1) {
      const float mx2 = __shfl_xor(mx, o, 64), sc2 = __shfl_xor(sc, o, 64);
      const int am2 = __shfl_xor(am, o, 64);
      merge3(mx, am, sc, mx2, am2, sc2);
    }
    float se = 0.f;
    for (int c = gl * 8; c < gl * 8 + 8; ++c)
      if (c0 + c < a.N) se += expf((lds[r * kTileN + c] - mx) * a.inv_T);
    for (int o = 1; o < 8; o <<= 1) se += __shfl_xor(se, o, 64);
    const int out = a.lm[m].out;
    if (gl == 0) {
      float* p = a.lm_part + ((size_t)tile * a.M + m) * 4;
      p[0] = mx;
      p[1] = sc;
      p[2] = se;
      p[3] = __int_as_float(am);
    }
    if (gl < a.lm[m].n_drafts) {
      const int tk = a.lm[m].draft_tok[gl];
      if (tk >= c0 && tk < c0 + kTileN) a.draft_logit[a.lm[m].draft_idx[gl]] = lds[r * kTileN + tk - c0];
    }
    if (a.logits) {
      for (int c = gl * 8; c < gl * 8 + 8; ++c)
        if (c0 + c < a.N) a.logits[(size_t)out * a.N + c0 + c] = lds[r * kTileN + c];
    }
  }
}

template <typename T, int MB, int NT, bool STATS>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmArgs a) {
  __shared__ float lds[16 * MB * kTileN];
  // block -> (tile, split, m-group), m-group fastest: neighbours share W rows
  const int mgroups = (a.M + 16 * MB - 1) / (16 * MB);
  int b = blockIdx.x;
  const int mg = b % mgroups;
  b /= mgroups;
  const int split = b % a.ksplit;
  const int tile = b / a.ksplit;
  const int m0 = mg * 16 * MB, c0 = tile * kTileN;
  const int steps = a.K >> 5, per = (steps + a.ksplit - 1) / a.ksplit;
  const int k_beg = min(steps, split * per) * 32, k_end = min(steps, (split + 1) * per) * 32;
  if constexpr (sizeof(T) == 2)
    tile_bf16<MB, NT>(a, c0, m0, k_beg, k_end, lds);
  else
    tile_f32<MB>(a, c0, m0, k_beg, k_end, lds);
  if constexpr (STATS) {
    epi_stats<MB>(a, tile, m0, lds);
  } else {
    float* P = a.part + (size_t)split * a.M * a.N;
    for (int e = threadIdx.x; e < 16 * MB * kTileN; e += kThreads) {
      const int r = e / kTileN, c = e - r * kTileN, m = m0 + r, col = c0 + c;
      if (m < a.M && col < a.N) P[(size_t)m * a.N + col] = lds[e];
    }
  }
}

template <typename T, int NT, bool STATS>
void launch_e(const GemmArgs& a, hipStream_t s) {
  // up to 32 rows per work-group (register budget); more rows take more
  // m-groups, whose neighbouring work-groups re-read the same W rows
  const int mb = a.M > 16 ? 2 : 1;
  const int mgroups = (a.M + 16 * mb - 1) / (16 * mb);
  dim3 grid(gemm_tiles(a.N) * a.ksplit * mgroups);
  if (mb == 1)
    hipLaunchKernelGGL((gemm_kernel<T, 1, NT, STATS>), grid, dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL((gemm_kernel<T, 2, NT, STATS>), grid, dim3(kThreads), 0, s, a);
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

int gemm_tiles(int N) { return (N + kTileN - 1) / kTileN; }

void launch_gemm(bool bf16, int terms, bool stats, const GemmArgs& a, hipStream_t s) {
  if (!bf16) {
    if (stats)
      launch_e<float, 1, true>(a, s);
    else
      launch_e<float, 1, false>(a, s);
  } else if (stats) {
    launch_e<uint16_t, 2, true>(a, s);
  } else if (terms >= 3) {
    launch_e<uint16_t, 3, false>(a, s);
  } else {
    launch_e<uint16_t, 2, false>(a, s);
  }
}

void launch_lm_finalize(const LmRow* lm, const float* lm_part, int n_lm, int ntiles, float inv_T, int32_t* row_argmax,
                        float* row_max, float* row_sumexp, float* row_gap, hipStream_t s) {
  hipLaunchKernelGGL(lm_finalize_kernel, dim3(n_lm), dim3(256), 0, s, lm, lm_part, n_lm, ntiles, inv_T, row_argmax,
                     row_max, row_sumexp, row_gap);
}

}  // namespace via
