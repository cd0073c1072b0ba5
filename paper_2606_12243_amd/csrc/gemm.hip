// Tall-skinny GEMMs of the verification forward.
//
// P[split][M][N] = X[M, K-slice] * W[N, K-slice]^T with M = fed rows (tens),
// W (bf16, packed) streamed once from HBM, X (activation fragments) from L2.
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
// K sub-block (l/16)*8 .. +7 of each 32-wide step.  Weights are pre-packed
// (via_pack_weight) and activations are written by their producer kernels
// as fragments (afrag_group), so every load instruction of a wave reads one
// contiguous 1 KB block and the inner loop is loads + MFMA only.  fp32
// activations enter the matrix cores as NT bf16 terms (x = hi + [mid +] lo),
// NT = 3 keeping ~24 significant bits and NT = 2 ~16.  Output register r of lane l is row (l/16)*4 + r,
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

// lds[16*MB][64] = X[m0 .., K slice] * W[c0 .. c0+64, K slice]^T, X given as
// NT bf16-term fragments and W packed: each load is one contiguous 1 KB block.
template <int MB, int NT>
__device__ void tile_bf16(const GemmArgs& a, int c0, int m0, int k_beg, int k_end, float* lds) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 15, g = lane >> 4;
  const int S = a.K >> 5;
  const int st_beg = k_beg >> 5, st_all = (k_end - k_beg) >> 5;
  const int per = (st_all + kWaves - 1) / kWaves;
  const int s0 = st_beg + wave * per, s1 = min(st_beg + st_all, s0 + per);
  const uint4* wt = (const uint4*)a.W + (size_t)(c0 >> 6) * S * (4 * 64) + lane;
  const uint4* xt = (const uint4*)a.X + (size_t)(m0 >> 4) * 64 + lane;
  const size_t x_step = (size_t)a.MBn * 64, x_term = (size_t)S * x_step;

  f32x4 acc[MB][kNB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  uint4 wb[2][kBatch][kNB], xb[2][kBatch][NT][MB];
  // steps past the slice re-read its last step and are skipped by compute
  auto issue = [&](int buf, int s) {
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int st = min(s + u, s1 - 1);
#pragma unroll
      for (int nb = 0; nb < kNB; ++nb) wb[buf][u][nb] = wt[(st * 4 + nb) * 64];
#pragma unroll
      for (int q = 0; q < NT; ++q)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) xb[buf][u][q][mb] = xt[q * x_term + st * x_step + mb * 64];
    }
  };
  auto compute = [&](int buf, int s) {
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      if (s + u >= s1) break;  // wave-uniform
#pragma unroll
      for (int q = 0; q < NT; ++q)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int nb = 0; nb < kNB; ++nb)
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(xb[buf][u][q][mb]),
                                                                as_bf16x8(wb[buf][u][nb]), acc[mb][nb], 0, 0, 0);
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

// fp32 tile on the vector ALUs (X fragments with one fp32 term).
template <int MB>
__device__ void tile_f32(const GemmArgs& a, int c0, int m0, int k_beg, int k_end, float* lds) {
  const float* W = (const float*)a.W;
  const float* X = (const float*)a.X;
  const size_t steps = a.K >> 5;
  for (int e = threadIdx.x; e < 16 * MB * kTileN; e += kThreads) {
    const int r = e / kTileN, c = e - r * kTileN;
    const int m = m0 + r, col = c0 + c;
    float acc = 0.f;
    if (m < a.M && col < a.N) {
      // packed weight element (col, k): group ((tile*steps + k/32)*4 + nb)*64 + ((k%32)/8)*16 + col%16
      const size_t base = (size_t)(col >> 6) * steps * 4 * 64 + ((col & 63) >> 4) * 64 + (col & 15);
      for (int k = k_beg; k < k_end; ++k) {
        const float xv = X[afrag_group(0, m, k & ~7, (int)steps, a.MBn) * 8 + (k & 7)];
        acc = fmaf(xv, W[(base + (size_t)(k >> 5) * 256 + ((k & 31) >> 3) * 16) * 8 + (k & 7)], acc);
      }
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
  const int mb = gemm_rows_per_group(a.M) / 16;
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

// Row-major [rows, cols] -> packed tiles; one thread per 8-element group.
template <typename T>
__global__ __launch_bounds__(256) void pack_kernel(const T* src, T* dst, int rows, int cols, size_t groups) {
  const size_t gidx = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (gidx >= groups) return;
  const int steps = cols >> 5;
  const int lane = (int)(gidx & 63);
  size_t q = gidx >> 6;
  const int nb = (int)(q & 3);
  q >>= 2;
  const int st = (int)(q % steps);
  const size_t tile = q / steps;
  const size_t r = tile * 64 + nb * 16 + (lane & 15);
  const size_t c = (size_t)st * 32 + (lane >> 4) * 8;
#pragma unroll
  for (int e = 0; e < 8; ++e) dst[gidx * 8 + e] = r < (size_t)rows ? src[r * cols + c + e] : T(0);
}

}  // namespace

void launch_pack(bool bf16, const void* src, void* dst, int rows, int cols, hipStream_t s) {
  const size_t groups = (size_t)((rows + 63) / 64) * 64 * (cols / 8);
  const dim3 grid((unsigned)((groups + 255) / 256));
  if (bf16)
    hipLaunchKernelGGL(pack_kernel<uint16_t>, grid, dim3(256), 0, s, (const uint16_t*)src, (uint16_t*)dst, rows, cols,
                       groups);
  else
    hipLaunchKernelGGL(pack_kernel<float>, grid, dim3(256), 0, s, (const float*)src, (float*)dst, rows, cols, groups);
}

int gemm_tiles(int N) { return (N + kTileN - 1) / kTileN; }

int gemm_rows_per_group(int M) { return M > 16 ? 32 : 16; }

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
