// Tall-skinny GEMMs of the verification forward.
//
// P[split][M][N] = X[M, K-slice] * W[N, K-slice]^T with M = fed rows (tens),
// W (bf16, packed) streamed once from HBM.  A work-group of 8 waves owns a
// 256-column tile, up to 64 rows and one K slice; each wave owns two
// 16-column blocks and streams their weights over the whole slice, two
// chunks of steps ahead of its multiply.  The activation fragments (X) of a
// chunk are loaded once per work-group into LDS (double-buffered) and read
// there by all eight waves, so X leaves L2 once per work-group and no
// cross-wave reduction is needed.  The K slices of a tile ("splits") are
// written as separate fp32 partial tiles and summed, in split order, by the
// consumer kernel after the kernel boundary: handing partial sums between
// work-groups inside one kernel would need a device-scope release, which
// costs an L2 writeback on this GPU.  Every reduction has a fixed order, so
// results are bitwise reproducible.
//
// bf16 path: v_mfma_f32_16x16x32_bf16.  Lane l holds row/column l%16 and
// K sub-block (l/16)*8 .. +7 of each 32-wide step.  Weights are pre-packed
// (via_pack_weight) and activations are written by their producer kernels
// as fragments (afrag_group), so every global load of a wave reads one
// contiguous 1 KB block and every LDS read is conflict-free.  fp32
// activations enter the matrix cores as NT bf16 terms (x = hi + [mid +] lo),
// NT = 3 keeping ~24 significant bits and NT = 2 ~16 (every projection
// takes 2; the kernels also build for 3).  Output register r of
// lane l is row (l/16)*4 + r, column l%16.  The head GEMM (split 1) reduces
// its tile to per-row (max, second, sum-exp, argmax) partials and
// draft-token logits in place.
// fp32 path: plain FMA on the vector ALUs (small models only).
#include <hip/hip_ext.h>

#include "kernels.h"

namespace via {

namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;
constexpr int kNBW = 2;                // 16-column blocks per wave
constexpr int kTileN = 8 * 16 * kNBW;   // columns per work-group tile (8 waves)

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// Work-group tile: 16*MB rows x (8 * 16 * NBW) columns, one K slice.  Wave
// w owns NBW 16-column blocks and streams their packed W over the whole
// slice in chunks of C steps, two chunks ahead of the one it multiplies;
// the X fragments of a chunk are loaded one chunk ahead and staged once in
// LDS (double-buffered), where all eight waves read them: X leaves L2 once
// per work-group and no cross-wave reduction is needed.  Columns past N are
// computed from a clamped tile and never stored.
template <int MB, int NT, int NBW, int C>
struct TileShape {
  static constexpr int kCols = 8 * 16 * NBW;
  static constexpr int kXChunk = C * NT * MB * 64;   // uint4 per staged chunk
  static constexpr int kXPT = kXChunk / kThreads;     // uint4 staged per thread
};

// `active` (wave-uniform) false: the wave helps stage X but loads no
// weights and multiplies nothing (its accumulators stay zero).
//
// M32 (two 16-column blocks per wave, an even number of row blocks): the
// products run on v_mfma_f32_32x32x16_bf16, twice the rate of the 16x16x32
// form on this GPU.  Its operands are gathered from the same 1 KB
// fragments: lane l of a 32-row (or 32-column) x 16-K operand takes
// row (column) l%32 -- block (l/16)%2 of the pair, row l%16 -- and K group
// 2h + l/32 of the 32-wide step (half h), i.e. fragment lane
// (2h + l/32)*16 + l%16.  acc is then f32x16[MB/2]: 32-row tile i holds
// rows 32i + (r/4)*8 + (l/32)*4 + r%4, column l%32 of the wave's 32.
template <int MB, int NT, int NBW, int C, bool M32 = false, typename Acc>
__device__ void tile_bf16(const GemmArgs& a, int c0, int m0, int st_beg, int st_end, uint4* sx, Acc& acc,
                          bool active = true) {
  using TS = TileShape<MB, NT, NBW, C>;
  static_assert(TS::kXChunk % kThreads == 0, "chunk must split evenly over the threads");
  static_assert(!M32 || (NBW == 2 && MB % 2 == 0), "32x32 tiles need two column blocks and row-block pairs");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int S = a.K >> 5;
  const int t64 = (a.N + 63) >> 6;
  const int sel = (lane >> 4) & 1;                        // M32: block of the pair
  const int fl = M32 ? ((lane >> 5) * 16 + (lane & 15)) : lane;  // M32: fragment lane of half 0
  const uint4* wt[NBW];
#pragma unroll
  for (int j = 0; j < NBW; ++j) {
    // M32: wt[j] is K half j of the lane's block; otherwise block j, own lane
    const int blk = (c0 >> 4) + wave * NBW + (M32 ? sel : j);  // global 16-column block
    const int pt = min(blk >> 2, t64 - 1);
    wt[j] = (const uint4*)a.W + (size_t)pt * S * 256 + (blk & 3) * 64 + (M32 ? fl + j * 32 : lane);
  }
  const uint4* xg = (const uint4*)a.X + (size_t)(m0 >> 4) * 64;
  const size_t x_step = (size_t)a.MBn * 64, x_term = (size_t)S * x_step;
  if constexpr (M32) {
#pragma unroll
    for (int i = 0; i < MB / 2; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;
  } else {
#pragma unroll
    for (int j = 0; j < NBW; ++j)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) acc[j][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const int nst = st_end - st_beg;
  if (nst <= 0) return;
  const int nch = (nst + C - 1) / C;

#define TILE_LOAD_W(w, ch)                                                  \
  if (active) {                                                             \
    _Pragma("unroll") for (int sc = 0; sc < C; ++sc) {                      \
      const size_t st = (size_t)min(st_beg + (ch) * C + sc, st_end - 1);    \
      _Pragma("unroll") for (int j = 0; j < NBW; ++j) w[sc][j] = wt[j][st * 256]; \
    }                                                                       \
  }
#define TILE_LOAD_X(ch)                                                     \
  {                                                                         \
    _Pragma("unroll") for (int u = 0; u < TS::kXPT; ++u) {                  \
      const int e = threadIdx.x + u * kThreads; /* [step][term][mb][lane] */ \
      const int l = e & 63, mb = (e >> 6) % MB, q = (e / (64 * MB)) % NT, sc = e / (64 * MB * NT); \
      const size_t st = (size_t)min(st_beg + (ch) * C + sc, st_end - 1);   \
      xs[u] = xg[q * x_term + st * x_step + mb * 64 + l];                   \
    }                                                                       \
  }
#define TILE_STORE_X(ch)                                                    \
  {                                                                         \
    uint4* d = sx + ((ch) & 1) * TS::kXChunk + threadIdx.x;                 \
    _Pragma("unroll") for (int u = 0; u < TS::kXPT; ++u) d[u * kThreads] = xs[u]; \
  }
#define TILE_COMPUTE(w, ch)                                                 \
  if (active) {                                                             \
    const int valid = nst - (ch) * C;                                       \
    if constexpr (M32) {                                                    \
      const uint4* xb = sx + ((ch) & 1) * TS::kXChunk + sel * 64 + fl;      \
      _Pragma("unroll") for (int sc = 0; sc < C; ++sc) {                    \
        if (sc < valid) {                                                   \
          _Pragma("unroll") for (int q = 0; q < NT; ++q)                    \
          _Pragma("unroll") for (int i = 0; i < MB / 2; ++i)                \
          _Pragma("unroll") for (int h = 0; h < 2; ++h) {                   \
            const uint4 xv = xb[((sc * NT + q) * MB + 2 * i) * 64 + h * 32]; \
            acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(xv), as_bf16x8(w[sc][h]), acc[i], 0, 0, 0); \
          }                                                                 \
        }                                                                   \
      }                                                                     \
    } else {                                                                \
      const uint4* xb = sx + ((ch) & 1) * TS::kXChunk + lane;               \
      _Pragma("unroll") for (int sc = 0; sc < C; ++sc) {                    \
        if (sc < valid) {                                                   \
          _Pragma("unroll") for (int q = 0; q < NT; ++q)                    \
          _Pragma("unroll") for (int mb = 0; mb < MB; ++mb) {               \
            const uint4 xv = xb[((sc * NT + q) * MB + mb) * 64];            \
            _Pragma("unroll") for (int j = 0; j < NBW; ++j)                 \
              acc[j][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(xv), as_bf16x8(w[sc][j]), acc[j][mb], 0, 0, 0); \
          }                                                                 \
        }                                                                   \
      }                                                                     \
    }                                                                       \
  }
  // one chunk: prefetch X(ch+1) and W(ch+2), multiply chunk ch, publish
  // X(ch+1).  Past the last chunk the prefetches repeat it (unconditional
  // code keeps the staging registers out of scratch memory); the buffer
  // they fill is never read.
#define TILE_CHUNK(wcur, wnext2, ch)                                        \
  {                                                                         \
    TILE_LOAD_X(min((ch) + 1, nch - 1));                                    \
    TILE_LOAD_W(wnext2, min((ch) + 2, nch - 1));                            \
    TILE_COMPUTE(wcur, ch);                                                 \
    TILE_STORE_X((ch) + 1);                                                 \
    __syncthreads();                                                        \
  }
  // buffer indices are compile-time constants (a runtime index would put
  // the buffers in scratch memory): the chunk loop is unrolled by three
  uint4 w0[C][NBW], w1[C][NBW], w2[C][NBW];
  uint4 xs[TS::kXPT];
  TILE_LOAD_X(0);
  TILE_LOAD_W(w0, 0);
  TILE_LOAD_W(w1, min(1, nch - 1));
  TILE_STORE_X(0);
  __syncthreads();
  for (int ch = 0; ch < nch; ch += 3) {
    TILE_CHUNK(w0, w2, ch);
    if (ch + 1 >= nch) break;
    TILE_CHUNK(w1, w0, ch + 1);
    if (ch + 2 >= nch) break;
    TILE_CHUNK(w2, w1, ch + 2);
  }
#undef TILE_CHUNK
#undef TILE_COMPUTE
#undef TILE_STORE_X
#undef TILE_LOAD_X
#undef TILE_LOAD_W
}

// fp32 tile on the vector ALUs (X fragments with one fp32 term): rows
// m0 .. m0+16*MB, columns c0 .. c0+ncols (ncols <= kTileN), K range
// [k_beg, k_end), written to lds[r * ldc + c].  Thread t owns column
// t % kTileN and every other 8-wide K group (t / kTileN selects which); the
// 8 consecutive weights of a column and K group are 32 contiguous bytes of
// the packed layout (two float4 loads), used for the 16 rows of a row block
// (row blocks run one after another, so 16 accumulators suffice).  The two
// halves are added in LDS, half 0 + half 1, so the order is fixed.
template <int MB>
__device__ void tile_f32(const GemmArgs& a, int c0, int m0, int k_beg, int k_end, float* lds, int ncols = kTileN,
                         int ldc = kTileN) {
  static_assert(kThreads == 2 * kTileN, "two threads per column");
  const float4* W = (const float4*)a.W;
  const float4* X = (const float4*)a.X;
  const int steps = a.K >> 5;
  const int c = threadIdx.x % kTileN, part = threadIdx.x / kTileN;
  const int col = c0 + c;
  const bool live = c < ncols && col < a.N;
  // group of (col, k) in the packed layout: wbase + (k/32) * 256 + ((k%32)/8) * 16
  const size_t wbase = (size_t)(col >> 6) * steps * 256 + ((col & 63) >> 4) * 64 + (col & 15);
#pragma unroll 1
  for (int mb = 0; mb < MB; ++mb) {
    const int r0 = m0 + mb * 16;
    if (r0 >= a.M) break;  // uniform
    const int nr = min(16, a.M - r0);
    float acc[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    if (live) {
      for (int kg = (k_beg >> 3) + part; kg < (k_end >> 3); kg += 2) {
        const size_t wg = wbase + (size_t)(kg >> 2) * 256 + (kg & 3) * 16;
        const float4 w0 = W[wg * 2], w1 = W[wg * 2 + 1];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          if (r >= nr) break;  // uniform
          const size_t xg = afrag_group(0, r0 + r, kg * 8, steps, a.MBn);
          const float4 x0 = X[xg * 2], x1 = X[xg * 2 + 1];
          float t = acc[r];
          t = fmaf(x0.x, w0.x, t);
          t = fmaf(x0.y, w0.y, t);
          t = fmaf(x0.z, w0.z, t);
          t = fmaf(x0.w, w0.w, t);
          t = fmaf(x1.x, w1.x, t);
          t = fmaf(x1.y, w1.y, t);
          t = fmaf(x1.z, w1.z, t);
          t = fmaf(x1.w, w1.w, t);
          acc[r] = t;
        }
      }
    }
    float* o = lds + (size_t)mb * 16 * ldc + c;
    if (part == 1 && c < ncols)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[r * ldc] = acc[r];
    __syncthreads();
    if (part == 0 && c < ncols)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[r * ldc] = acc[r] + o[r * ldc];
    __syncthreads();
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

// Head tile epilogue, per head row: partial (max, second, sum-exp at the tile
// max, argmax), the logit of each draft token inside the tile, and the
// optional fp32 logits dump.  16 threads per row, 8 columns each.
template <int MB>
__device__ void epi_stats(const GemmArgs& a, int tile, int m0, const float* lds) {
  const int grp = threadIdx.x >> 4, gl = threadIdx.x & 15;  // 32 groups of 16 threads
  const int c0 = tile * kTileN;
  for (int r = grp; r < 16 * MB; r += kThreads / 16) {
    const int m = m0 + r;
    if (m >= a.M) continue;  // uniform within the group
    // the row's final RMSNorm scale (the head is linear in it)
    const float rs = row_scale(a.ss, a.ss_stride, m, a.K, a.eps);
    float mx = -INFINITY, sc = -INFINITY;
    int am = 0x7fffffff;
    constexpr int CPT = kTileN / 16;
    for (int c = gl * CPT; c < gl * CPT + CPT; ++c)
      if (c0 + c < a.N) merge3(mx, am, sc, lds[r * kTileN + c] * rs, c0 + c, -INFINITY);
    for (int o = 1; o < 16; o <<= 1) {
      const float mx2 = __shfl_xor(mx, o, 64), sc2 = __shfl_xor(sc, o, 64);
      const int am2 = __shfl_xor(am, o, 64);
      merge3(mx, am, sc, mx2, am2, sc2);
    }
    float se = 0.f;
    for (int c = gl * CPT; c < gl * CPT + CPT; ++c)
      if (c0 + c < a.N) se += expf((lds[r * kTileN + c] * rs - mx) * a.inv_T);
    for (int o = 1; o < 16; o <<= 1) se += __shfl_xor(se, o, 64);
    const int out = a.lm[m].out;
    if (gl == 0) {
      float* p = a.lm_part + ((size_t)tile * a.M + m) * 4;
      p[0] = mx;
      p[1] = sc;
      p[2] = se;
      p[3] = __int_as_float(am);
    }
    if (gl < min(a.lm[m].n_drafts, kMaxChildren)) {
      const int tk = a.lm[m].draft_tok[gl];
      if (tk >= c0 && tk < c0 + kTileN) a.draft_logit[a.lm[m].draft_idx[gl]] = lds[r * kTileN + tk - c0] * rs;
    }
    if (a.logits) {
      for (int c = gl * CPT; c < gl * CPT + CPT; ++c)
        if (c0 + c < a.N) a.logits[(size_t)out * a.N + c0 + c] = lds[r * kTileN + c] * rs;
    }
  }
}

template <typename T, int MB, int NT, int NBW, int C, bool STATS>
__device__ __forceinline__ void gemm_body(const GemmArgs& a) {
  using TS = TileShape<MB, NT, NBW, C>;
  static_assert(TS::kCols == kTileN, "tile width");
  constexpr int kLdsX = 2 * TS::kXChunk * 16;               // bytes of the X double buffer
  constexpr int kLdsT = 16 * MB * kTileN * 4;                // bytes of an fp32 output tile
  constexpr int kLds = (sizeof(T) == 2 ? kLdsX : 0) > kLdsT ? (sizeof(T) == 2 ? kLdsX : 0) : kLdsT;
  __shared__ __align__(16) unsigned char smem[kLds];
  float* lds = (float*)smem;
  // block -> (tile, split, m-group), m-group fastest
  const int mgroups = (a.M + 16 * MB - 1) / (16 * MB);
  int b = blockIdx.x;
  const int mg = b % mgroups;
  b /= mgroups;
  const int split = b % a.ksplit;
  const int tile = b / a.ksplit;
  const int m0 = mg * 16 * MB, c0 = tile * kTileN;
  const int steps = a.K >> 5, per = (steps + a.ksplit - 1) / a.ksplit;
  const int st_beg = min(steps, split * per), st_end = min(steps, (split + 1) * per);
  if constexpr (sizeof(T) == 2 && MB % 2 == 0 && NBW == 2) {
    // 32x32x16 MFMAs: tile i, register r of lane l is row 32i + (r/4)*8 + (l/32)*4 + r%4,
    // column wave*32 + l%32 of the work-group's tile
    f32x16 acc[MB / 2];
    tile_bf16<MB, NT, NBW, C, true>(a, c0, m0, st_beg, st_end, (uint4*)smem, acc);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int cl = wave * 32 + (lane & 31), rl = (lane >> 5) * 4;
    if constexpr (STATS) {
      __syncthreads();  // the X buffers become the output tile
#pragma unroll
      for (int i = 0; i < MB / 2; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) lds[(i * 32 + (r >> 2) * 8 + rl + (r & 3)) * kTileN + cl] = acc[i][r];
      __syncthreads();
      epi_stats<MB>(a, tile, m0, lds);
    } else {
      float* P = a.part + (size_t)split * a.M * a.N;
      const int col = c0 + cl;
#pragma unroll
      for (int i = 0; i < MB / 2; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = m0 + i * 32 + (r >> 2) * 8 + rl + (r & 3);
          if (m < a.M && col < a.N) P[(size_t)m * a.N + col] = acc[i][r];
        }
    }
  } else if constexpr (sizeof(T) == 2) {
    f32x4 acc[NBW][MB];
    tile_bf16<MB, NT, NBW, C>(a, c0, m0, st_beg, st_end, (uint4*)smem, acc);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, n = lane & 15, g = lane >> 4;
    if constexpr (STATS) {
      __syncthreads();  // the X buffers become the output tile
#pragma unroll
      for (int j = 0; j < NBW; ++j)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int r = 0; r < 4; ++r) lds[(mb * 16 + g * 4 + r) * kTileN + (wave * NBW + j) * 16 + n] = acc[j][mb][r];
      __syncthreads();
      epi_stats<MB>(a, tile, m0, lds);
    } else {
      float* P = a.part + (size_t)split * a.M * a.N;
#pragma unroll
      for (int j = 0; j < NBW; ++j) {
        const int col = c0 + (wave * NBW + j) * 16 + n;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int m = m0 + mb * 16 + g * 4 + r;
            if (m < a.M && col < a.N) P[(size_t)m * a.N + col] = acc[j][mb][r];
          }
      }
    }
  } else {
    tile_f32<MB>(a, c0, m0, st_beg * 32, st_end * 32, lds);
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
}

// Gate/up projection with SwiGLU, h = silu(x W_g) * (x W_u) (the verifier's FFN).
// The packed weight interleaves gate and up rows by 8 (launch_pack with ffn),
// so 16-column block b holds gate and up columns of f = 8b .. 8b+7.  A
// work-group owns a.nb consecutive blocks (one wave each; waves past nb only
// stage X) over all of K, so no partial sums leave it: the tile goes to LDS
// and the epilogue writes h for its (row, 8-f group)s as 2-term fragments,
// the down projection's input.
template <typename T, int MB, int C>
__global__ __launch_bounds__(kThreads) void gemm_gate_up(GemmArgs a) {
  constexpr int NT = sizeof(T) == 2 ? 2 : 1;
  constexpr int kCols = kWaves * 16;                        // widest tile (nb = 8)
  constexpr int kLdsX = sizeof(T) == 2 ? 2 * TileShape<MB, NT, 1, C>::kXChunk * 16 : 0;
  constexpr int kLdsT = 16 * MB * kCols * 4;
  constexpr int kLds = kLdsX > kLdsT ? kLdsX : kLdsT;
  __shared__ __align__(16) unsigned char smem[kLds];
  float* lds = (float*)smem;
  const int nblocks = a.N >> 4;             // 16-column blocks (= F / 8 groups of h)
  const int blk0 = blockIdx.x * a.nb;
  const int m0 = blockIdx.y * 16 * MB;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int ncol = min(a.nb, nblocks - blk0) * 16;  // columns of this work-group
  if constexpr (sizeof(T) == 2 && MB % 2 == 0 && MB >= 4) {
    // 64 or more rows: each wave owns a pair of blocks on 32x32x16 MFMAs, so
    // every X fragment read from LDS serves 32 columns (a.nb even; waves past
    // nb / 2 only stage X).  One block per wave makes the LDS reads of X the
    // limit.
    f32x16 acc[MB / 2];
    const bool active = 2 * wave < a.nb && blk0 + 2 * wave < nblocks;
    tile_bf16<MB, NT, 2, C, true>(a, blk0 * 16, m0, 0, a.K >> 5, (uint4*)smem, acc, active);
    __syncthreads();  // the X buffers become the output tile
    if (active) {
      // tile i, register r of lane l: row 32i + (r/4)*8 + (l/32)*4 + r%4, column wave*32 + l%32
      const int cl = wave * 32 + (lane & 31), rl = (lane >> 5) * 4;
#pragma unroll
      for (int i = 0; i < MB / 2; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) lds[(i * 32 + (r >> 2) * 8 + rl + (r & 3)) * kCols + cl] = acc[i][r];
    }
  } else if constexpr (sizeof(T) == 2) {
    f32x4 acc[1][MB];
    const bool active = wave < a.nb && blk0 + wave < nblocks;
    tile_bf16<MB, NT, 1, C>(a, blk0 * 16, m0, 0, a.K >> 5, (uint4*)smem, acc, active);
    __syncthreads();  // the X buffers become the output tile
    if (active) {
      const int n = lane & 15, g = lane >> 4;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r) lds[(mb * 16 + g * 4 + r) * kCols + wave * 16 + n] = acc[0][mb][r];
    }
  } else {
    tile_f32<MB>(a, blk0 * 16, m0, 0, a.K, lds, ncol, kCols);
  }
  __syncthreads();
  const int ngroups = ncol >> 4;
  for (int e = threadIdx.x; e < 16 * MB * ngroups; e += kThreads) {
    const int r = e / ngroups, j = e - r * ngroups, m = m0 + r;
    if (m >= a.M) continue;
    const float* t = lds + r * kCols + j * 16;
    const float sc = row_scale(a.ss, a.ss_stride, m, a.K, a.eps);  // RMSNorm of the input row
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float gt = t[i] * sc, up = t[8 + i] * sc;
      v[i] = gt / (1.0f + expf(-gt)) * up;
    }
    put_afrag<sizeof(T) == 2, NT>(a.H, m, (blk0 + j) * 8, v, a.F >> 5, a.MBn);
  }
}

// Gate/up with SwiGLU for up to 32 rows, K-interleaved: wave w multiplies
// K steps w, w + 8, w + 16, ... of all a.nb (<= 8) column blocks of the
// work-group, loading its X fragments straight from global memory (each is
// used by one wave only, so neither LDS staging nor a barrier sits in the
// main loop), one step of loads ahead of its MFMAs.  Weights are read with
// non-temporal loads: streamed once, they should not displace X from the
// caches.  The eight waves' partial tiles are summed in LDS in wave order
// (fixed, so the result is reproducible) and the epilogue writes h as in
// gemm_gate_up.
__device__ __forceinline__ uint4 load_stream(const uint4* p) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 v = __builtin_nontemporal_load((const u32x4*)p);
  return make_uint4(v.x, v.y, v.z, v.w);
}

template <int MB>
__global__ __launch_bounds__(kThreads) void gemm_gate_up_ki(GemmArgs a) {
  constexpr int NT = 2, NBM = kWaves;
  __shared__ __align__(16) float red[kWaves][16 * MB][NBM * 16 + 4];
  const int nblocks = a.N >> 4;
  const int blk0 = blockIdx.x * a.nb;
  const int m0 = blockIdx.y * 16 * MB;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nb = min(a.nb, nblocks - blk0);
  const int S = a.K >> 5, t64 = (a.N + 63) >> 6;
  const uint4* wt[NBM];
#pragma unroll
  for (int j = 0; j < NBM; ++j) {
    const int blk = blk0 + min(j, nb - 1);
    wt[j] = (const uint4*)a.W + (size_t)min(blk >> 2, t64 - 1) * S * 256 + (blk & 3) * 64 + lane;
  }
  const uint4* xg = (const uint4*)a.X + (size_t)(m0 >> 4) * 64 + lane;
  const size_t x_step = (size_t)a.MBn * 64, x_term = (size_t)S * x_step;
  f32x4 acc[NBM][MB];
#pragma unroll
  for (int j = 0; j < NBM; ++j)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[j][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int nst = max(0, (S - wave + kWaves - 1) / kWaves);  // steps of this wave
  uint4 w[2][NBM], x[2][NT][MB];
  // loads of the wave's i-th step into buffer `buf` (past the last step the
  // last one is loaded again and never used)
  auto load = [&](int buf, int i) {
    const size_t st = (size_t)(wave + min(i, nst - 1) * kWaves);
#pragma unroll
    for (int j = 0; j < NBM; ++j)
      if (j < nb) w[buf][j] = load_stream(wt[j] + st * 256);
#pragma unroll
    for (int q = 0; q < NT; ++q)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) x[buf][q][mb] = xg[q * x_term + st * x_step + mb * 64];
  };
  auto compute = [&](int buf) {
#pragma unroll
    for (int q = 0; q < NT; ++q)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int j = 0; j < NBM; ++j)
          if (j < nb)
            acc[j][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(x[buf][q][mb]), as_bf16x8(w[buf][j]),
                                                                 acc[j][mb], 0, 0, 0);
  };
  if (nst > 0) {
    load(0, 0);
    for (int i = 0; i < nst; i += 2) {
      load(1, i + 1);
      compute(0);
      if (i + 1 >= nst) break;
      load(0, i + 2);
      compute(1);
    }
  }
  const int n = lane & 15, g = lane >> 4;
#pragma unroll
  for (int j = 0; j < NBM; ++j)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[wave][mb * 16 + g * 4 + r][j * 16 + n] = acc[j][mb][r];
  __syncthreads();
  for (int e = threadIdx.x; e < 16 * MB * nb; e += kThreads) {
    const int r = e / nb, j = e - r * nb, m = m0 + r;
    if (m >= a.M) continue;
    const float sc = row_scale(a.ss, a.ss_stride, m, a.K, a.eps);  // RMSNorm of the input row
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      float gt = 0.f, up = 0.f;
#pragma unroll
      for (int wv = 0; wv < kWaves; ++wv) {
        gt += red[wv][r][j * 16 + i];
        up += red[wv][r][j * 16 + 8 + i];
      }
      gt *= sc;
      up *= sc;
      v[i] = gt / (1.0f + expf(-gt)) * up;
    }
    put_afrag<true, NT>(a.H, m, (blk0 + j) * 8, v, a.F >> 5, a.MBn);
  }
}

// One entry point per projection, so kernel traces name the projection.
#define VIA_GEMM_ENTRY(NAME, NT_BF16, STATS)                                              \
  template <typename T, int MB, int C>                                                   \
  __global__ __launch_bounds__(kThreads) void NAME(GemmArgs a) {                         \
    gemm_body<T, MB, (sizeof(T) == 2 ? NT_BF16 : 1), kNBW, C, STATS>(a);                 \
  }
VIA_GEMM_ENTRY(gemm_qkv, kQkvTerms, false)
VIA_GEMM_ENTRY(gemm_o, 2, false)
VIA_GEMM_ENTRY(gemm_down, 2, false)
VIA_GEMM_ENTRY(gemm_head, 2, true)
#undef VIA_GEMM_ENTRY

// X chunk steps: the double-buffered chunk stays within 144 KB of LDS and
// splits evenly over the threads (C * NT * MB a multiple of 8).
template <typename T, int MB, int NT, int NBW = kNBW>
constexpr int chunk_steps() {
  if (sizeof(T) != 2) return 8;
  if (MB > 4) return NT * MB == 24 ? 2 : 4;  // 96 or 128 rows: 72-128 KB of buffers
  return (NBW == 1 && NT * MB <= 9) || (NT * MB) % 2 ? 8 : 4;
}
// With timing events the launch carries them in its dispatch, so they
// bracket the kernel itself rather than the stream around it.
#define VIA_GEMM_LAUNCH(NAME, NT_BF16)                                                       \
  template <typename T>                                                                      \
  void launch_##NAME(const GemmArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {       \
    constexpr int NT = sizeof(T) == 2 ? NT_BF16 : 1;                                         \
    const int mb = gemm_rows_per_group(a.M) / 16;                                            \
    const int mgroups = (a.M + 16 * mb - 1) / (16 * mb);                                     \
    const dim3 grid(gemm_tiles(a.N) * a.ksplit * mgroups);                                   \
    auto go = [&](auto kernel) {                                                             \
      if (e0)                                                                                \
        hipExtLaunchKernelGGL(kernel, grid, dim3(kThreads), 0, s, e0, e1, 0, a);             \
      else                                                                                   \
        hipLaunchKernelGGL(kernel, grid, dim3(kThreads), 0, s, a);                           \
    };                                                                                       \
    switch (mb) {                                                                            \
      case 1: go(NAME<T, 1, chunk_steps<T, 1, NT>()>); break;                                \
      case 2: go(NAME<T, 2, chunk_steps<T, 2, NT>()>); break;                                \
      case 3: go(NAME<T, 3, chunk_steps<T, 3, NT>()>); break;                                \
      case 4: go(NAME<T, 4, chunk_steps<T, 4, NT>()>); break;                                \
      case 6: go(NAME<T, 6, chunk_steps<T, 6, NT>()>); break;                                \
      default: go(NAME<T, 8, chunk_steps<T, 8, NT>()>); break;                               \
    }                                                                                        \
  }
VIA_GEMM_LAUNCH(gemm_qkv, kQkvTerms)
VIA_GEMM_LAUNCH(gemm_o, 2)

// Gate/up with SwiGLU: grid (work-groups of a.nb blocks, row groups).
template <typename T>
void launch_gemm_gate_up(const GemmArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  constexpr int NT = sizeof(T) == 2 ? 2 : 1;
  const int mb = gemm_rows_per_group(a.M) / 16;
  const int mgroups = (a.M + 16 * mb - 1) / (16 * mb);
  GemmArgs b = a;
  if (sizeof(T) == 2 && mb >= 4 && mb % 2 == 0)  // block pairs per wave: an even count, ~256 work-groups
    b.nb = std::min(kWaves, 2 * std::max(1, ((a.N >> 4) + 511) / 512));
  const dim3 grid(((b.N >> 4) + b.nb - 1) / b.nb, mgroups);
  auto go = [&](auto kernel) {
    if (e0)
      hipExtLaunchKernelGGL(kernel, grid, dim3(kThreads), 0, s, e0, e1, 0, b);
    else
      hipLaunchKernelGGL(kernel, grid, dim3(kThreads), 0, s, b);
  };
  if constexpr (sizeof(T) == 2) {
    if (mb <= 2) {  // up to 32 rows: K-interleaved waves
      if (mb == 1)
        go(gemm_gate_up_ki<1>);
      else
        go(gemm_gate_up_ki<2>);
      return;
    }
  }
  switch (mb) {
    case 1: go(gemm_gate_up<T, 1, chunk_steps<T, 1, NT, 1>()>); break;
    case 2: go(gemm_gate_up<T, 2, chunk_steps<T, 2, NT, 1>()>); break;
    case 3: go(gemm_gate_up<T, 3, chunk_steps<T, 3, NT, 1>()>); break;
    case 4: go(gemm_gate_up<T, 4, chunk_steps<T, 4, NT, 2>()>); break;  // block pairs (bf16)
    case 6: go(gemm_gate_up<T, 6, chunk_steps<T, 6, NT, 1>()>); break;
    default: go(gemm_gate_up<T, 8, chunk_steps<T, 8, NT, 1>()>); break;
  }
}
VIA_GEMM_LAUNCH(gemm_down, 2)
VIA_GEMM_LAUNCH(gemm_head, 2)
#undef VIA_GEMM_LAUNCH


// QKV, O and down projections of forwards of up to 32 rows (bf16): the
// weight-streaming decomposition of the gate/up kernel with split-K partials.
// A work-group owns a.nb 16-column blocks and K split blockIdx.x % a.ksplit (a.ksplit
// equal ranges of 32-wide steps); its 8 waves interleave the split's steps
// (wave w takes steps w, w+8, ...) over all its blocks, loading X fragments
// straight from global memory (each is used by one wave; they stay in L2)
// and weights with non-temporal loads, one step ahead.  The 8 wave partial
// tiles are summed in LDS in wave order and written to
// a.part[split][M][N], which the consumer sums in split order.  Fewer,
// longer splits than the LDS-staged kernels write a quarter of the partials.
template <int MB, int NT>
__global__ __launch_bounds__(kThreads) void gemm_ki_part(GemmArgs a) {
  constexpr int NBM = kWaves;
  __shared__ __align__(16) float red[kWaves][16 * MB][NBM * 16 + 4];
  const int nblocks = a.N >> 4;
  const int split = blockIdx.x % a.ksplit;
  const int blk0 = (blockIdx.x / a.ksplit) * a.nb;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nb = min(a.nb, nblocks - blk0);
  const int S = a.K >> 5, t64 = (a.N + 63) >> 6;
  const int per = (S + a.ksplit - 1) / a.ksplit;
  const int s_beg = min(S, split * per), s_end = min(S, s_beg + per);
  const uint4* wt[NBM];
#pragma unroll
  for (int j = 0; j < NBM; ++j) {
    const int blk = blk0 + min(j, nb - 1);
    wt[j] = (const uint4*)a.W + (size_t)min(blk >> 2, t64 - 1) * S * 256 + (blk & 3) * 64 + lane;
  }
  const uint4* xg = (const uint4*)a.X + lane;
  const size_t x_step = (size_t)a.MBn * 64, x_term = (size_t)S * x_step;
  f32x4 acc[NBM][MB];
#pragma unroll
  for (int j = 0; j < NBM; ++j)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[j][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int nst = max(0, (s_end - s_beg - wave + kWaves - 1) / kWaves);  // steps of this wave
  uint4 w[2][NBM], x[2][NT][MB];
  // loads of the wave's i-th step into buffer `buf` (past the last step the
  // last one is loaded again and never used)
  auto load = [&](int buf, int i) {
    const size_t st = (size_t)(s_beg + wave + min(i, nst - 1) * kWaves);
#pragma unroll
    for (int j = 0; j < NBM; ++j)
      if (j < nb) w[buf][j] = load_stream(wt[j] + st * 256);
#pragma unroll
    for (int q = 0; q < NT; ++q)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) x[buf][q][mb] = xg[q * x_term + st * x_step + mb * 64];
  };
  auto compute = [&](int buf) {
#pragma unroll
    for (int q = 0; q < NT; ++q)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int j = 0; j < NBM; ++j)
          if (j < nb)
            acc[j][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(x[buf][q][mb]), as_bf16x8(w[buf][j]),
                                                                 acc[j][mb], 0, 0, 0);
  };
  if (nst > 0) {
    load(0, 0);
    for (int i = 0; i < nst; i += 2) {
      load(1, i + 1);
      compute(0);
      if (i + 1 >= nst) break;
      load(0, i + 2);
      compute(1);
    }
  }
  const int n = lane & 15, g = lane >> 4;
#pragma unroll
  for (int j = 0; j < NBM; ++j)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[wave][mb * 16 + g * 4 + r][j * 16 + n] = acc[j][mb][r];
  __syncthreads();
  float* P = a.part + (size_t)split * a.M * a.N;
  const int cols = nb * 16;
  for (int e = threadIdx.x; e < 16 * MB * cols; e += kThreads) {
    const int r = e / cols, c = e - r * cols;
    if (r >= a.M) continue;
    float v = 0.f;
#pragma unroll
    for (int wv = 0; wv < kWaves; ++wv) v += red[wv][r][c];
    P[(size_t)r * a.N + blk0 * 16 + c] = v;
  }
}

// The same decomposition at a fixed shape: NB blocks per work-group and
// exactly NSW steps per wave, fully unrolled, with the loads of DEPTH steps
// in flight (a ring of DEPTH register buffers) instead of one.  Used when
// the K split and the column blocks divide evenly.
template <int MB, int NT, int NB, int NSW, int DEPTH>
__global__ __launch_bounds__(kThreads) void gemm_ki_fixed(GemmArgs a) {
  __shared__ __align__(16) float red[kWaves][16 * MB][NB * 16 + 4];
  const int split = blockIdx.x % a.ksplit;
  const int blk0 = (blockIdx.x / a.ksplit) * NB;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int S = a.K >> 5, t64 = (a.N + 63) >> 6;
  const int s_beg = split * NSW * kWaves;
  const uint4* wt[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int blk = blk0 + j;
    wt[j] = (const uint4*)a.W + (size_t)min(blk >> 2, t64 - 1) * S * 256 + (blk & 3) * 64 + lane;
  }
  const uint4* xg = (const uint4*)a.X + lane;
  const size_t x_step = (size_t)a.MBn * 64, x_term = (size_t)S * x_step;
  f32x4 acc[NB][MB];
#pragma unroll
  for (int j = 0; j < NB; ++j)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[j][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
  uint4 w[DEPTH][NB], x[DEPTH][NT][MB];
  // iteration i multiplies step i - DEPTH (its buffer) and then loads step i into it
#pragma unroll
  for (int i = 0; i < NSW + DEPTH; ++i) {
    if (i >= DEPTH) {
      const int b = (i - DEPTH) % DEPTH;
#pragma unroll
      for (int q = 0; q < NT; ++q)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int j = 0; j < NB; ++j)
            acc[j][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(x[b][q][mb]), as_bf16x8(w[b][j]),
                                                                 acc[j][mb], 0, 0, 0);
    }
    if (i < NSW) {
      const int b = i % DEPTH;
      const size_t st = (size_t)(s_beg + wave + i * kWaves);
#pragma unroll
      for (int j = 0; j < NB; ++j) w[b][j] = load_stream(wt[j] + st * 256);
#pragma unroll
      for (int q = 0; q < NT; ++q)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) x[b][q][mb] = xg[q * x_term + st * x_step + mb * 64];
    }
  }
  const int n = lane & 15, g = lane >> 4;
#pragma unroll
  for (int j = 0; j < NB; ++j)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[wave][mb * 16 + g * 4 + r][j * 16 + n] = acc[j][mb][r];
  __syncthreads();
  float* P = a.part + (size_t)split * a.M * a.N;
  constexpr int cols = NB * 16;
  for (int e = threadIdx.x; e < 16 * MB * cols; e += kThreads) {
    const int r = e / cols, c = e - r * cols;
    if (r >= a.M) continue;
    float v = 0.f;
#pragma unroll
    for (int wv = 0; wv < kWaves; ++wv) v += red[wv][r][c];
    P[(size_t)r * a.N + blk0 * 16 + c] = v;
  }
}

template <int NT>
void launch_ki_part(const GemmArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  // split-major order: work-group i takes K split i % ksplit, so with the
  // round-robin dispatch of work-groups over the 8 XCDs each XCD's
  // work-groups share 8 / ksplit splits (one for 8 splits) and its L2 holds
  // only their slices of the activations
  const dim3 grid((((a.N >> 4) + a.nb - 1) / a.nb) * a.ksplit);
  auto go = [&](auto kernel) {
    if (e0)
      hipExtLaunchKernelGGL(kernel, grid, dim3(kThreads), 0, s, e0, e1, 0, a);
    else
      hipLaunchKernelGGL(kernel, grid, dim3(kThreads), 0, s, a);
  };
  // fixed shapes (the 8B and 1B projections): even K splits and column blocks
  const int S = a.K >> 5, per = S / a.ksplit, nsw = per / kWaves;
  if (S % a.ksplit == 0 && per % kWaves == 0 && (a.N >> 4) % a.nb == 0) {
#define VIA_KI_FIXED(NB_, NSW_)                                                   \
  if (a.nb == NB_ && nsw == NSW_) {                                              \
    if (a.M <= 16)                                                               \
      go(gemm_ki_fixed<1, NT, NB_, NSW_, 2>);                                    \
    else                                                                         \
      go(gemm_ki_fixed<2, NT, NB_, NSW_, 2>);                                    \
    return;                                                                      \
  }
    VIA_KI_FIXED(6, 4)
    VIA_KI_FIXED(4, 4)
    VIA_KI_FIXED(8, 7)
    VIA_KI_FIXED(2, 4)
    VIA_KI_FIXED(1, 4)
#undef VIA_KI_FIXED
  }
  if (a.M <= 16)
    go(gemm_ki_part<1, NT>);
  else
    go(gemm_ki_part<2, NT>);
}

template <typename T>
void launch_role(GemmRole role, const GemmArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  switch (role) {
    case GemmRole::kQkv: launch_gemm_qkv<T>(a, s, e0, e1); break;
    case GemmRole::kO: launch_gemm_o<T>(a, s, e0, e1); break;
    case GemmRole::kGateUp: launch_gemm_gate_up<T>(a, s, e0, e1); break;
    case GemmRole::kDown: launch_gemm_down<T>(a, s, e0, e1); break;
    case GemmRole::kHead: launch_gemm_head<T>(a, s, e0, e1); break;
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

// Row-major [rows, cols] -> packed tiles; one thread per 8-element group.
template <typename T>
__global__ __launch_bounds__(256) void pack_kernel(const T* src, T* dst, int rows, int cols, int ffn, size_t groups) {
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
  // gate/up interleave: packed row 16 b + i <- gate row 8 b + i, or up row 8 b + i - 8
  const size_t sr = ffn > 0 ? ((r & 8) ? (size_t)ffn : 0) + (r >> 4) * 8 + (r & 7) : r;
#pragma unroll
  for (int e = 0; e < 8; ++e) dst[gidx * 8 + e] = r < (size_t)rows ? src[sr * cols + c + e] : T(0);
}

// ------------------------------------------------------------- prefill GEMM
// Many-row GEMM (prefill-sized M): C[M, N] = sum over the NT activation terms
// of X_q[M, K] W[N, K]^T, fp32, written as one partial tile (split 1) so the
// consumers of the verify GEMMs read it unchanged.  Compute-bound: a
// work-group of 8 waves owns a 256 x 256 tile; wave (wm, wn) computes rows
// wm*128 .. +128 and columns wn*64 .. +64 with v_mfma_f32_16x16x32_bf16.  A
// stage is one 32-wide K step of the tile: 16 row blocks of X and 16 column
// blocks of W, each a contiguous 1 KB fragment in both layouts, copied
// verbatim into LDS by global_load_lds_dwordx4 (16 bytes per lane written at
// m0 + 16 * lane).  Four stages rotate in LDS, two K steps per barrier:
// stage s is copied two to four steps ahead, read into registers during step
// s - 1 and multiplied in step s, so a wave's products never wait for LDS
// after a barrier; the reads of the next step are pinned between the
// products (one read per two MFMAs) so that the compiler cannot sink them
// next to their use again.  The copies are issued
// by inline asm with wave-uniform bases in SGPRs (one lane-offset VGPR for
// all of them) so that the compiler, which would otherwise make every LDS
// read wait for all outstanding copies, leaves their completion to the
// explicit vmcnt waits below.  Work-groups are dispatched
// round-robin over the 8 XCDs; XCD x takes a contiguous range of tiles, taken
// in groups of 8 row tiles so that co-resident work-groups share operand
// blocks in its L2.
//
// SWIGLU (the gate/up projection): instead of the fp32 product the tile's
// epilogue writes h = silu(g s) * (u s) with the input row's RMSNorm scale
// s, as 2-term fragments of the down projection's input.  A 16-column block
// of the packed gate/up weight holds the gate (columns 0-7) and up (8-15)
// rows of the same 8 FFN indices, so lane n < 8 of an output block takes its
// up value from lane n + 8; h of the tile's 128 FFN indices is staged in LDS
// (the freed operand stages) and written 8 indices per fragment group.
constexpr int kPfBM = 256, kPfBN = 256, kPfStages = 4, kPfStage = 32 * 1024;
constexpr int kPfGroupM = 8;
constexpr int kPfHStride = kPfBN / 2 + 4;  // fp32 per staged h row (padded: no bank conflicts)
constexpr int kPfLds = kPfStages * kPfStage > kPfBM * kPfHStride * 4 ? kPfStages * kPfStage : kPfBM * kPfHStride * 4;

// 16 bytes per lane from base + voff to LDS at lds + 16 * lane (base wave-uniform)
__device__ __forceinline__ void lds_dma16(const void* base, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(base), "s"(lds) : "memory", "m0");
}

template <bool SWIGLU, bool PAIR>
__global__ __launch_bounds__(kThreads, 1) void gemm_prefill(GemmArgs a, int nt) {
  __shared__ __align__(1024) unsigned char smem[SWIGLU ? kPfLds : kPfStages * kPfStage];
  const int S = a.K >> 5, t64 = (a.N + 63) >> 6;
  const int tiles_n = (a.N + kPfBN - 1) / kPfBN, tiles_m = (a.M + kPfBM - 1) / kPfBM;
  const int ntiles = tiles_m * tiles_n;
  const int per = (ntiles + 7) / 8;
  const int tile = (blockIdx.x % 8) * per + blockIdx.x / 8;
  if (tile >= ntiles) return;  // uniform
  const int grp = tile / (kPfGroupM * tiles_n), in = tile % (kPfGroupM * tiles_n);
  const int gm = min(kPfGroupM, tiles_m - grp * kPfGroupM);
  const int m0 = (grp * kPfGroupM + in % gm) * kPfBM, n0 = (in / gm) * kPfBN;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave >> 2, wn = wave & 3;
  // K32 steps over all terms.  PAIR (two terms): step it is term it % 2 of
  // K step it / 2, so a K step's two terms run back to back and the second
  // reuses the first's W operands (no W copy or W read for it); otherwise
  // term-major, step it is term it / S of K step it % S.
  const int iters = nt * S;
  // wave w copies row blocks w, w + 8 and column blocks w, w + 8 of each stage;
  // blocks past the matrix are clamped (their products are never stored)
  const uint4* xs[2];
  const uint4* ws[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    xs[h] = (const uint4*)a.X + (size_t)min((m0 >> 4) + h * 8 + wave, a.MBn - 1) * 64;
    const int cb = (n0 >> 4) + h * 8 + wave;
    ws[h] = (const uint4*)a.W + (size_t)min(cb >> 2, t64 - 1) * S * 256 + (cb & 3) * 64;
  }
  const size_t xstep = (size_t)a.MBn * 64;
  const uint32_t voff = lane * 16;
  const uint32_t lds_base =
      __builtin_amdgcn_readfirstlane((uint32_t)(size_t)(__attribute__((address_space(3))) void*)(smem + wave * 1024));
  auto issue = [&](int it) {
    const int q = PAIR ? (it & 1) : it / S, ks = PAIR ? it >> 1 : it - q * S;
    const uint32_t d = lds_base + (it % kPfStages) * kPfStage;
    lds_dma16(xs[0] + ((size_t)q * S + ks) * xstep, voff, d);
    lds_dma16(xs[1] + ((size_t)q * S + ks) * xstep, voff, d + 8 * 1024);
    if (!PAIR || q == 0) {
      lds_dma16(ws[0] + (size_t)ks * 256, voff, d + 16 * 1024);
      lds_dma16(ws[1] + (size_t)ks * 256, voff, d + 24 * 1024);
    }
  };
  f32x4 acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int p = 0; p < kPfStages - 1; ++p) issue(min(p, iters - 1));
  // SwiGLU: the RMSNorm scales of the tile's input rows, read while the
  // first stages are in flight
  __shared__ float rscale[SWIGLU ? kPfBM : 1];
  if constexpr (SWIGLU)
    for (int r = threadIdx.x; r < kPfBM; r += kThreads)
      rscale[r] = m0 + r < a.M ? row_scale(a.ss, a.ss_stride, m0 + r, a.K, a.eps) : 0.f;
  // operands of one step: 8 row blocks of X, 4 column blocks of W
  uint4 pa[8], pb[4], qa[8], qb[4];
  auto read = [&](int it, uint4* A, uint4* B) {  // B null: X only
    const uint4* st = (const uint4*)(smem + (it % kPfStages) * kPfStage);
#pragma unroll
    for (int i = 0; i < 8; ++i) A[i] = st[(wm * 8 + i) * 64 + lane];
    if (B)
#pragma unroll
      for (int j = 0; j < 4; ++j) B[j] = st[(16 + wn * 4 + j) * 64 + lane];
  };
  auto mma = [&](const uint4* A, const uint4* B) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(A[i]), as_bf16x8(B[j]), acc[i][j], 0, 0, 0);
  };
  // the products of one step with the reads of the next (NR of them) pinned
  // between them
#define VIA_PF_PIN(NR)                                                                 \
  _Pragma("unroll") for (int g = 0; g < (NR); ++g) {                                   \
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0); /* 2 MFMAs */                   \
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0); /* 1 LDS read */                \
  }                                                                                    \
  __builtin_amdgcn_sched_group_barrier(0x008, 32 - 2 * (NR), 0);
  // stage 0 in LDS (the oldest 4 copies of the 12, PAIR: of 10) and in registers
  __builtin_amdgcn_s_waitcnt((PAIR ? 6 : 4 * (kPfStages - 2)) | (0x7 << 4) | (0xF << 8));
  __builtin_amdgcn_s_barrier();
  read(0, pa, pb);
  // two steps per barrier, it and it + 1, with the register sets swapped: at
  // the barrier every copy has landed (stages it + 1 and it + 2 are read in
  // this trip) and every wave's reads of stages it - 1 and it are back
  // (lgkmcnt 0), so their buffers take stages it + 3 and it + 4 (past the end
  // the last stage is copied again into a buffer nothing reads).  One exit
  // only: an exit between the halves makes the compiler spill.
  int it = 0;
  for (; it + 1 < iters; it += 2) {
    __builtin_amdgcn_s_waitcnt(0x0 | (0x7 << 4) | (0x0 << 8));
    __builtin_amdgcn_s_barrier();
    issue(min(it + 3, iters - 1));
    issue(min(it + 4, iters - 1));
    // PAIR: step it + 1 (second term) multiplies its X with step it's W
    // (pb), and the next K step's W goes to qb, moved to pb afterwards
    read(min(it + 1, iters - 1), qa, PAIR ? nullptr : qb);
    mma(pa, pb);
    VIA_PF_PIN(PAIR ? 8 : 12)
    read(min(it + 2, iters - 1), pa, PAIR ? qb : pb);
    mma(qa, PAIR ? pb : qb);
    VIA_PF_PIN(12)
    if constexpr (PAIR)
#pragma unroll
      for (int j = 0; j < 4; ++j) pb[j] = qb[j];
  }
#undef VIA_PF_PIN
  if (it < iters) mma(pa, pb);  // odd step count (not PAIR): the last stage is in pa, pb
  __builtin_amdgcn_s_waitcnt(0);  // the trailing copies land before the work-group ends
  const int n = lane & 15, g = lane >> 4;
  if constexpr (SWIGLU) {
    __syncthreads();  // every wave's copies have landed and its stage reads are done
    float* hl = (float*)smem;  // [row][FFN index of the tile]
    // lane n < 8 of a 16-lane row holds the gate value of FFN index n, lane
    // n + 8 its up value (rows g * 4 + r).  The pair swaps its four values
    // with a DPP rotate by 8 within the row (xor 8: no LDS round trip), and
    // lane n < 8 computes h for rows r = 0, 1, lane n + 8 for rows 2, 3, so
    // every lane runs the same instructions.
    const bool lo8 = n < 8;
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float other[4];
#pragma unroll
        for (int r = 0; r < 4; ++r)
          other[r] = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(acc[i][j][r]), 0x128, 0xf, 0xf, false));
#pragma unroll
        for (int rr = 0; rr < 2; ++rr) {
          const float gv = lo8 ? acc[i][j][rr] : other[rr + 2];
          const float uv = lo8 ? other[rr] : acc[i][j][rr + 2];
          const int rl = wm * 128 + i * 16 + g * 4 + rr + (lo8 ? 0 : 2);
          const float sc = rscale[rl], gt = gv * sc, u = uv * sc;
          hl[rl * kPfHStride + wn * 32 + j * 8 + (n & 7)] = gt / (1.0f + expf(-gt)) * u;
        }
      }
    __syncthreads();
    // consecutive lanes take consecutive rows of one 8-index group: 16 of
    // them write 256 contiguous bytes of a fragment term
    const int f0 = n0 >> 1;
    for (int e = threadIdx.x; e < kPfBM * (kPfBN / 16); e += kThreads) {
      const int rl = e % kPfBM, gq = e / kPfBM, m = m0 + rl, f = f0 + gq * 8;
      if (m >= a.M || f >= a.F) continue;
      float v[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) v[t] = hl[rl * kPfHStride + gq * 8 + t];
      put_afrag<true, 2>(a.H, m, f, v, a.F >> 5, a.MBn);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int col = n0 + wn * 64 + j * 16 + n;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = m0 + wm * 128 + i * 16 + g * 4 + r;
          if (row < a.M && col < a.N) a.part[(size_t)row * a.N + col] = acc[i][j][r];
        }
      }
  }
}

void launch_prefill(const GemmArgs& a, int nt, bool swiglu, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const int ntiles = ((a.M + kPfBM - 1) / kPfBM) * ((a.N + kPfBN - 1) / kPfBN);
  const dim3 grid((ntiles + 7) / 8 * 8);
  auto go = [&](auto kernel) {
    if (e0)
      hipExtLaunchKernelGGL(kernel, grid, dim3(kThreads), 0, s, e0, e1, 0, a, nt);
    else
      hipLaunchKernelGGL(kernel, grid, dim3(kThreads), 0, s, a, nt);
  };
  if (swiglu && nt == 2)
    go(gemm_prefill<true, true>);
  else if (swiglu)
    go(gemm_prefill<true, false>);
  else if (nt == 2)
    go(gemm_prefill<false, true>);
  else
    go(gemm_prefill<false, false>);
}

}  // namespace

void launch_pack(bool bf16, const void* src, void* dst, int rows, int cols, int ffn, hipStream_t s) {
  const size_t groups = (size_t)((rows + 63) / 64) * 64 * (cols / 8);
  const dim3 grid((unsigned)((groups + 255) / 256));
  if (bf16)
    hipLaunchKernelGGL(pack_kernel<uint16_t>, grid, dim3(256), 0, s, (const uint16_t*)src, (uint16_t*)dst, rows, cols,
                       ffn, groups);
  else
    hipLaunchKernelGGL(pack_kernel<float>, grid, dim3(256), 0, s, (const float*)src, (float*)dst, rows, cols, ffn,
                       groups);
}

int gate_up_blocks_per_group(int F) {
  const int nblocks = F / 8;  // 2 F columns in blocks of 16
  return std::max(1, std::min(kWaves, (nblocks + 255) / 256));
}

int gemm_tiles(int N) { return (N + kTileN - 1) / kTileN; }

bool gemm_uses_ki(GemmRole role, int M, int N) {
  return (role == GemmRole::kQkv || role == GemmRole::kO || role == GemmRole::kDown) && M <= 32 && N % 16 == 0;
}

void gemm_ki_plan(int N, int K, int* nb, int* ksplit) {
  const int S = K / 32, blocks = N / 16;
  // at least 4 steps per wave in a split; long K (the down projection) in 8
  // splits, which with 8 blocks per work-group halves the activation reads
  // per weight byte and keeps the grid at one round
  const int ks = S >= 256 ? 8 : std::max(1, std::min(4, S / 32));
  *ksplit = ks;
  *nb = std::max(1, std::min(kWaves, (blocks * ks + 255) / 256));
}

int gemm_rows_per_group(int M) {
  return M > 96 ? 128 : M > 64 ? 96 : M > 48 ? 64 : M > 32 ? 48 : M > 16 ? 32 : 16;
}

int gemm_padded_rows(int M) {
  const int g = gemm_rows_per_group(M);
  return (M + g - 1) / g * g;
}

bool gemm_is_prefill(bool bf16, int M) { return bf16 && M > kPrefillMinRows; }

void launch_gemm(bool bf16, GemmRole role, const GemmArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (role != GemmRole::kHead && gemm_is_prefill(bf16, a.M)) {
    // many rows: the compute-bound tile kernel (one partial, ksplit 1; the
    // gate/up projection writes h itself)
    const int nt = role == GemmRole::kQkv ? kQkvTerms : 2;
    launch_prefill(a, nt, role == GemmRole::kGateUp, s, e0, e1);
    return;
  }
  if (bf16 && a.nb > 0 && gemm_uses_ki(role, a.M, a.N)) {
    if (role == GemmRole::kQkv)
      launch_ki_part<kQkvTerms>(a, s, e0, e1);
    else
      launch_ki_part<2>(a, s, e0, e1);
    return;
  }
  if (bf16)
    launch_role<uint16_t>(role, a, s, e0, e1);
  else
    launch_role<float>(role, a, s, e0, e1);
}

void launch_gemm_bf16(const GemmArgs& a, hipStream_t s) { launch_prefill(a, 1, false, s, nullptr, nullptr); }

void launch_lm_finalize(const LmRow* lm, const float* lm_part, int n_lm, int ntiles, float inv_T, int32_t* row_argmax,
                        float* row_max, float* row_sumexp, float* row_gap, hipStream_t s) {
  hipLaunchKernelGGL(lm_finalize_kernel, dim3(n_lm), dim3(256), 0, s, lm, lm_part, n_lm, ntiles, inv_T, row_argmax,
                     row_max, row_sumexp, row_gap);
}

}  // namespace via
