// Draft-window attention over the paged KV cache (scaled dot-product
// attention of every fed row against the visible cache slots).
//
// Queries of one KV head are packed across the GQA group: a work item holds
// up to 32 (row, head-in-group) queries of one sequence (one MFMA column
// block), so every K/V byte a work-group streams serves all query heads that
// share it.  Work-groups are dispatched round-robin over the 8 XCDs in
// linear order and the item index is the grid's slowest, so when splits x
// KV heads is a multiple of 8 the items of a sequence that share a (KV head,
// split) run on one XCD and their repeated K/V reads can hit its L2.  The keys of a sequence are split into spans of `span` keys (a
// multiple of 32 the host picks so that the whole launch has about 192
// work-groups, or more when that would take spans well past 4096 keys); a work-group streams its span and writes
// one (max, sum, output) partial per query, and a combine kernel merges the
// partials of a query in split order.  When every item has one split (long
// forwards: prefills), the work-group applies the combine's arithmetic to its
// one partial and writes the output itself, and no combine runs.  Visibility of slot p for row r:
// p < vis_len[r], or p is a window slot whose bit is set in the row's tree
// mask.
//
// bf16 path: four waves per work-group; wave w takes the 32-key blocks
// w, w+4, ... of the span and streams them with the loads of its next block
// in flight while the current one is multiplied (online softmax per wave,
// the four waves merged in a fixed order at the end).  Both products run on
// v_mfma_f32_32x32x16_bf16:
//   S^T = K Q^T: A = 32 keys x 16 dims (keys as rows, so each lane owns one
//     query column and 16 keys; the row statistics of a query need only the
//     lane and its partner l^32); B = Q^T staged in LDS;
//   O^T += V^T P^T: B = P^T straight from the S^T registers, A = V^T read
//     from the transposed V pages (16 contiguous bytes per lane).
//   A-row m of the K tile holds key pi(m) = (m/16)*16 + ((m/4)%2)*8 +
//     ((m/8)%2)*4 + m%4 of the block, which makes register r of lane l hold
//     key (r/8)*16 + (l/32)*8 + r%8: the B-operand slice of the PV step r/8.
//   Q (fp32) and P are fed as bf16 hi + lo terms (two products each), so
//     both keep ~16 significant bits; K and V are the cache's bf16 values,
//     exact operands.  Maxima are kept in log2 units.
#include <algorithm>

#include "kernels.h"

namespace via {

namespace {

__device__ __forceinline__ bool key_visible(int key, int kv_len, const RowInfo& ri, int win_base) {
  if (key >= kv_len) return false;
  if (key < ri.vis_len) return true;
  int o = key - win_base;
  return o >= 0 && o < 64 && ((ri.mask >> o) & 1ull);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f32x16 mfma32(uint4 a, uint4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

// K and V operands of one 32-key block (block b of the work-group's span).
template <int HD>
struct KvRegs {
  uint4 k[HD / 16];     // S-step ks: key pi(l%32), dims ks*16 + (l/32)*8 .. +7
  uint4 v[HD / 32][2];  // d tile dt, PV step t: dim dt*32 + l%32, keys t*16 + (l/32)*8 .. +7
};

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
// K/V are read once per forward: streamed past the caches (nontemporal)
__device__ __forceinline__ uint4 load_stream(const uint4* p) {
  const u32x4 v = __builtin_nontemporal_load((const u32x4*)p);
  return make_uint4(v[0], v[1], v[2], v[3]);
}

template <int HD>
__device__ __forceinline__ void load_block(KvRegs<HD>& r, const uint16_t* pool, const AttnArgs& a, int g,
                                           const int* spage, int b, int ql, int half) {
  const int m = ql;
  const int key = ((m >> 4) << 4) + (((m >> 2) & 1) << 3) + (((m >> 3) & 1) << 2) + (m & 3);
  const uint4* kp =
      (const uint4*)(pool + k_off(a.layer_slot, spage[2 * b + (key >> 4)], a.pool_blocks, a.KVH, HD, g, key & 15, half * 8));
#pragma unroll
  for (int ks = 0; ks < HD / 16; ++ks) r.k[ks] = load_stream(kp + ks * 2 * kBlock);  // dim group 2*ks + half
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const uint4* vp =
        (const uint4*)(pool + v_off(a.layer_slot, spage[2 * b + t], a.pool_blocks, a.KVH, HD, g, half * 8, ql));
#pragma unroll
    for (int dt = 0; dt < HD / 32; ++dt) r.v[dt][t] = load_stream(vp + dt * 32 * kBlock / 8);
  }
}

// The lane's query (lane % 32 of the work item's 32).
struct QueryState {
  bool valid;
  int row, head, vis;
  uint64_t mask;
};

template <int HD>
__device__ __forceinline__ void compute_block(KvRegs<HD>& r, int kb, const AttnItem& it, const QueryState& qs,
                                              const uint4 (*sq)[HD / 16][64], int lane, int half, float sl2,
                                              f32x16 (&o)[HD / 32], float& mrun, float& lrun) {
  constexpr int KS = HD / 16, DT = HD / 32;
  if (kb + 32 > it.kv_len) {  // zero V of keys past the written slots (their page rows may hold anything)
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int valid8 = it.kv_len - (kb + t * 16 + half * 8);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        uint32_t w[4];
        __builtin_memcpy(w, &r.v[dt][t], 16);
#pragma unroll
        for (int q = 0; q < 4; ++q)
          w[q] &= (2 * q + 1 < valid8 ? 0xFFFF0000u : 0u) | (2 * q < valid8 ? 0xFFFFu : 0u);
        __builtin_memcpy(&r.v[dt][t], w, 16);
      }
    }
  }
  // Q is re-read from LDS for every block rather than held in registers
  // (which the register budget of two work-groups per compute unit does not
  // allow): an opaque zero keeps the compiler from hoisting the reads
  int zero;
  asm volatile("v_mov_b32 %0, 0" : "=v"(zero));
  {
    f32x16 s;
#pragma unroll
    for (int i = 0; i < 16; ++i) s[i] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      s = mfma32(r.k[ks], sq[0][ks][lane + zero], s);
      s = mfma32(r.k[ks], sq[1][ks][lane + zero], s);
    }
    // masked scores become -inf; the max is taken on unscaled scores (scale > 0)
    const bool full = __all(!qs.valid || (kb + 32 <= qs.vis && kb + 32 <= it.kv_len));
    if (!full) {
      RowInfo ri;
      ri.vis_len = qs.vis;
      ri.mask = qs.mask;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = kb + (i >> 3) * 16 + half * 8 + (i & 7);
        if (!(qs.valid && key_visible(key, it.kv_len, ri, it.win_base))) s[i] = -INFINITY;
      }
    }
    float bm = s[0];
#pragma unroll
    for (int i = 1; i < 16; ++i) bm = fmaxf(bm, s[i]);
    bm = fmaxf(bm, __shfl_xor(bm, 32, 64));
    const float mn = fmaxf(mrun, bm * sl2);  // log2 units; -inf stays -inf
    if (__any(mn > mrun)) {
      const float alpha = mn == mrun ? 1.f : __builtin_amdgcn_exp2f(mrun - mn);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) o[dt] *= alpha;
      lrun *= alpha;
      mrun = mn;
    }
    const float neg_m = mrun == -INFINITY ? 0.f : -mrun;  // nothing visible yet: every p is 0
    // P = 2^(s * scale * log2(e) - max) as bf16 hi (truncated) + lo (rounded) terms
    uint4 ph[2], pl[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      uint32_t hw[4], lw[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(s[t * 8 + 2 * e], sl2, neg_m));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(s[t * 8 + 2 * e + 1], sl2, neg_m));
        lrun += p0;
        lrun += p1;
        hw[e] = __builtin_amdgcn_perm(__float_as_uint(p1), __float_as_uint(p0), 0x07060302u);
        const float r0 = p0 - __uint_as_float(__float_as_uint(p0) & 0xFFFF0000u);
        const float r1 = p1 - __uint_as_float(__float_as_uint(p1) & 0xFFFF0000u);
        const bf16x2 lo = {(__bf16)r0, (__bf16)r1};
        lw[e] = __builtin_bit_cast(uint32_t, lo);
      }
      ph[t] = make_uint4(hw[0], hw[1], hw[2], hw[3]);
      pl[t] = make_uint4(lw[0], lw[1], lw[2], lw[3]);
    }
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        o[dt] = mfma32(r.v[dt][t], ph[t], o[dt]);
        o[dt] = mfma32(r.v[dt][t], pl[t], o[dt]);
      }
  }
}

template <int HD>
__global__ __launch_bounds__(256, 2) void attn_split_kernel(AttnArgs a) {
  constexpr int KS = HD / 16, DT = HD / 32;
  const AttnItem it = a.items[blockIdx.z];
  const int split = blockIdx.x;
  if (split >= it.n_chunks) return;
  const int g = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, ql = lane & 31, half = lane >> 5;
  const int G = a.H / a.KVH;
  const int k0 = split * a.span;
  const int k1 = min(it.kv_len, k0 + a.span);
  const int nblk = (k1 - k0 + 31) >> 5;  // 32-key blocks of the span
  const uint16_t* pool = (const uint16_t*)a.pool;

  __shared__ int spage[kAttnMaxSpan / kBlock];
  __shared__ uint4 sq[2][KS][64];  // Q hi/lo terms in the B-operand layout of S^T = K Q^T
  __shared__ float mo[2][DT * 16][64];    // wave merge: unscaled outputs, max, sum
  __shared__ float mm[2][64], ml[2][64];

  for (int t = threadIdx.x; t < 2 * nblk; t += 256) spage[t] = a.btab[it.bt + min((k0 >> 4) + t, it.n_blocks - 1)];
  constexpr int QPT = 2 * KS * 64 / 256;  // staged uint4 per thread
#pragma unroll
  for (int u = 0; u < QPT; ++u) {
    const int e = threadIdx.x + u * 256;
    const int l = e & 63, ks = (e >> 6) % KS, term = e / (64 * KS);
    const int qi = it.q0 + (l & 31);
    const int rl = qi / G;
    const bool ok = rl < it.n_rows;
    const int rw = it.row_start + (ok ? rl : 0), hh = g * G + (qi - rl * G);
    const uint16_t* src = term ? a.q_lo : (const uint16_t*)a.q_hi;
    const uint4 v = *(const uint4*)(src + ((size_t)rw * a.H + (ok ? hh : 0)) * HD + ks * 16 + (l >> 5) * 8);
    sq[term][ks][l] = ok ? v : make_uint4(0, 0, 0, 0);
  }
  QueryState qs;
  {
    const int qi = it.q0 + ql;
    const int rl = qi / G;
    qs.valid = rl < it.n_rows;
    qs.row = it.row_start + (qs.valid ? rl : 0);
    qs.head = g * G + (qi - rl * G);
    const RowInfo ri = a.rows[qs.row];
    qs.vis = ri.vis_len;
    qs.mask = ri.mask;
  }
  __syncthreads();

  const float sl2 = a.scale * 1.4426950408889634f;
  f32x16 o[DT];
  float mrun = -INFINITY, lrun = 0.f;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[dt][i] = 0.f;
  // wave w streams blocks w, w+4, ...: two register sets, the next block's
  // loads in flight while the current one is multiplied.  The load past the
  // wave's last block re-reads that block (an L2 hit) so that every load is
  // unconditional and the waits stay exact.
  const int cnt = nblk > wave ? (nblk - wave + 3) >> 2 : 0;
  if (cnt > 0) {
    auto blk = [&](int i) { return wave + 4 * min(i, cnt - 1); };
    KvRegs<HD> r0, r1;
    load_block<HD>(r0, pool, a, g, spage, blk(0), ql, half);
    for (int i = 0; i < cnt; i += 2) {
      load_block<HD>(r1, pool, a, g, spage, blk(i + 1), ql, half);
      compute_block<HD>(r0, k0 + blk(i) * 32, it, qs, sq, lane, half, sl2, o, mrun, lrun);
      if (i + 1 >= cnt) break;
      load_block<HD>(r0, pool, a, g, spage, blk(i + 2), ql, half);
      compute_block<HD>(r1, k0 + blk(i + 1) * 32, it, qs, sq, lane, half, sl2, o, mrun, lrun);
    }
  }

  // merge the four waves in a fixed order: (w0 + w2) + (w1 + w3)
  float lt = lrun + __shfl_xor(lrun, 32, 64);
  float mx = mrun;
  auto merge_from = [&](int buf) {
    const float mb = mm[buf][lane], lb = ml[buf][lane];
    const float M = fmaxf(mx, mb);
    const float ca = M == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mx - M);
    const float cb = M == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mb - M);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int i = 0; i < 16; ++i) o[dt][i] = o[dt][i] * ca + mo[buf][dt * 16 + i][lane] * cb;
    lt = lt * ca + lb * cb;
    mx = M;
  };
  auto store_to = [&](int buf) {
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int i = 0; i < 16; ++i) mo[buf][dt * 16 + i][lane] = o[dt][i];
    mm[buf][lane] = mx;
    ml[buf][lane] = lt;
  };
  if (wave >= 2) store_to(wave - 2);
  __syncthreads();
  if (wave < 2) merge_from(wave);
  __syncthreads();
  if (wave == 1) store_to(0);
  __syncthreads();
  if (wave == 0 && a.direct) {
    // one split: the combine's arithmetic for a single partial (weight
    // exp2(max - max), sum and outputs accumulated from zero, then scaled by
    // 1 / sum), written as activation fragments here.  The 8 dims of a
    // fragment group are split over lanes l and l ^ 32: lane half 0 writes
    // group 2p of each pair of groups, half 1 group 2p + 1.
    merge_from(0);
    const float w = __builtin_amdgcn_exp2f(mx - mx);
    float L = 0.f;
    L += lt * w;
    const float inv = 1.f / L;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        float v[8];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const float own0 = o[dt][8 * p + c], own1 = o[dt][8 * p + 4 + c];
          const float recv = __shfl_xor(half ? own0 : own1, 32, 64);
          v[c] = half ? recv : own0;
          v[4 + c] = half ? own1 : recv;
        }
        float O[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          O[e] = 0.f;
          O[e] += v[e] * w;
          O[e] *= inv;
        }
        if (qs.valid) put_afrag<true, 2>(a.out, qs.row, qs.head * HD + dt * 32 + (2 * p + half) * 8, O, (a.H * HD) >> 5, a.MBn);
      }
  } else if (wave == 0) {
    merge_from(0);
    if (qs.valid) {
      // O^T lane l, register i of d tile dt -> dim dt*32 + (i/4)*8 + (l/32)*4 + i%4
      float* po = a.part_o + (((size_t)split * a.M + qs.row) * a.H + qs.head) * HD;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int i4 = 0; i4 < 4; ++i4)
          *(float4*)(po + dt * 32 + i4 * 8 + half * 4) =
              make_float4(o[dt][4 * i4], o[dt][4 * i4 + 1], o[dt][4 * i4 + 2], o[dt][4 * i4 + 3]);
      if (half == 0) {
        float* pm = a.part_ml + (((size_t)split * a.M + qs.row) * a.H + qs.head) * 2;
        pm[0] = mx;
        pm[1] = lt;
      }
    }
  }
}

// Merge the split partials of each query in split order and write the
// normalised output as activation fragments.  Work-group: QPW queries of
// one item and KV head, HD/8 threads per query (8 dims each).
template <int HD>
__global__ __launch_bounds__(128) void attn_combine_kernel(AttnArgs a) {
  constexpr int TPQ = HD / 8, QPW = 128 / TPQ, GROUPS = kAttnQueries / QPW;
  const AttnItem it = a.items[blockIdx.x / GROUPS];
  const int g = blockIdx.y, G = a.H / a.KVH;
  const int qi = it.q0 + (blockIdx.x % GROUPS) * QPW + threadIdx.x / TPQ, d0 = (threadIdx.x % TPQ) * 8;
  const int rl = qi / G;
  if (qi - it.q0 >= kAttnQueries || rl >= it.n_rows) return;
  const int row = it.row_start + rl, head = g * G + (qi - rl * G);
  const int n = it.n_chunks;
  const size_t stride_ml = (size_t)a.M * a.H * 2, stride_o = (size_t)a.M * a.H * HD;
  const float* pml = a.part_ml + ((size_t)row * a.H + head) * 2;
  const float* po = a.part_o + ((size_t)row * a.H + head) * HD + d0;
  // the first 8 splits' outputs are loaded with the statistics (no
  // dependence between them), so the common case is one round of loads
  float4 v[8][2];
#pragma unroll
  for (int c = 0; c < 8; ++c)
    if (c < n) {
      v[c][0] = *(const float4*)(po + c * stride_o);
      v[c][1] = *(const float4*)(po + c * stride_o + 4);
    }
  float2 ml[kAttnMaxSplits];
#pragma unroll
  for (int c = 0; c < kAttnMaxSplits; ++c)
    if (c < n) ml[c] = *(const float2*)(pml + c * stride_ml);
  float M = -INFINITY;
#pragma unroll
  for (int c = 0; c < kAttnMaxSplits; ++c)
    if (c < n) M = fmaxf(M, ml[c].x);
  float L = 0.f, O[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) O[e] = 0.f;
#pragma unroll
  for (int c0 = 0; c0 < kAttnMaxSplits; c0 += 8) {
    if (c0 >= n) break;
    if (c0 > 0) {
#pragma unroll
      for (int c = 0; c < 8; ++c)
        if (c0 + c < n) {
          v[c][0] = *(const float4*)(po + (c0 + c) * stride_o);
          v[c][1] = *(const float4*)(po + (c0 + c) * stride_o + 4);
        }
    }
#pragma unroll
    for (int c = 0; c < 8; ++c)
      if (c0 + c < n) {
        const float w = __builtin_amdgcn_exp2f(ml[c0 + c].x - M);  // partial maxima are in log2 units
        L += ml[c0 + c].y * w;
        O[0] += v[c][0].x * w;
        O[1] += v[c][0].y * w;
        O[2] += v[c][0].z * w;
        O[3] += v[c][0].w * w;
        O[4] += v[c][1].x * w;
        O[5] += v[c][1].y * w;
        O[6] += v[c][1].z * w;
        O[7] += v[c][1].w * w;
      }
  }
  const float inv = 1.f / L;
#pragma unroll
  for (int e = 0; e < 8; ++e) O[e] *= inv;
  put_afrag<true, 2>(a.out, row, head * HD + d0, O, (a.H * HD) >> 5, a.MBn);
}

// fp32: one wave per (row, head); lane holds head_dim/64 dims.
template <int HD>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnArgs a) {
  constexpr int PER = HD / 64;
  const int row = blockIdx.x, head = blockIdx.y, lane = threadIdx.x;
  const RowInfo ri = a.rows[row];
  const SeqInfo si = a.seqs[ri.seq];
  const int G = a.H / a.KVH, g = head / G;
  const float* Q = (const float*)a.q_hi;
  const float* pool = (const float*)a.pool;
  float q[PER], acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    q[e] = Q[((size_t)row * a.H + head) * HD + lane * PER + e];
    acc[e] = 0.f;
  }
  float m_run = -INFINITY, l_run = 0.f;
  for (int key = 0; key < si.kv_len; ++key) {
    if (!key_visible(key, si.kv_len, ri, si.win_base)) continue;
    int blk = a.btab[si.bt + key / kBlock], t = key % kBlock;
    float dot = 0.f;
#pragma unroll
    for (int e = 0; e < PER; ++e) dot += q[e] * pool[k_off(a.layer_slot, blk, a.pool_blocks, a.KVH, HD, g, t, lane * PER + e)];
    float s = wave_sum(dot) * a.scale;
    float m_new = fmaxf(m_run, s);
    float alpha = expf(m_run - m_new), p = expf(s - m_new);
    l_run = l_run * alpha + p;
#pragma unroll
    for (int e = 0; e < PER; ++e)
      acc[e] = acc[e] * alpha + p * pool[v_off(a.layer_slot, blk, a.pool_blocks, a.KVH, HD, g, t, lane * PER + e)];
    m_run = m_new;
  }
  __shared__ float o_s[HD];
#pragma unroll
  for (int e = 0; e < PER; ++e) o_s[lane * PER + e] = acc[e] / l_run;
  __syncthreads();
  if (lane < HD / 8) {
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = o_s[lane * 8 + e];
    put_afrag<false, 1>(a.out, row, head * HD + lane * 8, v, (a.H * HD) >> 5, a.MBn);
  }
}

}  // namespace

void launch_attention(bool bf16, const AttnArgs& a, hipStream_t s) {
  if (bf16) {
    AttnArgs b = a;
    b.direct = a.max_chunks == 1;
    dim3 grid(a.max_chunks, a.KVH, a.n_items);
    if (a.hd == 128) {
      hipLaunchKernelGGL(attn_split_kernel<128>, grid, dim3(256), 0, s, b);
      if (!b.direct)
        hipLaunchKernelGGL(attn_combine_kernel<128>, dim3(a.n_items * (kAttnQueries / 8), a.KVH), dim3(128), 0, s, b);
    } else {
      hipLaunchKernelGGL(attn_split_kernel<64>, grid, dim3(256), 0, s, b);
      if (!b.direct)
        hipLaunchKernelGGL(attn_combine_kernel<64>, dim3(a.n_items * (kAttnQueries / 16), a.KVH), dim3(128), 0, s, b);
    }
  } else {
    dim3 grid(a.M, a.H);
    if (a.hd == 128)
      hipLaunchKernelGGL(attn_f32_kernel<128>, grid, dim3(64), 0, s, a);
    else
      hipLaunchKernelGGL(attn_f32_kernel<64>, grid, dim3(64), 0, s, a);
  }
}

}  // namespace via
