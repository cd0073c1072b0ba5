// Draft-window attention over the paged KV cache.
//
// Queries of one KV head are packed across the GQA group: a tile holds 32
// (row, head-in-group) queries of one sequence, so every K/V byte a
// work-group streams serves all query heads that share it.  Keys are split
// into chunks of kAttnChunk slots (one work-group each, split-KV); a
// combine kernel merges the per-chunk (max, sum, output) partials in chunk
// order.  Visibility of slot p for row r: p < vis_len[r], or p is a window
// slot whose bit is set in the row's tree mask.
//
// bf16 path (one wave per work-group, v_mfma_f32_32x32x16_bf16):
//   S^T = K Q^T: A = 32 keys x hd (keys as rows, so each lane owns one
//     query column and 16 keys: the softmax row statistics need only the
//     lane itself and its partner lane l^32);
//   O^T += V^T P^T: B = P^T straight from the S^T registers, A = V^T read
//     from the transposed V pages (16 contiguous bytes per lane);
//   A-row m of the K tile holds key pi(m) = (m/16)*16 + ((m/4)%2)*8 +
//     ((m/8)%2)*4 + m%4, which makes register r of S^T hold key
//     (r/8)*16 + (l/32)*8 + r%8: the 8-key groups the PV step consumes.
//   Q (fp32) and P are fed to the MFMA as bf16 hi + lo terms (two
//   products each), so both keep ~16 significant bits; K and V are the
//   cache's bf16 values, exact operands.
// fp32 path: one wave per (row, head), keys streamed with an online softmax.
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

template <int HD>
__global__ __launch_bounds__(64) void attn_mfma_kernel(AttnArgs a) {
  constexpr int NQ = HD / 16;   // uint4 per lane of Q / K (HD/2 bf16)
  constexpr int NDB = HD / 32;  // 32-wide d blocks of the output
  const AttnItem it = a.items[blockIdx.z];
  const int chunk = blockIdx.x;
  if (chunk >= it.n_chunks) return;
  const int g = blockIdx.y;
  const int lane = threadIdx.x, n = lane & 31, hq = lane >> 5;
  const SeqInfo si = a.seqs[it.seq];
  const int G = a.H / a.KVH;
  // this lane's query column
  const int qi = it.q0 + n;
  const int rloc = qi / G, gq = qi - rloc * G;
  const bool qvalid = rloc < si.n_rows;
  const int row = si.row_start + (qvalid ? rloc : 0);
  const int head = g * G + gq;
  const RowInfo ri = a.rows[row];
  const uint16_t* pool = (const uint16_t*)a.pool;

  // Q (fp32) as bf16 hi + lo terms, in the B-operand layout of S^T = K Q^T
  uint4 qh[NQ], ql[NQ];
  {
    const float4* qp = (const float4*)(a.q + ((size_t)row * a.H + head) * HD + hq * (HD / 2));
#pragma unroll
    for (int i = 0; i < NQ; ++i) {
      float4 u = qp[2 * i], w = qp[2 * i + 1];  // unconditional: row is a valid row of this sequence
      float f[8] = {u.x, u.y, u.z, u.w, w.x, w.y, w.z, w.w};
      uint16_t hi[8], lo[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float v = qvalid ? f[e] : 0.f;
        hi[e] = (uint16_t)(__float_as_uint(v) >> 16);
        lo[e] = f2bf(v - bf2f(hi[e]));
      }
      __builtin_memcpy(&qh[i], hi, 16);
      __builtin_memcpy(&ql[i], lo, 16);
    }
  }
  // key pi(m) loaded by this lane as an A row of the K tile
  const int km = ((n >> 4) << 4) + (((n >> 2) & 1) << 3) + (((n >> 3) & 1) << 2) + (n & 3);

  float m_run = -INFINITY, l_run = 0.f;
  f32x16 o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;

  const int k_beg = chunk * kAttnChunk;
  const int k_end = min(si.kv_len, k_beg + kAttnChunk);
  const int last_blk = si.n_blocks - 1;
  for (int kb = k_beg; kb < k_end; kb += 32) {
    // ---- S^T block: 32 keys x 32 queries
    const int key_m = kb + km;
    int pg = min(key_m / kBlock, last_blk);
    int blk = a.btab[si.bt + pg];
    const uint4* kp = (const uint4*)(pool + k_off(a.layer_slot, blk, a.pool_blocks, a.KVH, HD, g, key_m % kBlock, hq * (HD / 2)));
    uint4 kv[NQ];
#pragma unroll
    for (int i = 0; i < NQ; ++i) kv[i] = kp[i];
    // V^T operands for the two 16-key halves (pages kb/16 and kb/16 + 1)
    uint4 vv[2][NDB];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      int kh = kb + st * 16;
      int vpg = min(kh / kBlock, last_blk);
      int vblk = a.btab[si.bt + vpg];
      bool in = (kh + hq * 8) < si.kv_len;
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const uint4* vp = (const uint4*)(pool + v_off(a.layer_slot, vblk, a.pool_blocks, a.KVH, HD, g, hq * 8, db * 32 + n));
        uint4 v = *vp;  // page index is clamped to the table: always a valid address
        if (!in) v = make_uint4(0, 0, 0, 0);
        // zero keys past the written slots (their page rows may hold anything)
        int valid8 = si.kv_len - (kh + hq * 8);
        if (in && valid8 < 8) {
          uint16_t e[8];
          __builtin_memcpy(e, &v, 16);
#pragma unroll
          for (int q = 0; q < 8; ++q)
            if (q >= valid8) e[q] = 0;
          __builtin_memcpy(&v, e, 16);
        }
        vv[st][db] = v;
      }
    }
    f32x16 s;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = 0.f;
#pragma unroll
    for (int i = 0; i < NQ; ++i) {
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kv[i]), as_bf16x8(qh[i]), s, 0, 0, 0);
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kv[i]), as_bf16x8(ql[i]), s, 0, 0, 0);
    }
    // ---- online softmax for this lane's query
    float sv[16];
    float bmax = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      int key = kb + ((r >> 3) << 4) + hq * 8 + (r & 7);
      bool vis = qvalid && key_visible(key, si.kv_len, ri, si.win_base);
      sv[r] = vis ? s[r] * a.scale : -INFINITY;
      bmax = fmaxf(bmax, sv[r]);
    }
    bmax = fmaxf(bmax, __shfl_xor(bmax, 32, 64));
    const float m_new = fmaxf(m_run, bmax);
    float alpha = 1.f, psum = 0.f;
    float p[16];
    if (m_new == -INFINITY) {
#pragma unroll
      for (int r = 0; r < 16; ++r) p[r] = 0.f;
    } else {
      alpha = expf(m_run - m_new);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        p[r] = expf(sv[r] - m_new);
        psum += p[r];
      }
    }
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
    // ---- O^T += V^T P^T, P as bf16 hi + lo
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      uint16_t hi[8], lo[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float pv = p[st * 8 + e];
        hi[e] = f2bf(pv);
        lo[e] = f2bf(pv - bf2f(hi[e]));
      }
      uint4 hv, lv;
      __builtin_memcpy(&hv, hi, 16);
      __builtin_memcpy(&lv, lo, 16);
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vv[st][db]), as_bf16x8(hv), o[db], 0, 0, 0);
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vv[st][db]), as_bf16x8(lv), o[db], 0, 0, 0);
      }
    }
  }
  if (!qvalid) return;
  // partials: O^T lane (query n), register r -> d = db*32 + (r/4)*8 + hq*4 + r%4
  float* po = a.part_o + (((size_t)chunk * a.M + row) * a.H + head) * HD;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) po[db * 32 + (r >> 2) * 8 + hq * 4 + (r & 3)] = o[db][r];
  if (hq == 0) {
    float* pm = a.part_ml + (((size_t)chunk * a.M + row) * a.H + head) * 2;
    pm[0] = m_run;
    pm[1] = l_run;
  }
}

__global__ __launch_bounds__(128) void attn_combine_kernel(AttnArgs a) {
  __shared__ float o_s[128];
  const int row = blockIdx.x, head = blockIdx.y, d = threadIdx.x;
  const RowInfo ri = a.rows[row];
  const SeqInfo si = a.seqs[ri.seq];
  const int nch = (si.kv_len + kAttnChunk - 1) / kAttnChunk;
  float M = -INFINITY;
  for (int c = 0; c < nch; ++c) M = fmaxf(M, a.part_ml[(((size_t)c * a.M + row) * a.H + head) * 2]);
  float L = 0.f, O = 0.f;
  for (int c = 0; c < nch; ++c) {
    const float* pm = a.part_ml + (((size_t)c * a.M + row) * a.H + head) * 2;
    float w = expf(pm[0] - M);
    L += pm[1] * w;
    if (d < a.hd) O += a.part_o[(((size_t)c * a.M + row) * a.H + head) * a.hd + d] * w;
  }
  if (d < a.hd) o_s[d] = O / L;
  __syncthreads();
  if (d < a.hd / 8) {
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = o_s[d * 8 + e];
    put_afrag<true, 2>(a.out, row, head * a.hd + d * 8, v, (a.H * a.hd) >> 5, a.MBn);
  }
}

// fp32: one wave per (row, head); lane holds head_dim/64 dims.
template <int HD>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnArgs a) {
  constexpr int PER = HD / 64;
  const int row = blockIdx.x, head = blockIdx.y, lane = threadIdx.x;
  const RowInfo ri = a.rows[row];
  const SeqInfo si = a.seqs[ri.seq];
  const int G = a.H / a.KVH, g = head / G;
  const float* Q = a.q;
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
    dim3 grid(a.max_chunks, a.KVH, a.n_items);
    if (a.hd == 128)
      hipLaunchKernelGGL(attn_mfma_kernel<128>, grid, dim3(64), 0, s, a);
    else
      hipLaunchKernelGGL(attn_mfma_kernel<64>, grid, dim3(64), 0, s, a);
    hipLaunchKernelGGL(attn_combine_kernel, dim3(a.M, a.H), dim3(128), 0, s, a);
  } else {
    dim3 grid(a.M, a.H);
    if (a.hd == 128)
      hipLaunchKernelGGL(attn_f32_kernel<128>, grid, dim3(64), 0, s, a);
    else
      hipLaunchKernelGGL(attn_f32_kernel<64>, grid, dim3(64), 0, s, a);
  }
}

}  // namespace via
