// Draft-window attention over the paged KV cache.
//
// Queries of one KV head are packed across the GQA group: a work item holds
// up to 64 (row, head-in-group) queries of one sequence, processed as two
// sets of 32, so every K/V byte a work-group streams serves all query heads
// that share it.  Keys are split into chunks of kAttnChunk slots (one
// work-group each, split-KV); a combine kernel merges the per-chunk (max,
// sum, output) partials in chunk order.  Visibility of slot p for row r:
// p < vis_len[r], or p is a window slot whose bit is set in the row's tree
// mask.
//
// bf16 path (four waves per work-group, v_mfma_f32_32x32x16_bf16; each wave
// issues all loads of its two 32-key blocks at once and keeps them in
// registers for both query sets; per set, a wave computes the scores of
// both blocks, so its softmax max is final before any P.V product, and the
// four waves' (max, sum, output) are merged in LDS in wave order):
//   S^T = K Q^T: A = 32 keys x hd (keys as rows, so each lane owns one
//     query column and 16 keys: the softmax row statistics need only the
//     lane itself and its partner lane l^32); B = Q^T staged in LDS;
//   O^T += V^T P^T: B = P^T straight from the S^T registers, A = V^T read
//     from the transposed V pages (16 contiguous bytes per lane);
//   A-row m of the K tile holds key pi(m) = (m/16)*16 + ((m/4)%2)*8 +
//     ((m/8)%2)*4 + m%4, which makes register r of S^T hold key
//     (r/8)*16 + (l/32)*8 + r%8: the 8-key groups the PV step consumes.
//   Q (fp32) and P are fed to the MFMA as bf16 hi + lo terms (two
//   products each), so both keep ~16 significant bits; K and V are the
//   cache's bf16 values, exact operands.  Partial maxima are in log2 units.
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
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

template <int HD>
__global__ __launch_bounds__(256, 2) void attn_mfma_kernel(AttnArgs a) {
  constexpr int KS = HD / 32;                // 32-dim contraction steps of S^T
  constexpr int NDB = HD / 16;               // 16-row d blocks of O^T
  constexpr int BPW = kAttnChunk / 4 / 32;   // 32-key blocks per wave
  constexpr int QSETS = kAttnQueries / 16;   // 16-query sets per item
  const AttnItem si = a.items[blockIdx.z];
  const int chunk = blockIdx.x;
  if (chunk >= si.n_chunks) return;
  const int g = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, c = lane & 15, grp = lane >> 4;
  const int G = a.H / a.KVH;
  const int nq = min(kAttnQueries, si.n_rows * G - si.q0);
  const int nsets = (nq + 15) >> 4;  // work-group uniform
  const uint16_t* pool = (const uint16_t*)a.pool;
  const int last_blk = si.n_blocks - 1;

  // Q hi/lo terms in the B-operand layout of S^T = K Q^T, [set][term][step][lane]:
  // lane (c, grp) holds query c of the set, dims step*32 + grp*8 .. +7, so
  // each ds_read of a wave is one contiguous 1 KB block.
  __shared__ uint4 sq[QSETS][2][KS][64];
  __shared__ float4 sh_o[4][NDB][64];  // the four waves' unscaled outputs
  __shared__ float sh_m[4][64], sh_l[4][64];
  constexpr int QPT = QSETS * 2 * KS * 64 / 256;  // staged uint4 per thread
  static_assert(QPT % QSETS == 0, "a thread's staged entries of one set must share a wave-uniform set index");
  uint4 qst[QPT];
#pragma unroll
  for (int u = 0; u < QPT; ++u) {
    const int e = threadIdx.x + u * 256;
    const int l = e & 63, ks = (e >> 6) % KS, term = (e / (64 * KS)) & 1, set = e / (128 * KS);
    qst[u] = make_uint4(0, 0, 0, 0);
    if (set < nsets) {  // uniform across the work-group for a given u
      const int qi = si.q0 + set * 16 + (l & 15);
      const int rl = qi / G;
      const bool ok = rl < si.n_rows;
      const int rw = si.row_start + (ok ? rl : 0), hh = g * G + (qi - rl * G);
      const uint16_t* src = term ? a.q_lo : (const uint16_t*)a.q_hi;
      const uint4 v = *(const uint4*)(src + ((size_t)rw * a.H + hh) * HD + ks * 32 + (l >> 4) * 8);
      qst[u] = ok ? v : make_uint4(0, 0, 0, 0);
    }
  }

  // This wave's keys: two 32-key blocks.  K tile h (16 keys) of block j has
  // A-row m = key pi_h(m) = (m/4)*8 + h*4 + m%4 of the block, which makes the
  // S^T registers of lane (c, grp) hold keys grp*8 .. grp*8+7 of the block:
  // exactly the contraction slice of the P^T operand of the PV product.
  const int kw = chunk * kAttnChunk + wave * (BPW * 32);
  const int k_end = min(si.kv_len, chunk * kAttnChunk + kAttnChunk);
  const int nb = kw >= k_end ? 0 : min(BPW, (k_end - kw + 31) / 32);  // wave-uniform
  uint4 kr[BPW][2][KS], vr[BPW][NDB];
#pragma unroll
  for (int j = 0; j < BPW; ++j) {
    if (j >= nb) break;
    const int kb = kw + j * 32;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int key = kb + (c >> 2) * 8 + h * 4 + (c & 3);
      const int blk = a.btab[si.bt + min(key / kBlock, last_blk)];
      const uint4* kp = (const uint4*)(pool + k_off(a.layer_slot, blk, a.pool_blocks, a.KVH, HD, g, key % kBlock, grp * 8));
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kr[j][h][ks] = kp[ks * 4 * kBlock];  // dim group ks*4 + grp
    }
    const int vkey = kb + grp * 8;
    const int vblk = a.btab[si.bt + min(vkey / kBlock, last_blk)];
#pragma unroll
    for (int db = 0; db < NDB; ++db)
      vr[j][db] = *(const uint4*)(pool + v_off(a.layer_slot, vblk, a.pool_blocks, a.KVH, HD, g, vkey % kBlock, db * 16 + c));
  }
#pragma unroll
  for (int u = 0; u < QPT; ++u) {
    const int e = threadIdx.x + u * 256;
    sq[e / (128 * KS)][(e / (64 * KS)) & 1][(e >> 6) % KS][e & 63] = qst[u];
  }
  // zero V of keys past the written slots (their page rows may hold anything)
#pragma unroll
  for (int j = 0; j < BPW; ++j) {
    if (j >= nb) break;
    const int valid8 = si.kv_len - (kw + j * 32 + grp * 8);
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      uint32_t w[4];
      __builtin_memcpy(w, &vr[j][db], 16);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t keep = (2 * q + 1 < valid8 ? 0xFFFF0000u : 0u) | (2 * q < valid8 ? 0xFFFFu : 0u);
        w[q] &= keep;
      }
      __builtin_memcpy(&vr[j][db], w, 16);
    }
  }
  const float sl2 = a.scale * 1.4426950408889634f;

  // fully unrolled over the compile-time set count: the rolled form of this
  // loop was compiled to code that produced wrong outputs from the second
  // set on (an all-sets harness against an fp64 reference showed it)
#pragma unroll
  for (int set = 0; set < QSETS; ++set) {
    if (set >= nsets) break;
    __syncthreads();  // Q staged; the previous set's readers of sh_* are done
    const int qi = si.q0 + set * 16 + c;
    const int rloc = qi / G;
    const bool qvalid = rloc < si.n_rows;
    const int row = si.row_start + (qvalid ? rloc : 0);
    const int head = g * G + (qi - rloc * G);
    const RowInfo ri = a.rows[row];

    f32x4 sacc[BPW][2];
#pragma unroll
    for (int j = 0; j < BPW; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h) sacc[j][h] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const uint4 qh = sq[set][0][ks][lane], ql = sq[set][1][ks][lane];
#pragma unroll
      for (int j = 0; j < BPW; ++j) {
        if (j >= nb) break;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          sacc[j][h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kr[j][h][ks]), as_bf16x8(qh), sacc[j][h], 0, 0, 0);
          sacc[j][h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kr[j][h][ks]), as_bf16x8(ql), sacc[j][h], 0, 0, 0);
        }
      }
    }
    // masked scores become -inf; the max is taken on unscaled scores (scale > 0)
    float m_raw = -INFINITY;
#pragma unroll
    for (int j = 0; j < BPW; ++j) {
      if (j >= nb) break;
      const int kb = kw + j * 32;
      // a block every key of which is visible to every valid query skips the masks
      const bool full = __all(!qvalid || (kb + 32 <= ri.vis_len && kb + 32 <= si.kv_len));
      if (!full) {
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int key = kb + grp * 8 + h * 4 + r;
            if (!(qvalid && key_visible(key, si.kv_len, ri, si.win_base))) sacc[j][h][r] = -INFINITY;
          }
      }
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int r = 0; r < 4; ++r) m_raw = fmaxf(m_raw, sacc[j][h][r]);
    }
    m_raw = fmaxf(m_raw, __shfl_xor(m_raw, 16, 64));
    m_raw = fmaxf(m_raw, __shfl_xor(m_raw, 32, 64));
    const float m_run = m_raw * sl2;                        // log2 units (-inf stays -inf)
    const float neg_m = m_run == -INFINITY ? 0.f : -m_run;  // all-masked query: every p is 0

    float l_run = 0.f;
    f32x4 o[NDB];
#pragma unroll
    for (int db = 0; db < NDB; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < BPW; ++j) {
      if (j >= nb) break;
      // P = 2^(s * scale * log2(e) - max') as bf16 hi (truncated) + lo (rounded) terms
      uint32_t hw[4], lw[4];
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(sacc[j][e2 >> 1][(e2 & 1) * 2], sl2, neg_m));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(sacc[j][e2 >> 1][(e2 & 1) * 2 + 1], sl2, neg_m));
        l_run += p0;
        l_run += p1;
        hw[e2] = __builtin_amdgcn_perm(__float_as_uint(p1), __float_as_uint(p0), 0x07060302u);
        const float r0 = p0 - __uint_as_float(__float_as_uint(p0) & 0xFFFF0000u);
        const float r1 = p1 - __uint_as_float(__float_as_uint(p1) & 0xFFFF0000u);
        const bf16x2 lo = {(__bf16)r0, (__bf16)r1};
        lw[e2] = __builtin_bit_cast(uint32_t, lo);
      }
      const uint4 hv = make_uint4(hw[0], hw[1], hw[2], hw[3]);
      const uint4 lv = make_uint4(lw[0], lw[1], lw[2], lw[3]);
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vr[j][db]), as_bf16x8(hv), o[db], 0, 0, 0);
        o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vr[j][db]), as_bf16x8(lv), o[db], 0, 0, 0);
      }
    }
    l_run += __shfl_xor(l_run, 16, 64);
    l_run += __shfl_xor(l_run, 32, 64);

    // merge the four waves' (max, sum, output) in wave order; wave w
    // finishes d blocks w*NDB/4 .. of the set's partials
    sh_m[wave][lane] = m_run;
    sh_l[wave][lane] = l_run;
#pragma unroll
    for (int db = 0; db < NDB; ++db) sh_o[wave][db][lane] = make_float4(o[db][0], o[db][1], o[db][2], o[db][3]);
    __syncthreads();
    float mw[4], cw[4];
#pragma unroll
    for (int w = 0; w < 4; ++w) mw[w] = sh_m[w][lane];
    const float M = fmaxf(fmaxf(mw[0], mw[1]), fmaxf(mw[2], mw[3]));
#pragma unroll
    for (int w = 0; w < 4; ++w) cw[w] = M == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mw[w] - M);
    if (qvalid) {
      // O^T lane (c, grp), register r -> query c, d = db*16 + grp*4 + r
      float* po = a.part_o + (((size_t)chunk * a.M + row) * a.H + head) * HD;
#pragma unroll
      for (int dd = 0; dd < NDB / 4; ++dd) {
        const int db = wave * (NDB / 4) + dd;
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const float4 v = sh_o[w][db][lane];
          acc.x += v.x * cw[w];
          acc.y += v.y * cw[w];
          acc.z += v.z * cw[w];
          acc.w += v.w * cw[w];
        }
        *(float4*)(po + db * 16 + grp * 4) = acc;
      }
      if (wave == 0 && grp == 0) {
        float L = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) L += sh_l[w][lane] * cw[w];
        float* pm = a.part_ml + (((size_t)chunk * a.M + row) * a.H + head) * 2;
        pm[0] = M;
        pm[1] = L;
      }
    }
  }
}

__global__ __launch_bounds__(128) void attn_combine_kernel(AttnArgs a) {
  __shared__ float o_s[128];
  const int row = blockIdx.x, head = blockIdx.y, d = threadIdx.x;
  const RowInfo ri = a.rows[row];
  const SeqInfo si = a.seqs[ri.seq];
  const int nch = (si.kv_len + kAttnChunk - 1) / kAttnChunk;
  float M = -INFINITY;
#pragma unroll 4
  for (int c = 0; c < nch; ++c) M = fmaxf(M, a.part_ml[(((size_t)c * a.M + row) * a.H + head) * 2]);
  float L = 0.f, O = 0.f;
#pragma unroll 4
  for (int c = 0; c < nch; ++c) {
    const float* pm = a.part_ml + (((size_t)c * a.M + row) * a.H + head) * 2;
    const float w = exp2f(pm[0] - M);  // partial maxima are in log2 units
    const float ov = d < a.hd ? a.part_o[(((size_t)c * a.M + row) * a.H + head) * a.hd + d] : 0.f;
    L += pm[1] * w;
    O += ov * w;
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
    dim3 grid(a.max_chunks, a.KVH, a.n_items);
    if (a.hd == 128)
      hipLaunchKernelGGL(attn_mfma_kernel<128>, grid, dim3(256), 0, s, a);
    else
      hipLaunchKernelGGL(attn_mfma_kernel<64>, grid, dim3(256), 0, s, a);
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
