// Routing-mask cost of DIMR: the KL-style verification cost R^KL(q || q'_z)
// of Sec. 3 (Eq. 11, ReLU surrogate) for every row of a pair of logit
// matrices, q = the full verifier, p = q'_z the routed slim verifier.  With
// l = log softmax(logits / T):
//   R = sum_v p(v) ReLU(log(1-alpha) + l_p(v) - l_q(v))
//     + sum_v q(v) ReLU(log(beta)    + l_p(v) - l_q(v)).
// One 1024-thread work-group per row streams both rows twice (16 loads of
// each matrix in flight per thread): an online (max, sum of exponentials)
// pass for the two log-partition functions, then the cost pass.  Partial sums are combined in a fixed order (fp64), so the result is
// reproducible.
#include "kernels.h"

namespace via {

namespace {

constexpr int kDimrThreads = 1024;
// ids per thread per round: all their loads are issued before any use, so a
// thread keeps kDimrUnroll loads of each matrix in flight
constexpr int kDimrUnroll = 16;

__device__ __forceinline__ void online_add(float& m, float& s, float z) {
  if (z > m) {
    s = s * expf(m - z) + 1.0f;
    m = z;
  } else {
    s += expf(z - m);
  }
}

__device__ __forceinline__ void online_merge(float& m, float& s, float m2, float s2) {
  if (m2 == -INFINITY) return;
  if (m == -INFINITY) {
    m = m2;
    s = s2;
    return;
  }
  const float M = fmaxf(m, m2);
  s = s * expf(m - M) + s2 * expf(m2 - M);
  m = M;
}

__global__ __launch_bounds__(kDimrThreads) void dimr_cost_kernel(DimrArgs a) {
  const int row = blockIdx.x, t = threadIdx.x;
  const float* q = a.q + (size_t)row * a.ld;
  const float* p = a.p + (size_t)row * a.ld;
  __shared__ float sm[4][kDimrThreads];
  __shared__ double sd[2][kDimrThreads];
  constexpr int kRound = kDimrThreads * kDimrUnroll;
  float mq = -INFINITY, sq = 0.f, mp = -INFINITY, sp = 0.f;
  for (int base = 0; base < a.vocab; base += kRound) {
    float zq[kDimrUnroll], zp[kDimrUnroll];
#pragma unroll
    for (int u = 0; u < kDimrUnroll; ++u) {
      const int v = min(base + u * kDimrThreads + t, a.vocab - 1);  // past the end: re-read, then dropped
      zq[u] = q[v];
      zp[u] = p[v];
    }
#pragma unroll
    for (int u = 0; u < kDimrUnroll; ++u)
      if (base + u * kDimrThreads + t < a.vocab) {
        online_add(mq, sq, zq[u] * a.inv_T);
        online_add(mp, sp, zp[u] * a.inv_T);
      }
  }
  sm[0][t] = mq;
  sm[1][t] = sq;
  sm[2][t] = mp;
  sm[3][t] = sp;
  __syncthreads();
  // tree merge in a fixed order
  for (int w = kDimrThreads / 2; w > 0; w >>= 1) {
    if (t < w) {
      float m1 = sm[0][t], s1 = sm[1][t];
      online_merge(m1, s1, sm[0][t + w], sm[1][t + w]);
      sm[0][t] = m1;
      sm[1][t] = s1;
      float m2 = sm[2][t], s2 = sm[3][t];
      online_merge(m2, s2, sm[2][t + w], sm[3][t + w]);
      sm[2][t] = m2;
      sm[3][t] = s2;
    }
    __syncthreads();
  }
  // log partition functions: l(v) = z(v) - lz
  const float lzq = sm[0][0] + logf(sm[1][0]);
  const float lzp = sm[2][0] + logf(sm[3][0]);
  double c1 = 0.0, c2 = 0.0;
  for (int base = 0; base < a.vocab; base += kRound) {
    float zq[kDimrUnroll], zp[kDimrUnroll];
#pragma unroll
    for (int u = 0; u < kDimrUnroll; ++u) {
      const int v = min(base + u * kDimrThreads + t, a.vocab - 1);
      zq[u] = q[v];
      zp[u] = p[v];
    }
#pragma unroll
    for (int u = 0; u < kDimrUnroll; ++u) {
      if (base + u * kDimrThreads + t >= a.vocab) continue;
      const float lq = zq[u] * a.inv_T - lzq;
      const float lp = zp[u] * a.inv_T - lzp;
      const float d = lp - lq;
      const float z1 = a.log_1m_alpha + d, z2 = a.log_beta + d;
      if (z1 > 0.f) c1 += (double)(expf(lp) * z1);
      if (z2 > 0.f) c2 += (double)(expf(lq) * z2);
    }
  }
  sd[0][t] = c1;
  sd[1][t] = c2;
  __syncthreads();
  for (int w = kDimrThreads / 2; w > 0; w >>= 1) {
    if (t < w) {
      sd[0][t] += sd[0][t + w];
      sd[1][t] += sd[1][t + w];
    }
    __syncthreads();
  }
  if (t == 0) a.cost[row] = (float)(sd[0][0] + sd[1][0]);
}

}  // namespace

void launch_dimr_cost(const DimrArgs& a, hipStream_t s) {
  if (a.rows > 0) hipLaunchKernelGGL(dimr_cost_kernel, dim3(a.rows), dim3(kDimrThreads), 0, s, a);
}

}  // namespace via
