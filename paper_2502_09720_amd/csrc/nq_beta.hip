// Choosing the beta set (App. F of the NestQuant paper): the per-vector statistics and the
// dynamic program of Alg. 6.
//
//   beta_stats_kernel: one thread per (sample vector p, candidate beta i).  The lattice
//     input is y = fl32(v * fl32(1 / beta_i)); P = Q_E8(y) (Alg. 5, the encoder's tie
//     rules); the code of P is decoded with the chosen decoder (Alg. 2) to X2, overload is
//     X2 != P (Sec. 4.1), and mse = sum over l = 0..7, in that order, of
//     (fl64(beta_i X2_l) / 2 - v_l)^2 in fp64 (no contraction).
//   beta_cost_kernel: cost[s][i] = sum over p, in index order, of mse[p][i] over the vectors
//     that overload at s but not at i (s = 0 is a virtual beta at which every vector
//     overloads).  One wave per i, lane s; each lane adds its terms one at a time in vector
//     order, so the sums are those of a sequential loop.  The wave also records whether any
//     vector overloads at i.
//   beta_dp_kernel: Alg. 6 in one workgroup.  dp[i][j] = min over s < i (first s on ties)
//     of dp[s][j-1] + cost[s][i], dp[0][0] = 0; the answer is the least dp[i][k] (first i)
//     over the betas at which no vector overloads, and the backtracked indices.
#include "nq_device.hpp"
#include "nq_kernels.hpp"

namespace nq {

__global__ __launch_bounds__(256) void beta_stats_kernel(const float* __restrict__ v, int64_t n,
                                                         BetaGrid g, int q, float rq,
                                                         uint32_t m2q, uint32_t mq, int decoder,
                                                         double* __restrict__ mse,
                                                         uint8_t* __restrict__ ov) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= n * g.m) return;
  const int64_t p = idx / g.m;
  const int i = (int)(idx - p * g.m);
  const f32x4 a = *reinterpret_cast<const f32x4*>(v + 8 * p);
  const f32x4 b = *reinterpret_cast<const f32x4*>(v + 8 * p + 4);
  const float x[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  const double beta = g.beta[i];
  const float c = (float)(1.0 / beta);
  float y[8];
#pragma unroll
  for (int l = 0; l < 8; ++l) y[l] = x[l] * c;
  int P[8];
  nearest_e8(y, P);
  const uint32_t w = encode_codes(P, q, rq, mq);
  uint32_t X2p[4];
  if (decoder) {
    decode_word_pk<true>(w, q, m2q, X2p);
  } else {
    decode_word_pk<false>(w, q, m2q, X2p);
  }
  bool over = false;
  double err = 0.0;
#pragma unroll
  for (int l = 0; l < 8; ++l) {
    const int x2 = (int)(short)((X2p[l >> 1] >> (16 * (l & 1))) & 0xFFFFu);
    over |= x2 != P[l];
    const double d = beta * (double)x2 / 2.0 - (double)x[l];
    err = err + d * d;
  }
  mse[idx] = err;
  ov[idx] = over ? 1 : 0;
}

// cost[s * (m + 1) + i] for 0 <= s < i <= m, and any[i] = some vector overloads at beta i.
// Wave i - 1 handles column i; lane s < i accumulates cost[s][i].
__global__ __launch_bounds__(64) void beta_cost_kernel(const double* __restrict__ mse,
                                                       const uint8_t* __restrict__ ov,
                                                       int64_t n, int m,
                                                       double* __restrict__ cost,
                                                       uint8_t* __restrict__ any) {
  const int i = blockIdx.x + 1;
  const int s = threadIdx.x;
  const bool live = s < i;
  double acc = 0.0;
  uint32_t seen = 0u;
  constexpr int U = 8;
  int64_t p = 0;
  for (; p + U <= n; p += U) {
    double w[U];
    uint32_t oi[U], os[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t row = (p + u) * m;
      w[u] = mse[row + i - 1];
      oi[u] = ov[row + i - 1];
      os[u] = (live && s > 0) ? ov[row + s - 1] : 1u;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (os[u] && !oi[u]) acc = acc + w[u];
      seen |= oi[u];
    }
  }
  for (; p < n; ++p) {
    const int64_t row = p * m;
    const double w = mse[row + i - 1];
    const uint32_t oi = ov[row + i - 1];
    const uint32_t os = (live && s > 0) ? ov[row + s - 1] : 1u;
    if (os && !oi) acc = acc + w;
    seen |= oi;
  }
  if (live) cost[s * (m + 1) + i] = acc;
  if (s == 0) any[i] = seen ? 1 : 0;
}

constexpr int kDpMax = 64;

__global__ __launch_bounds__(64) void beta_dp_kernel(const double* __restrict__ cost,
                                                     const uint8_t* __restrict__ any, int m,
                                                     int k, int32_t* __restrict__ chosen,
                                                     double* __restrict__ loss) {
  __shared__ double dp[kDpMax + 1][kDpMax + 1];
  __shared__ int frm[kDpMax + 1][kDpMax + 1];
  const int tid = threadIdx.x;
  for (int e = tid; e < (m + 1) * (k + 1); e += 64) {
    const int i = e / (k + 1), j = e % (k + 1);
    dp[i][j] = (i == 0 && j == 0) ? 0.0 : INFINITY;
    frm[i][j] = -1;
  }
  __syncthreads();
  for (int j = 1; j <= k; ++j) {
    // dp[i][j] reads only dp[.][j - 1]: every i of this j in parallel (thread i - 1)
    const int i = tid + 1;
    if (i <= m) {
      double best = INFINITY;
      int arg = -1;
      for (int s = 0; s < i; ++s) {
        const double prev = dp[s][j - 1];
        if (prev == INFINITY) continue;
        const double cand = prev + cost[s * (m + 1) + i];
        if (best > cand) {
          best = cand;
          arg = s;
        }
      }
      dp[i][j] = best;
      frm[i][j] = arg;
    }
    __syncthreads();
  }
  if (tid == 0) {
    double best = INFINITY;
    int pos = -1;
    for (int i = 1; i <= m; ++i)
      if (!any[i] && dp[i][k] < best) {
        best = dp[i][k];
        pos = i;
      }
    if (pos < 0) {
      for (int j = 0; j < k; ++j) chosen[j] = -1;
      *loss = INFINITY;
    } else {
      *loss = best;
      for (int j = k; j >= 1; --j) {   // indices come out largest first
        chosen[j - 1] = pos - 1;
        pos = frm[pos][j];
      }
    }
  }
}

hipError_t launch_beta_stats(const float* v, int64_t n, const BetaGrid& g, int q, int decoder,
                             double* mse, uint8_t* ov, hipStream_t st) {
  const int64_t total = n * g.m;
  const int64_t grid = (total + 255) / 256;
  hipLaunchKernelGGL(beta_stats_kernel, dim3((unsigned)grid), dim3(256), 0, st, v, n, g, q,
                     (float)(1.0 / q), magic_2q(q), magic_q(q), decoder, mse, ov);
  return hipGetLastError();
}

size_t beta_dp_workspace(int m) { return (size_t)(m + 1) * (m + 1) * 8 + 256; }

hipError_t launch_beta_dp(const double* mse, const uint8_t* ov, int64_t n, int m, int k,
                          int32_t* chosen, double* loss, void* ws, hipStream_t st) {
  double* cost = reinterpret_cast<double*>(ws);
  uint8_t* any = reinterpret_cast<uint8_t*>(cost + (m + 1) * (m + 1));
  hipLaunchKernelGGL(beta_cost_kernel, dim3((unsigned)m), dim3(64), 0, st, mse, ov, n, m, cost,
                     any);
  hipLaunchKernelGGL(beta_dp_kernel, dim3(1), dim3(64), 0, st, cost, any, m, k, chosen, loss);
  return hipGetLastError();
}

}  // namespace nq
