// Choosing the beta set (App. F of the NestQuant paper): the per-vector statistics and the
// dynamic program of Alg. 6.
//
//   beta_stats_kernel: one thread per (sample vector p, candidate beta i).  The lattice
//     input is y = fl32(v * fl32(1 / beta_i)); P = Q_E8(y) (Alg. 5, the encoder's tie
//     rules); the code of P is decoded with the chosen decoder (Alg. 2) to X2, overload is
//     X2 != P (Sec. 4.1), and mse = sum over l = 0..7, in that order, of
//     (fl64(beta_i X2_l) / 2 - v_l)^2 in fp64 (no contraction).
//   beta_cost_*_kernel: cost[s][i] = sum over p of mse[p][i] over the vectors that overload
//     at s but not at i (s = 0 is a virtual beta at which every vector overloads), and the
//     number of vectors that overload at i, each summed in a fixed 64-ary tree over the
//     vectors (groups of 64 consecutive terms in order, level by level), so that the sums
//     are reproducible and the work spreads over the chip.
//   beta_dp_kernel: Alg. 6 in one workgroup.  dp[i][j] = min over s < i (first s on ties)
//     of dp[s][j-1] + cost[s][i], dp[0][0] = 0; the answer is the least dp[i][k] (first i)
//     over the betas at which no vector overloads, and the backtracked indices.
#include <algorithm>

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
  // the byte decoder: X2_l + 128 in byte l of xs (every X2 of a code word fits a byte)
  uint32_t xs[2];
  if (decoder) {
    decode_word_b8<true>(w, q, m2q, xs[0], xs[1]);
  } else {
    decode_word_b8<false>(w, q, m2q, xs[0], xs[1]);
  }
  bool over = false;
  double err = 0.0;
#pragma unroll
  for (int l = 0; l < 8; ++l) {
    const int x2 = (int)((xs[l >> 2] >> (8 * (l & 3))) & 0xFFu) - 128;
    over |= x2 != P[l];
    const double d = beta * (double)x2 / 2.0 - (double)x[l];
    err = err + d * d;
  }
  mse[idx] = err;
  ov[idx] = over ? 1 : 0;
}

// The DP's transition costs, one entry per pair 0 <= s < i <= m at index i (i - 1) / 2 + s
// (P = m (m + 1) / 2 of them), followed by m overload counts (entry P + i - 1: how many
// samples overload at beta i).  Each entry is a sum over the samples in a fixed 64-ary tree:
// consecutive groups of 64 terms are added in order, then groups of 64 group sums, and so
// on; a short last group adds only the terms it has.
constexpr int kFan = kBetaFan;

__device__ __forceinline__ void pair_of(int idx, int P, int& s, int& i) {
  if (idx >= P) {               // overload count of beta idx - P + 1
    s = -1;
    i = idx - P + 1;
    return;
  }
  int r = (int)((1.0f + sqrtf(1.0f + 8.0f * (float)idx)) * 0.5f);
  while (r * (r - 1) / 2 > idx) --r;
  while ((r + 1) * r / 2 <= idx) ++r;
  i = r;
  s = idx - r * (r - 1) / 2;
}

// First two tree levels: workgroup x sums samples [4096 x, 4096 x + 4096) for 256 entries
// (grid y picks which): each group of 64 samples is staged in LDS (two buffers; the next
// group's rows are loaded into registers while the current one is summed), summed per entry
// in sample order, and the 64 group sums are added in order.
__global__ __launch_bounds__(256) void beta_cost_leaf_kernel(const double* __restrict__ mse,
                                                            const uint8_t* __restrict__ ov,
                                                            int64_t n, int m, int Q,
                                                            double* __restrict__ out) {
  constexpr int PER = kFan * 64 / 256;       // staged elements per thread (64 rows, m <= 64)
  __shared__ double wsh[2][kFan * 64];
  __shared__ uint8_t osh[2][kFan * 64];
  const int P = m * (m + 1) / 2;
  const int idx = blockIdx.y * 256 + threadIdx.x;
  int s = 0, i = 1;
  if (idx < Q) pair_of(idx, P, s, i);
  const int cs = s > 0 ? s - 1 : i - 1;      // column of the smaller beta (s = 0: none)
  const int64_t first = (int64_t)blockIdx.x * kFan * kFan;
  const int groups = (int)(n - first < (int64_t)kFan * kFan ? (n - first + kFan - 1) / kFan : kFan);
  // buffer resources over this workgroup's samples (at most 4096 m entries, 32-bit offsets);
  // offsets past a group's rows carry the top bit, outside every range, and read 0
  constexpr uint32_t OOB = 0x80000000u;
  const int64_t nsamp = n - first < (int64_t)kFan * kFan ? n - first : (int64_t)kFan * kFan;
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(mse + first * m), (short)0, (int)(nsamp * m * 8), 0x00020000);
  const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(ov + first * m), (short)0, (int)(nsamp * m), 0x00020000);
  double wr[PER];
  uint32_t orr[PER];
  auto fetch = [&](int b) {
    const int base = b * kFan * m;
    const int len = (int)(nsamp - (int64_t)b * kFan < kFan ? nsamp - (int64_t)b * kFan : kFan) * m;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = (int)threadIdx.x + 256 * u;
      const uint32_t ok = e < len ? 0u : OOB;
      const uint2 pair = __builtin_bit_cast(
          uint2, __builtin_amdgcn_raw_buffer_load_b64(rw, (uint32_t)(base + e) * 8u | ok, 0, 0));
      wr[u] = __builtin_bit_cast(double, pair);
      orr[u] = __builtin_amdgcn_raw_buffer_load_b8(ro, (uint32_t)(base + e) | ok, 0, 0);
    }
  };
  double node = 0.0;
  fetch(0);
  for (int b = 0; b < groups; ++b) {
    const int buf = b & 1;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      wsh[buf][threadIdx.x + 256 * u] = wr[u];
      osh[buf][threadIdx.x + 256 * u] = (uint8_t)orr[u];
    }
    __syncthreads();
    if (b + 1 < groups) fetch(b + 1);      // in flight while this group is summed
    const int64_t p0 = first + (int64_t)b * kFan;
    const int rows = (int)(n - p0 < kFan ? n - p0 : kFan);
    if (idx < Q) {
      // terms of the samples this entry skips are +0, which leaves every partial sum as it
      // is; the LDS reads of eight samples are issued before their additions
      const double* wb = wsh[buf];
      const uint8_t* ob = osh[buf];
      double leaf = 0.0;
      for (int j0 = 0; j0 < rows; j0 += 8) {
        double t[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          // every value is read unconditionally and the term selected by a multiply by 0 or
          // 1 (exact: errors are finite and >= 0), so that no read sits behind a branch
          const int j = j0 + u < rows ? j0 + u : rows - 1;
          const uint32_t oi = ob[j * m + i - 1];
          const uint32_t os = (uint32_t)ob[j * m + cs] | (uint32_t)(s == 0);
          const double wv = wb[j * m + i - 1];
          const uint32_t keep = (j0 + u < rows) ? ((s < 0 ? oi : (os & (oi ^ 1u))) & 1u) : 0u;
          t[u] = (s < 0 ? 1.0 : wv) * (double)keep;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) leaf = leaf + t[u];
      }
      node = node + leaf;
    }
  }
  if (idx < Q) out[(int64_t)blockIdx.x * Q + idx] = node;
}

// Higher levels: output node x is the in-order sum of input nodes 64 x .. 64 x + 63.
__global__ __launch_bounds__(256) void beta_cost_node_kernel(const double* __restrict__ in,
                                                            int64_t cnt, int Q,
                                                            double* __restrict__ out) {
  const int idx = blockIdx.y * 256 + threadIdx.x;
  if (idx >= Q) return;
  const int64_t c0 = (int64_t)blockIdx.x * kFan;
  const int kids = (int)(cnt - c0 < kFan ? cnt - c0 : kFan);
  double acc = 0.0;
  for (int c = 0; c < kids; ++c) acc = acc + in[(c0 + c) * Q + idx];
  out[(int64_t)blockIdx.x * Q + idx] = acc;
}

__global__ __launch_bounds__(256) void beta_cost_zero_kernel(int Q, double* __restrict__ out) {
  for (int e = threadIdx.x; e < Q; e += 256) out[e] = 0.0;
}

constexpr int kDpMax = 64;

__global__ __launch_bounds__(64) void beta_dp_kernel(const double* __restrict__ cost, int m,
                                                     int k, int32_t* __restrict__ chosen,
                                                     double* __restrict__ loss) {
  const int P = m * (m + 1) / 2;   // cost of (s, i) at i (i - 1) / 2 + s; counts after
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
        const double cand = prev + cost[i * (i - 1) / 2 + s];
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
      if (cost[P + i - 1] == 0.0 && dp[i][k] < best) {
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

hipError_t launch_beta_dp(const double* mse, const uint8_t* ov, int64_t n, int m, int k,
                          int32_t* chosen, double* loss, void* ws, hipStream_t st) {
  const int Q = (int)beta_cost_entries(m);
  const unsigned qy = (unsigned)((Q + 255) / 256);
  double* buf[2] = {reinterpret_cast<double*>(ws), nullptr};
  int64_t cnt = beta_level2_nodes(n);
  buf[1] = buf[0] + std::max<int64_t>(cnt, 1) * Q;
  int cur = 0;
  if (n == 0) {
    hipLaunchKernelGGL(beta_cost_zero_kernel, dim3(1), dim3(256), 0, st, Q, buf[0]);
  } else {
    hipLaunchKernelGGL(beta_cost_leaf_kernel, dim3((unsigned)cnt, qy), dim3(256), 0, st, mse,
                       ov, n, m, Q, buf[0]);
    while (cnt > 1) {
      const int64_t next = (cnt + kFan - 1) / kFan;
      hipLaunchKernelGGL(beta_cost_node_kernel, dim3((unsigned)next, qy), dim3(256), 0, st,
                         buf[cur], cnt, Q, buf[cur ^ 1]);
      cur ^= 1;
      cnt = next;
    }
  }
  hipLaunchKernelGGL(beta_dp_kernel, dim3(1), dim3(64), 0, st, buf[cur], m, k, chosen, loss);
  return hipGetLastError();
}

}  // namespace nq
