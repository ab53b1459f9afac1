// Decode-once coded matrix product for large M (prefill shapes).
//
// The product C = A_hat W_hat^T is Alg. 4 of the NestQuant paper for every pair of rows.
// With M and N in the thousands, decoding inside every output tile would repeat each
// block's decode N/BN (resp. M/BM) times, and the decode (Alg. 2 + Alg. 5) costs far more
// vector-ALU work per block than the matrix cores spend on it.  So each block is decoded
// exactly once:
//
//   1. tiles_kernel: Alg. 2 on every code word; writes t * X2 (an integer in [-128, 128],
//      exact in bf16) as 8 bf16 into a K-contiguous workspace tile, zero-padded to the GEMM
//      tile grid.  The workspace (a few tens of MB) stays in the 256 MB Infinity Cache.
//   2. gemm_kernel: bf16 MFMA GEMM (C = T_A T_W^T, fp32 accumulation) with the epilogue
//      C_ij = acc * r_Ai * r_Wj * base_A * base_W / 4.
//
// GEMM tiling (gfx950): a 256-thread workgroup owns a 256 x 128 tile of C; its four waves
// (2 x 2) own 128 x 64 each, as 4 x 2 v_mfma_f32_32x32x16_bf16 tiles (128 fp32
// accumulators per lane).  K advances 64 per stage through two LDS buffers (row stride
// 144 B: 128 B of data + 16 B pad keeps the 16-byte fragment reads conflict-free); the
// next stage's global loads are issued before the current stage's MFMAs.  Workgroups are
// mapped so that the tiles resident on one XCD (workgroup id mod 8) form a compact 4 x 8
// block of the tile grid and share their A and W rows in that XCD's L2.
#include "nq_device.hpp"
#include "nq_kernels.hpp"

namespace nq {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

namespace gemm {
constexpr int BM = 256;
constexpr int BN = 128;
constexpr int BK = 64;            // bf16 per stage
constexpr int ROWB = BK * 2 + 16;  // LDS bytes per tile row (padded)
constexpr int GROUP_M = 4;
}  // namespace gemm

// t * X2 of every block of a coded operand, as bf16, into ws[rows_p][k_p] (zero padding).
__global__ __launch_bounds__(256) void tiles_kernel(const uint32_t* __restrict__ codes,
                                                    const uint32_t* __restrict__ beta,
                                                    int64_t rows, int nb, int64_t rows_p,
                                                    int nb_p, int q, uint32_t m2q,
                                                    u32x4* __restrict__ ws) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t row = gid / nb_p;
  if (row >= rows_p) return;
  const int j = (int)(gid - row * nb_p);
  u32x4 out = {0u, 0u, 0u, 0u};
  if (row < rows && j < nb) {
    const uint32_t w = __builtin_nontemporal_load(codes + row * nb + j);
    const uint32_t bw = beta[row * ((nb + 15) >> 4) + (j >> 4)];
    const int t = (int)((bw >> (2 * (j & 15))) & 3u) + 1;
    int X2[8];
    decode_word(w, q, m2q, X2);
    uint32_t h[8];
#pragma unroll
    for (int l = 0; l < 8; ++l) h[l] = __float_as_uint((float)(t * X2[l])) >> 16;
    out = u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
  }
  ws[gid] = out;
}

__device__ __forceinline__ void tile_coords(int bid, int tm, int tn, int& pm, int& pn) {
  // XCD-contiguous numbering: workgroups bid, bid+8, ... run on one XCD
  const int total = tm * tn;
  int t = bid;
  if ((total & 7) == 0) t = (bid & 7) * (total >> 3) + (bid >> 3);
  const int width = gemm::GROUP_M * tn;
  const int g = t / width;
  const int first = g * gemm::GROUP_M;
  const int gm = min(tm - first, gemm::GROUP_M);
  const int r = t - g * width;
  pm = first + r % gm;
  pn = r / gm;
}

__global__ __launch_bounds__(256, 1) void gemm_kernel(const u32x4* __restrict__ ta,
                                                      const u32x4* __restrict__ tw, int kp,
                                                      int tm, int tn, const float* __restrict__ ra,
                                                      const float* __restrict__ rw, int64_t M,
                                                      int64_t N, float* __restrict__ c,
                                                      int64_t ldc, float scale) {
  using namespace gemm;
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  // buffer b of the A tile at lds + b*BM*ROWB; of the W tile after both A buffers
  auto As = [&](int b) { return lds + b * (BM * ROWB); };
  auto Ws = [&](int b) { return lds + 2 * BM * ROWB + b * (BN * ROWB); };

  int pm, pn;
  tile_coords(blockIdx.x, tm, tn, pm, pn);
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1;
  const int kc = kp >> 3;  // 16-byte chunks per row

  // global -> register staging: thread loads chunk (tid & 7) of rows (tid >> 3) + 32 i
  const u32x4* ga = ta + ((int64_t)pm * BM + (tid >> 3)) * kc + (tid & 7);
  const u32x4* gw = tw + ((int64_t)pn * BN + (tid >> 3)) * kc + (tid & 7);
  const int soff = (tid >> 3) * ROWB + (tid & 7) * 16;
  u32x4 ra_[BM / 32], rw_[BN / 32];

  auto gload = [&](int ks) {
#pragma unroll
    for (int i = 0; i < BM / 32; ++i) ra_[i] = __builtin_nontemporal_load(ga + (int64_t)i * 32 * kc + ks * (BK / 8));
#pragma unroll
    for (int i = 0; i < BN / 32; ++i) rw_[i] = __builtin_nontemporal_load(gw + (int64_t)i * 32 * kc + ks * (BK / 8));
  };
  auto swrite = [&](int b) {
#pragma unroll
    for (int i = 0; i < BM / 32; ++i) *reinterpret_cast<u32x4*>(As(b) + soff + i * 32 * ROWB) = ra_[i];
#pragma unroll
    for (int i = 0; i < BN / 32; ++i) *reinterpret_cast<u32x4*>(Ws(b) + soff + i * 32 * ROWB) = rw_[i];
  };

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  const int nks = kp / BK;
  gload(0);
  swrite(0);
  __syncthreads();
  // fragment read offsets: row (lane & 31) of the 32-row tile, 16-byte chunk (lane >> 5)
  const int aoff = (wm * 128 + (lane & 31)) * ROWB + (lane >> 5) * 16;
  const int woff = (wn * 64 + (lane & 31)) * ROWB + (lane >> 5) * 16;
  for (int ks = 0; ks < nks; ++ks) {
    const int b = ks & 1;
    if (ks + 1 < nks) gload(ks + 1);
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8 af[4], bfr[2];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(As(b) + aoff + i * 32 * ROWB + kk * 32);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8*>(Ws(b) + woff + j * 32 * ROWB + kk * 32);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (ks + 1 < nks) swrite(b ^ 1);
    __syncthreads();
  }

  // Epilogue.  32x32 accumulator layout: lane l holds column l%32; register e holds row
  // 8*(e/4) + 4*(l/32) + (e%4).
  const int64_t m0 = (int64_t)pm * BM + wm * 128;
  const int64_t n0 = (int64_t)pn * BN + wn * 64;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int64_t col = n0 + j * 32 + (lane & 31);
    const float sw = col < N ? rw[col] * scale : 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int64_t row = m0 + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        if (row < M && col < N) c[row * ldc + col] = acc[i][j][e] * (ra[row] * sw);
      }
  }
}

size_t decode_once_workspace(int64_t M, int64_t N, int64_t K) {
  using namespace gemm;
  const int64_t mp = (M + BM - 1) / BM * BM;
  const int64_t np = (N + BN - 1) / BN * BN;
  const int64_t kp = (K + BK - 1) / BK * BK;
  return (size_t)((mp + np) * kp * 2);
}

hipError_t launch_matmul_decode_once(const MatmulOperand& A, const MatmulOperand& W, int64_t K,
                                     float* c, int64_t ldc, float scale, void* ws,
                                     hipStream_t st) {
  using namespace gemm;
  const int nb = (int)(K / 8);
  const int64_t mp = (A.rows + BM - 1) / BM * BM;
  const int64_t np = (W.rows + BN - 1) / BN * BN;
  const int kp = (int)((K + BK - 1) / BK * BK);
  const int nbp = kp / 8;
  u32x4* wa = reinterpret_cast<u32x4*>(ws);
  u32x4* ww = wa + mp * nbp;
  hipLaunchKernelGGL(tiles_kernel, dim3((unsigned)((mp * nbp + 255) / 256)), dim3(256), 0, st,
                     A.codes, A.beta, A.rows, nb, mp, nbp, A.q, A.m2q, wa);
  hipLaunchKernelGGL(tiles_kernel, dim3((unsigned)((np * nbp + 255) / 256)), dim3(256), 0, st,
                     W.codes, W.beta, W.rows, nb, np, nbp, W.q, W.m2q, ww);
  const int tm = (int)(mp / BM), tn = (int)(np / BN);
  const size_t lds = (size_t)2 * (BM + BN) * ROWB;
  hipLaunchKernelGGL(gemm_kernel, dim3((unsigned)(tm * tn)), dim3(256), lds, st, wa, ww, kp, tm,
                     tn, A.scales, W.scales, A.rows, W.rows, c, ldc, scale);
  return hipGetLastError();
}

hipError_t gemm_set_attributes() {
  using namespace gemm;
  return hipFuncSetAttribute((const void*)gemm_kernel,
                             hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)(2 * (BM + BN) * ROWB));
}

}  // namespace nq
