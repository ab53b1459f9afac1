// Coded matrix product C = A_hat * W_hat^T (Alg. 4 of the NestQuant paper for every pair of
// rows), fused: code words are decoded (Alg. 2) into LDS as exact bf16 integer tiles t*X2
// and contracted on the bf16 matrix cores with fp32 accumulation; the per-row scales and
// base_A * base_W / 4 are applied in the epilogue.
//
// Tiling: a 256-thread workgroup (4 waves) owns a 128 x 128 tile of C; each wave owns a
// 64 x 64 quadrant as 2 x 2 v_mfma_f32_32x32x16_bf16 tiles.  The K loop steps over 8 blocks
// (64 entries): the 128 rows of A and of W times 8 blocks are decoded (4 + 4 per thread)
// into LDS, one 16-byte bf16x8 per block.  The MFMA A operand of lane l is the 8 K-values
// of row l%32 at K offset 8*(l/32), i.e. exactly one decoded block, so each fragment load is
// one 16-byte LDS read.
#include "nq_device.hpp"
#include "nq_kernels.hpp"

namespace nq {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int BM = 128;
constexpr int BN = 128;
constexpr int KBLK = 8;         // blocks per K step
constexpr int LDS_STRIDE = 9;   // uint4 per tile row (8 blocks + 1 pad against bank conflicts)

__device__ __forceinline__ void decode_tile(const MatmulOperand& op, int64_t row0, int nb, int kb0,
                                            uint4 (*lds)[LDS_STRIDE]) {
  const int nbw = (nb + 15) >> 4;
#pragma unroll
  for (int it = 0; it < (BM * KBLK) / 256; ++it) {
    const int idx = threadIdx.x + it * 256;
    const int r = idx / KBLK;
    const int b = idx % KBLK;
    const int64_t gr = row0 + r;
    const int gb = kb0 + b;
    uint4 val = make_uint4(0, 0, 0, 0);
    if (gr < op.rows && gb < nb) {
      const uint32_t w = op.codes[gr * nb + gb];
      const uint32_t bw = op.beta[gr * nbw + (gb >> 4)];
      const int t = (int)((bw >> (2 * (gb & 15))) & 3u) + 1;
      const u32x4 v = decode_tile_bf16(w, t, op.q, op.m2q);
      val = make_uint4(v.x, v.y, v.z, v.w);
    }
    lds[r][b] = val;
  }
}

__global__ __launch_bounds__(256) void matmul_kernel(MatmulOperand A, MatmulOperand W, int nb,
                                                     int tiles_n, float* __restrict__ c,
                                                     int64_t ldc, float scale) {
  __shared__ uint4 As[BM][LDS_STRIDE];
  __shared__ uint4 Ws[BN][LDS_STRIDE];

  const int tile = blockIdx.x;
  const int64_t m0 = (int64_t)(tile / tiles_n) * BM;
  const int64_t n0 = (int64_t)(tile % tiles_n) * BN;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int wm = wave >> 1, wn = wave & 1;

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  for (int kb0 = 0; kb0 < nb; kb0 += KBLK) {
    decode_tile(A, m0, nb, kb0, As);
    decode_tile(W, n0, nb, kb0, Ws);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < KBLK / 2; ++kk) {
      bf16x8 af[2], bfr[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const uint4 u = As[wm * 64 + i * 32 + (lane & 31)][2 * kk + (lane >> 5)];
        af[i] = __builtin_bit_cast(bf16x8, u);
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const uint4 u = Ws[wn * 64 + j * 32 + (lane & 31)][2 * kk + (lane >> 5)];
        bfr[j] = __builtin_bit_cast(bf16x8, u);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }

  // Epilogue.  32x32 accumulator layout: lane l holds column l%32; register e holds row
  // 8*(e/4) + 4*(l/32) + (e%4).
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t col = n0 + wn * 64 + j * 32 + (lane & 31);
      if (col >= W.rows) continue;
      const float sw = W.scales[col] * scale;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int64_t row = m0 + wm * 64 + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        if (row < A.rows) c[row * ldc + col] = acc[i][j][e] * (A.scales[row] * sw);
      }
    }
}

hipError_t launch_matmul(const MatmulOperand& A, const MatmulOperand& W, int64_t K, float* c,
                         int64_t ldc, float scale, hipStream_t st) {
  const int nb = (int)(K / 8);
  const int64_t tiles_m = (A.rows + BM - 1) / BM;
  const int64_t tiles_n = (W.rows + BN - 1) / BN;
  hipLaunchKernelGGL(matmul_kernel, dim3((unsigned)(tiles_m * tiles_n)), dim3(256), 0, st, A, W,
                     nb, (int)tiles_n, c, ldc, scale);
  return hipGetLastError();
}

}  // namespace nq
