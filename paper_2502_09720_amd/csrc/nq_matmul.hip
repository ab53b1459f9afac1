// Coded matrix product for small M (decode-shaped layers: a few activation rows against a
// large coded weight), C = A_hat * W_hat^T, Alg. 4 of the NestQuant paper for every pair of
// rows.
//
// Here the weight decode dominates (the product is a few flops per decoded weight entry),
// so every block of W is decoded exactly once, straight into a matrix-core operand: for
// v_mfma_f32_16x16x32_bf16 the B operand of lane l is the 8 K-values of column l % 16 at
// K offset 8 (l / 16), i.e. exactly one decoded block (t * X2, exact in bf16), so each lane
// decodes its own block and no LDS staging is needed.  The activation (at most 64 rows) is
// decoded once beforehand into a bf16 tile (tiles_kernel) that stays in cache; its
// fragments are loaded per step for up to four 16-row M tiles.  A workgroup owns 16
// columns of C; its four waves split K and combine their partial sums through LDS before
// the epilogue C_ij = acc * r_Ai * r_Wj * base_A * base_W / 4.
#include "nq_device.hpp"
#include "nq_kernels.hpp"

namespace nq {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__global__ __launch_bounds__(256) void tiles_kernel(const uint32_t* __restrict__ codes,
                                                    const uint32_t* __restrict__ beta,
                                                    int64_t rows, int nb, int64_t rows_p,
                                                    int nb_p, int q, uint32_t m2q, int lg,
                                                    u32x4* __restrict__ ws);

template <int MT>
__global__ __launch_bounds__(256) void skinny_kernel(const u32x4* __restrict__ ta, int nbp,
                                                     MatmulOperand A, MatmulOperand W, int nb,
                                                     float* __restrict__ c, int64_t ldc,
                                                     float scale) {
  __shared__ f32x4 part[3][MT][64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, kg = lane >> 4;
  const int64_t n = (int64_t)blockIdx.x * 16 + col;
  const bool nok = n < W.rows;
  const int nbw = (nb + 15) >> 4;
  const uint32_t* wc = W.codes + (nok ? n : 0) * nb;
  const uint32_t* wb = W.beta + (nok ? n : 0) * nbw;

  // K in steps of 32 (4 blocks); wave w takes a contiguous quarter of the steps
  const int nsteps = nbp / 4;
  const int s0 = (int)((int64_t)nsteps * wave / 4), s1 = (int)((int64_t)nsteps * (wave + 1) / 4);

  f32x4 acc[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int s = s0; s < s1; ++s) {
    const int blk = 4 * s + kg;
    u32x4 b = {0u, 0u, 0u, 0u};
    if (nok && blk < nb) {
      const uint32_t w = wc[blk];
      const int t = (int)((wb[blk >> 4] >> (2 * (blk & 15))) & 3u) + 1;
      b = decode_tile_bf16(w, t, W.q, W.m2q);
    }
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const u32x4 a = ta[(int64_t)(16 * m + col) * nbp + blk];
      acc[m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), acc[m],
                                                       0, 0, 0);
    }
  }

  if (wave > 0) {
#pragma unroll
    for (int m = 0; m < MT; ++m) part[wave - 1][m][lane] = acc[m];
  }
  __syncthreads();
  if (wave == 0) {
    // 16x16 accumulator layout: lane l holds column l % 16, register e holds row 4 (l/16) + e
    const float sw = nok ? W.scales[n] * scale : 0.0f;
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      f32x4 v = acc[m];
#pragma unroll
      for (int w = 0; w < 3; ++w) {
        const f32x4 o = part[w][m][lane];
        v.x += o.x; v.y += o.y; v.z += o.z; v.w += o.w;
      }
      const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t row = 16 * m + 4 * kg + e;
        if (nok && row < A.rows) c[row * ldc + n] = vv[e] * (A.scales[row] * sw);
      }
    }
  }
}

size_t skinny_workspace(int64_t M, int64_t K) {
  const int64_t mp = (M + 15) / 16 * 16;
  const int64_t kp = (K + 31) / 32 * 32;
  return (size_t)(mp * kp * 2);
}

hipError_t launch_matmul_skinny(int stages, const MatmulOperand& A, const MatmulOperand& W,
                                int64_t K, float* c, int64_t ldc, float scale, void* ws,
                                hipStream_t st) {
  const int nb = (int)(K / 8);
  const int64_t mp = (A.rows + 15) / 16 * 16;
  const int nbp = (int)((K + 31) / 32 * 32 / 8);
  u32x4* ta = reinterpret_cast<u32x4*>(ws);
  if (stages & 1) {
    int lg;
    int64_t wgs;
    grid_shape(mp, nbp, lg, wgs);
    hipLaunchKernelGGL(tiles_kernel, dim3((unsigned)wgs), dim3(256), 0, st, A.codes, A.beta,
                       A.rows, nb, mp, nbp, A.q, A.m2q, lg, ta);
  }
  if (!(stages & 2)) return hipGetLastError();
  const unsigned grid = (unsigned)((W.rows + 15) / 16);
  switch (mp / 16) {
    case 1: hipLaunchKernelGGL(skinny_kernel<1>, dim3(grid), dim3(256), 0, st, ta, nbp, A, W, nb, c, ldc, scale); break;
    case 2: hipLaunchKernelGGL(skinny_kernel<2>, dim3(grid), dim3(256), 0, st, ta, nbp, A, W, nb, c, ldc, scale); break;
    case 3: hipLaunchKernelGGL(skinny_kernel<3>, dim3(grid), dim3(256), 0, st, ta, nbp, A, W, nb, c, ldc, scale); break;
    default: hipLaunchKernelGGL(skinny_kernel<4>, dim3(grid), dim3(256), 0, st, ta, nbp, A, W, nb, c, ldc, scale); break;
  }
  return hipGetLastError();
}

}  // namespace nq
