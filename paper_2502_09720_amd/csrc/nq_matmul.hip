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
#include <type_traits>

#include "nq_device.hpp"
#include "nq_kernels.hpp"

namespace nq {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

template <bool I8>
void launch_tiles(const MatmulOperand& X, int nb, int64_t rows_p, int nb_p, void* ws,
                  hipStream_t st);

// W block j of this lane's column as a matrix-core operand.  bf16: one block (8 values,
// 16 B); int8: two consecutive blocks (16 values, 16 B).
template <bool I8, bool M>
__device__ __forceinline__ u32x4 w_operand(const uint32_t* wc, const uint32_t* wb, int blk,
                                           int nb, const MatmulOperand& W) {
  if constexpr (I8) {
    u32x2 lo = {0u, 0u}, hi = {0u, 0u};
    if (blk < nb) {
      lo = decode_tile_i8<M>(wc[blk], (int)((wb[blk >> 4] >> (2 * (blk & 15))) & 3u) + 1, W.q,
                          W.m2q);
    }
    if (blk + 1 < nb) {
      const int b1 = blk + 1;
      hi = decode_tile_i8<M>(wc[b1], (int)((wb[b1 >> 4] >> (2 * (b1 & 15))) & 3u) + 1, W.q,
                          W.m2q);
    }
    return u32x4{lo.x, lo.y, hi.x, hi.y};
  } else {
    if (blk >= nb) return u32x4{0u, 0u, 0u, 0u};
    return decode_tile_bf16<M>(wc[blk], (int)((wb[blk >> 4] >> (2 * (blk & 15))) & 3u) + 1, W.q,
                            W.m2q);
  }
}

// One workgroup per 16 columns of C; four waves split K.  Per step a wave covers 32 (bf16,
// v_mfma_f32_16x16x32_bf16) or 64 (int8, v_mfma_i32_16x16x64_i8) values of K: lane l holds
// column l % 16 at K offset (step size / 4) * (l / 16), 16 B of it.  ta is the decoded A
// tile, [16 * MT][kcb] 16-byte chunks.
template <int MT, bool I8, bool MW>
__global__ __launch_bounds__(256) void skinny_kernel(const u32x4* __restrict__ ta, int kcb,
                                                     MatmulOperand A, MatmulOperand W, int nb,
                                                     float* __restrict__ c, int64_t ldc,
                                                     float scale) {
  using Acc = typename std::conditional<I8, i32x4, f32x4>::type;
  __shared__ Acc part[3][MT][64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, kg = lane >> 4;
  const int64_t n = (int64_t)blockIdx.x * 16 + col;
  const bool nok = n < W.rows;
  const int nbw = (nb + 15) >> 4;
  const uint32_t* wc = W.codes + (nok ? n : 0) * nb;
  const uint32_t* wb = W.beta + (nok ? n : 0) * nbw;
  constexpr int BPL = I8 ? 2 : 1;   // blocks per lane per step

  // K in steps of 4 * BPL blocks; wave w takes a contiguous quarter of the steps
  const int nsteps = kcb / 4;
  const int s0 = (int)((int64_t)nsteps * wave / 4), s1 = (int)((int64_t)nsteps * (wave + 1) / 4);

  Acc acc[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) acc[m] = Acc{};

  for (int s = s0; s < s1; ++s) {
    const int blk = (4 * s + kg) * BPL;
    const u32x4 b = nok ? w_operand<I8, MW>(wc, wb, blk, nb, W) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const u32x4 a = ta[(int64_t)(16 * m + col) * kcb + 4 * s + kg];
      if constexpr (I8) {
        acc[m] = __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, a),
                                                       __builtin_bit_cast(i32x4, b), acc[m],
                                                       0, 0, 0);
      } else {
        acc[m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                         __builtin_bit_cast(bf16x8, b), acc[m],
                                                         0, 0, 0);
      }
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
      Acc v = acc[m];
#pragma unroll
      for (int w = 0; w < 3; ++w) {
        const Acc o = part[w][m][lane];
        v.x += o.x; v.y += o.y; v.z += o.z; v.w += o.w;
      }
      const float vv[4] = {(float)v.x, (float)v.y, (float)v.z, (float)v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t row = 16 * m + 4 * kg + e;
        if (nok && row < A.rows) c[row * ldc + n] = vv[e] * (A.scales[row] * sw);
      }
    }
  }
}

// Rows of the A tile are padded to 128 B (64 bf16 or 128 int8) and to 16 rows.
size_t skinny_workspace(int64_t M, int64_t K) {
  const int64_t mp = (M + 15) / 16 * 16;
  const int64_t kp = (K + 63) / 64 * 64;
  return (size_t)(mp * kp * 2);
}

template <bool I8>
static hipError_t skinny(int stages, const MatmulOperand& A, const MatmulOperand& W, int64_t K,
                         float* c, int64_t ldc, float scale, void* ws, hipStream_t st) {
  const int nb = (int)(K / 8);
  const int64_t mp = (A.rows + 15) / 16 * 16;
  constexpr int EB = I8 ? 1 : 2;
  const int64_t kp = (K * EB + 127) / 128 * 128 / EB;
  const int nbp = (int)(kp / 8);
  const int kcb = (int)(kp * EB / 16);
  u32x4* ta = reinterpret_cast<u32x4*>(ws);
  if (stages & 1) launch_tiles<I8>(A, nb, mp, nbp, (void*)ta, st);
  if (!(stages & 2)) return hipGetLastError();
  const unsigned grid = (unsigned)((W.rows + 15) / 16);
#define NQ_SK(MT, MW)                                                                     \
  hipLaunchKernelGGL((skinny_kernel<MT, I8, MW>), dim3(grid), dim3(256), 0, st, ta, kcb, A, W, \
                     nb, c, ldc, scale)
#define NQ_SK2(MT) \
  if (W.decoder) NQ_SK(MT, true); else NQ_SK(MT, false)
  switch (mp / 16) {
    case 1: NQ_SK2(1); break;
    case 2: NQ_SK2(2); break;
    case 3: NQ_SK2(3); break;
    default: NQ_SK2(4); break;
  }
#undef NQ_SK2
#undef NQ_SK
  return hipGetLastError();
}

hipError_t launch_matmul_skinny(int stages, bool i8, const MatmulOperand& A,
                                const MatmulOperand& W, int64_t K, float* c, int64_t ldc,
                                float scale, void* ws, hipStream_t st) {
  return i8 ? skinny<true>(stages, A, W, K, c, ldc, scale, ws, st)
            : skinny<false>(stages, A, W, K, c, ldc, scale, ws, st);
}

}  // namespace nq
