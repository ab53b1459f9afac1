// Coded matrix product that needs no workspace (nq_matmul): every workgroup decodes the code
// words of its own A and W rows straight into LDS as m * X2 tiles and contracts them there.
//
// C = A_hat W_hat^T is Alg. 4 of the NestQuant paper for every pair of rows.  Here Alg. 2
// (with Alg. 5) runs inside the product: for each stage of 8 blocks (64 values of K) the
// threads of a workgroup fetch the code and beta words of the tile's BM + BN rows, decode
// them into bf16 (or fp16) integers m * X2, exact, and store them in LDS with the swizzle of
// the decode-once GEMM; the waves then multiply the stage on 32x32x16 matrix cores with fp32
// accumulation, and the epilogue scales by r_Ai r_Wj base_A base_W / 4.  Two LDS buffers:
// stage s + 1 is decoded while stage s is multiplied, and the code words of stage s + 2 are
// in flight meanwhile.
//
// The price of needing no memory: a block of A is decoded once per BN columns of C and a
// block of W once per BM rows, where the decode-once path (nq_matmul_ex) decodes each block
// once into a caller's workspace.  Decoding costs more vector instructions than the matrix
// cores spend on the block, so this path is bound by its decodes.  Rows of the tile past M
// (or N) are never decoded (their LDS rows stay zero) and waves whose rows all lie past M
// skip their matrix-core work, which keeps decode-shaped products (M <= 64) cheap: there W
// is decoded once and A once per BN columns.
#include <algorithm>
#include <type_traits>

#include "nq_device.hpp"
#include "nq_gemm_common.hpp"
#include "nq_kernels.hpp"

namespace nq {

namespace fused {
// BM x BN tile, WM x WN waves of (BM / WM) x (BN / WN) outputs; every stage holds 8 blocks
// (128 bytes of 16-bit values) of each of the BM + BN rows.
template <int BM_, int BN_, int WM_, int WN_>
struct Cfg {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_;
  static constexpr int NW = WM * WN, NT = NW * 64;
  static constexpr int TM = BM / WM / 32, TN = BN / WN / 32;
  static constexpr int SB = 128, CH = 8, BPS = 8;           // bytes, chunks, blocks per row
  static constexpr int STAGE_BYTES = (BM + BN) * SB;
  static constexpr int ROWSTEP = NT / BPS;                  // rows covered by one pass
  static constexpr int ITEMS = (BM + BN) / ROWSTEP;         // blocks per thread per stage
  static constexpr int AITEMS = BM / ROWSTEP;               // the first AITEMS are A's
  static_assert(BM % ROWSTEP == 0 && BN % ROWSTEP == 0, "rows must split evenly");
  static_assert(TM >= 1 && TN >= 1, "wave tiles of 32 x 32 at least");
  static_assert(2 * STAGE_BYTES <= 160 * 1024, "LDS is 160 KB");
};
using CfgLarge = Cfg<256, 128, 4, 2>;   // M > 64
using CfgSmall = Cfg<64, 64, 2, 2>;     // M <= 64: more workgroups along N
}  // namespace fused

template <bool F16>
__device__ __forceinline__ u32x4 decode16_dv(uint32_t w, int m, int q, uint32_t m2q, int dv) {
  if (dv == 0) return decode_tile_16<0, F16>(w, m, q, m2q);
  if (dv == 1) return decode_tile_16<1, F16>(w, m, q, m2q);
  return decode_tile_16<2, F16>(w, m, q, m2q);
}

template <class C, int ET>
__global__ __launch_bounds__(C::NT, 1) void fused_kernel(MatmulOperand A, MatmulOperand W,
                                                         int dva, int dvw, int nb, int tm,
                                                         int tn, float* __restrict__ c,
                                                         int64_t ldc, float scale) {
  constexpr int BM = C::BM, BN = C::BN, WM = C::WM, WN = C::WN, TM = C::TM, TN = C::TN;
  constexpr int SB = C::SB, CH = C::CH, BPS = C::BPS, NT = C::NT;
  constexpr int STAGE_BYTES = C::STAGE_BYTES, ROWSTEP = C::ROWSTEP;
  constexpr int ITEMS = C::ITEMS, AITEMS = C::AITEMS;
  constexpr bool F16 = ET == ET_F16;
  constexpr uint32_t OOB = 0x80000000u;   // beyond every buffer range below: reads 0
  extern __shared__ __attribute__((aligned(1024))) unsigned char lds[];

  int pm, pn;
  tile_coords(blockIdx.x, tm, tn, pm, pn);
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int wm = wave / WN, wn = wave % WN;
  const int nbw = (nb + 15) >> 4;

  // This tile's rows of each operand (>= 1), read through buffer resources based at the
  // tile's first row: 32-bit offsets, and the range check returns 0 past the operand.
  const int64_t a0 = (int64_t)pm * BM, w0 = (int64_t)pn * BN;
  const int arows = (int)std::min<int64_t>(BM, A.rows - a0);
  const int wrows = (int)std::min<int64_t>(BN, W.rows - w0);
  const __amdgpu_buffer_rsrc_t rac = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(A.codes + a0 * nb), (short)0, arows * nb * 4, 0x00020000);
  const __amdgpu_buffer_rsrc_t rab = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(A.beta + a0 * nbw), (short)0, arows * nbw * 4, 0x00020000);
  const __amdgpu_buffer_rsrc_t rwc = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(W.codes + w0 * nb), (short)0, wrows * nb * 4, 0x00020000);
  const __amdgpu_buffer_rsrc_t rwb = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(W.beta + w0 * nbw), (short)0, wrows * nbw * 4, 0x00020000);

  // Item j of this thread: tile row lr + ROWSTEP j (A's rows first, then W's), block lb of
  // each stage.  Eight consecutive threads read the eight consecutive words of one row.
  const int lr = tid / BPS, lb = tid % BPS;
  bool valid[ITEMS];
  uint32_t coff[ITEMS], boff[ITEMS];
  int loff[ITEMS];
#pragma unroll
  for (int j = 0; j < ITEMS; ++j) {
    const int row = lr + ROWSTEP * j;
    const int r = j < AITEMS ? row : row - BM;
    valid[j] = r < (j < AITEMS ? arows : wrows);
    coff[j] = (uint32_t)(r * nb) * 4u;
    boff[j] = (uint32_t)(r * nbw) * 4u;
    loff[j] = row * SB + ((lb ^ swz<CH>(row)) * 16);
  }
  uint32_t cw[ITEMS], bw[ITEMS];
  auto fetch = [&](int ks) {
    const int jb = ks * BPS + lb;
    const bool in = jb < nb;
#pragma unroll
    for (int j = 0; j < ITEMS; ++j) {
      if (!valid[j]) continue;
      const uint32_t co = in ? coff[j] + 4u * (uint32_t)jb : OOB;
      const uint32_t bo = in ? boff[j] + 4u * (uint32_t)(jb >> 4) : OOB;
      if (j < AITEMS) {
        cw[j] = __builtin_amdgcn_raw_buffer_load_b32(rac, co, 0, 0);
        bw[j] = __builtin_amdgcn_raw_buffer_load_b32(rab, bo, 0, 0);
      } else {
        cw[j] = __builtin_amdgcn_raw_buffer_load_b32(rwc, co, 0, 0);
        bw[j] = __builtin_amdgcn_raw_buffer_load_b32(rwb, bo, 0, 0);
      }
    }
  };
  // m * X2 of the fetched words of stage ks into buffer ks % 2 (a zero word, read past the
  // row, decodes to zero)
  auto decode_store = [&](int ks) {
    unsigned char* base = lds + (ks & 1) * STAGE_BYTES;
    const uint32_t sh = 2u * (uint32_t)((ks * BPS + lb) & 15);
#pragma unroll
    for (int j = 0; j < ITEMS; ++j) {
      if (!valid[j]) continue;
      u32x4 v;
      if (j < AITEMS) {
        v = decode16_dv<F16>(cw[j], beta_mult(A.mtab, (bw[j] >> sh) & 3u), A.q, A.m2q, dva);
      } else {
        v = decode16_dv<F16>(cw[j], beta_mult(W.mtab, (bw[j] >> sh) & 3u), W.q, W.m2q, dvw);
      }
      *reinterpret_cast<u32x4*>(base + loff[j]) = v;
    }
  };

  using Acc = f32x16;
  Acc acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = Acc{};
  // fragment reads as in the decode-once GEMM: row (lane & 31) of a 32-row tile, logical
  // chunk 2 kk + (lane >> 5)
  const int frow = lane & 31;
  const int abase = (wm * (BM / WM) + frow) * SB;
  const int wbase = BM * SB + (wn * (BN / WN) + frow) * SB;
  int fo[CH / 2];
#pragma unroll
  for (int kk = 0; kk < CH / 2; ++kk) fo[kk] = ((2 * kk + (lane >> 5)) ^ swz<CH>(frow)) * 16;
  // waves whose A rows (or W rows) all lie past the operand have nothing to multiply
  const bool active = wm * (BM / WM) < arows && wn * (BN / WN) < wrows;
  auto multiply = [&](int ks) {
    const unsigned char* sb = lds + (ks & 1) * STAGE_BYTES;
#pragma unroll
    for (int kk = 0; kk < CH / 2; ++kk) {
      u32x4 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *reinterpret_cast<const u32x4*>(sb + abase + i * 32 * SB + fo[kk]);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = *reinterpret_cast<const u32x4*>(sb + wbase + j * 32 * SB + fo[kk]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          if constexpr (F16) {
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(
                __builtin_bit_cast(f16x8, af[i]), __builtin_bit_cast(f16x8, bfr[j]), acc[i][j],
                0, 0, 0);
          } else {
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8, af[i]), __builtin_bit_cast(bf16x8, bfr[j]),
                acc[i][j], 0, 0, 0);
          }
        }
    }
  };

  // Both buffers start zeroed: the rows past the operands are never written.
  for (int o = tid * 16; o < 2 * STAGE_BYTES; o += NT * 16)
    *reinterpret_cast<u32x4*>(lds + o) = u32x4{0u, 0u, 0u, 0u};
  const int nks = (nb + BPS - 1) / BPS;
  fetch(0);
  __syncthreads();
  decode_store(0);
  if (nks > 1) fetch(1);
  for (int ks = 0; ks < nks; ++ks) {
    // stage ks is complete in LDS, and nobody still reads the other buffer (stage ks - 1)
    __syncthreads();
    if (ks + 1 < nks) {
      decode_store(ks + 1);
      if (ks + 2 < nks) fetch(ks + 2);
    }
    if (active) multiply(ks);
  }
  if (!active) return;

  // Epilogue: C = acc * r_A * (r_W * scale).  32x32 accumulator layout: lane l holds column
  // l % 32; register e holds row 8 (e / 4) + 4 (l / 32) + (e % 4).
  const int64_t M = A.rows, N = W.rows;
  const int64_t m0 = a0 + wm * (BM / WM) + 4 * (lane >> 5);
  const int64_t n0 = w0 + wn * (BN / WN) + (lane & 31);
  float* cp = c + m0 * ldc + n0;
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int64_t col = n0 + j * 32;
    if (col >= N) continue;
    const float cs = W.scales[col] * scale;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int r = i * 32 + 8 * (e >> 2) + (e & 3);
        if (m0 + r < M)
          __builtin_nontemporal_store(acc[i][j][e] * (A.scales[m0 + r] * cs),
                                      &cp[r * ldc + j * 32]);
      }
  }
}

template <class C, int ET>
static hipError_t launch_fused_cfg(const MatmulOperand& A, const MatmulOperand& W, int64_t K,
                                   float* c, int64_t ldc, float scale, hipStream_t st) {
  const int nb = (int)(K / 8);
  const int tm = (int)((A.rows + C::BM - 1) / C::BM), tn = (int)((W.rows + C::BN - 1) / C::BN);
  const int dva = decoder_variant(A.decoder, A.q), dvw = decoder_variant(W.decoder, W.q);
  hipLaunchKernelGGL((fused_kernel<C, ET>), dim3((unsigned)(tm * tn)), dim3(C::NT),
                     (size_t)(2 * C::STAGE_BYTES), st, A, W, dva, dvw, nb, tm, tn, c, ldc,
                     scale);
  return hipGetLastError();
}

hipError_t launch_matmul_fused(int et, const MatmulOperand& A, const MatmulOperand& W,
                               int64_t K, float* c, int64_t ldc, float scale, hipStream_t st) {
  using namespace fused;
  const bool small = A.rows <= kFusedMaxM;
  if (et == ET_F16)
    return small ? launch_fused_cfg<CfgSmall, ET_F16>(A, W, K, c, ldc, scale, st)
                 : launch_fused_cfg<CfgLarge, ET_F16>(A, W, K, c, ldc, scale, st);
  return small ? launch_fused_cfg<CfgSmall, ET_BF16>(A, W, K, c, ldc, scale, st)
               : launch_fused_cfg<CfgLarge, ET_BF16>(A, W, K, c, ldc, scale, st);
}

hipError_t fused_set_attributes() {
  using namespace fused;
  const void* k[4] = {(const void*)fused_kernel<CfgLarge, ET_BF16>,
                      (const void*)fused_kernel<CfgLarge, ET_F16>,
                      (const void*)fused_kernel<CfgSmall, ET_BF16>,
                      (const void*)fused_kernel<CfgSmall, ET_F16>};
  const int bytes[4] = {2 * CfgLarge::STAGE_BYTES, 2 * CfgLarge::STAGE_BYTES,
                        2 * CfgSmall::STAGE_BYTES, 2 * CfgSmall::STAGE_BYTES};
  for (int i = 0; i < 4; ++i) {
    const hipError_t e =
        hipFuncSetAttribute(k[i], hipFuncAttributeMaxDynamicSharedMemorySize, bytes[i]);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace nq
