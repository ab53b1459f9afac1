// NestQuant decoder: Alg. 2 (Voronoi decode over 2E8, with the Gosset oracle of Alg. 5 or
// NestQuantM's of App. D) followed by the inverse scaling x_hat = r * beta_t * p (Alg. 3's
// normalization undone).
//
// One lane per 8-entry block: read one code word, the row's beta word and scale, decode in
// exact integer arithmetic, and write the 8 values (32 B fp32 or 16 B fp16/bf16) with one
// or two vector stores; consecutive lanes handle consecutive blocks of a row.
#include "nq_device.hpp"
#include "nq_kernels.hpp"

namespace nq {

template <int OUT, int DV>  // OUT: 0 = fp32, 1 = fp16, 2 = bf16; DV: decoder_variant
__global__ __launch_bounds__(256) void decode_kernel(const uint32_t* __restrict__ codes,
                                                     const uint32_t* __restrict__ beta,
                                                     const float* __restrict__ scales,
                                                     int64_t rows, int nb, int lg,
                                                     void* __restrict__ out, int64_t ld_out,
                                                     DecodeArgs a) {
  const GridPos g = grid_block(nb, lg);
  if (g.rb + g.lr >= rows || g.j >= nb) return;
  const int j = g.j;
  const int nbw = (nb + 15) >> 4;
  const uint32_t w = __builtin_nontemporal_load(codes + g.rb * nb + (uint32_t)(g.lr * nb + j));
  const uint32_t bw = beta[g.rb * nbw + (uint32_t)(g.lr * nbw + (j >> 4))];
  const int t = (int)((bw >> (2 * (j & 15))) & 3u);
  const double sc = (double)scales[g.rb + g.lr] * a.half_beta[t];
  uint32_t X2p[4];
  if constexpr (DV == 2) {
    // byte-SIMD NestQuantM at q = 16: repack the signed bytes as int16 pairs
    uint32_t xa, xb;
    int x0;
    decode_word_m16(w, xa, xb, x0);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t x = i < 2 ? xa : xb;
      const int lo = i == 0 ? x0 : ((int)(int8_t)(uint8_t)(x >> (16 * (i & 1))) >> 2);
      const int hi = (int)(int8_t)(uint8_t)(x >> (16 * (i & 1) + 8)) >> 2;
      X2p[i] = ((uint32_t)lo & 0xFFFFu) | ((uint32_t)hi << 16);
    }
  } else {
    decode_word_pk<DV == 1>(w, a.q, a.m2q, X2p);
  }
  if constexpr (OUT == 0) {
    // fp32: each value rounded once from its fp64 product
    float v[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = (float)(sc * (double)(int)(short)(X2p[i] & 0xFFFFu));
      v[2 * i + 1] = (float)(sc * (double)((int)X2p[i] >> 16));
    }
    f32x4* o = reinterpret_cast<f32x4*>((float*)out + (g.rb + g.lr) * ld_out + 8 * j);
    const f32x4 lo = {v[0], v[1], v[2], v[3]};
    const f32x4 hi = {v[4], v[5], v[6], v[7]};
    __builtin_nontemporal_store(lo, o);
    __builtin_nontemporal_store(hi, o + 1);
  } else {
    // 16-bit outputs: X2 (|X2| <= 32) times the fp32-rounded scale is within two fp32
    // roundings (relative 2^-23) of the exact value, far below half an fp16 / bf16 ulp,
    // so the final rounding lands on the nearest or the adjacent 16-bit value
    const float s32 = (float)sc;
    uint32_t pk[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float lo = (float)(int)(short)(X2p[i] & 0xFFFFu) * s32;
      const float hi = (float)((int)X2p[i] >> 16) * s32;
      if constexpr (OUT == 1) {
        pk[i] = (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)lo) |
                ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)hi) << 16);
      } else {
        pk[i] = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)lo) |
                ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)hi) << 16);
      }
    }
    const u32x4 v = {pk[0], pk[1], pk[2], pk[3]};
    __builtin_nontemporal_store(
        v, reinterpret_cast<u32x4*>((uint16_t*)out + (g.rb + g.lr) * ld_out + 8 * j));
  }
}

hipError_t launch_decode(const uint32_t* codes, const uint32_t* beta, const float* scales,
                         int64_t rows, int cols, void* out, int out_dtype, int64_t ld_out,
                         const DecodeArgs& a, hipStream_t st) {
  const int nb = cols / 8;
  int lg;
  int64_t wgs;
  grid_shape(rows, nb, lg, wgs);
  const unsigned grid = (unsigned)wgs;
#define NQ_DEC(O, DV)                                                                       \
  hipLaunchKernelGGL((decode_kernel<O, DV>), dim3(grid), dim3(256), 0, st, codes, beta,     \
                     scales, rows, nb, lg, out, ld_out, a)
#define NQ_DEC3(O) \
  if (dv == 0) NQ_DEC(O, 0); else if (dv == 1) NQ_DEC(O, 1); else NQ_DEC(O, 2)
  const int dv = decoder_variant(a.decoder, a.q);
  switch (out_dtype) {
    case 0: NQ_DEC3(0); break;
    case 1: NQ_DEC3(1); break;
    default: NQ_DEC3(2); break;
  }
#undef NQ_DEC3
#undef NQ_DEC
  return hipGetLastError();
}

}  // namespace nq
