// NestQuant decoder: Alg. 2 (Voronoi decode over 2E8, with the Gosset oracle of Alg. 5 or
// NestQuantM's of App. D) followed by the inverse scaling x_hat = r * beta_t * p (Alg. 3's
// normalization undone).
//
// Each block: read its code word, the row's beta word and scale, decode in exact integer
// arithmetic, and write the 8 values (32 B fp32 or 16 B fp16/bf16) with one or two vector
// stores; consecutive lanes handle consecutive blocks.
#include <type_traits>

#include "nq_device.hpp"
#include "nq_kernels.hpp"

namespace nq {

constexpr int kDecodePerThread = 8;

// The half-beta of index t from the kernel arguments (threads 0-3 copy the four into LDS,
// which the blocks then index).
__device__ __forceinline__ double pick_half_beta(const DecodeArgs& a, uint32_t t) {
  return t == 0 ? a.half_beta[0] : (t == 1 ? a.half_beta[1] : (t == 2 ? a.half_beta[2] : a.half_beta[3]));
}

// The blocks of the rows x nb matrix, in row-major order, are dealt to workgroups in runs
// of 256 * kDecodePerThread; thread t takes blocks t + 256 i of its run, so that every load
// and store instruction of a wave touches consecutive blocks.  A thread splits its first
// block's position into (row, column) once and steps it by 256 blocks for the next ones.
// It issues the loads of all its blocks (code word, beta word, row scale: buffer loads based
// at the run's first row, out-of-range offsets reading 0) before decoding any.
template <int OUT, int DV>  // OUT: 0 = fp32, 1 = fp16, 2 = bf16; DV: decoder_variant
__global__ __launch_bounds__(256) void decode_kernel(const uint32_t* __restrict__ codes,
                                                     const uint32_t* __restrict__ beta,
                                                     const float* __restrict__ scales,
                                                     int64_t rows, int nb, float inv_nb,
                                                     void* __restrict__ out, int64_t ld_out,
                                                     DecodeArgs a) {
  constexpr int TPB = kDecodePerThread;
  constexpr uint32_t OOB = 0x80000000u;
  const int64_t total = rows * nb;
  const int64_t g0 = (int64_t)blockIdx.x * (256 * TPB);
  const int64_t row0 = g0 / nb;
  const int j0 = (int)(g0 - row0 * nb);
  const int nbw = (nb + 15) >> 4;
  const int reach = (j0 + 256 * TPB + nb - 1) / nb;           // rows this workgroup touches
  const int span = (int)(rows - row0 < reach ? rows - row0 : reach);
  const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(codes + row0 * nb), (short)0, span * nb * 4, 0x00020000);
  const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(beta + row0 * nbw), (short)0, span * nbw * 4, 0x00020000);
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(scales + row0), (short)0, span * 4, 0x00020000);
  // the first block's (row, column) from o < nb + 256 TPB <= 2^14 by a float division checked
  // once in each direction; each further block is dr rows and dj columns on, with one carry
  const int o = j0 + (int)threadIdx.x;
  int r = (int)((float)o * inv_nb);
  if ((int)__umul24((uint32_t)r, (uint32_t)nb) > o) --r;
  if ((int)__umul24((uint32_t)(r + 1), (uint32_t)nb) <= o) ++r;
  int j = o - (int)__umul24((uint32_t)r, (uint32_t)nb);
  const int dr = 256 / nb, dj = 256 - dr * nb;
  // offset of the block's first output value from the run's first row, stepped with (r, j)
  // (one 64-bit multiply per thread; the steps are uniform)
  int64_t oo = (int64_t)r * ld_out + 8 * j;
  const int64_t ostep = (int64_t)dr * ld_out + 8 * dj, owrap = ld_out - 8 * (int64_t)nb;
  // blocks of this thread still inside the matrix: block i exists iff 256 i < left
  const int64_t left64 = total - g0 - (int64_t)threadIdx.x;
  const int left = left64 > 256 * TPB ? 256 * TPB : (int)left64;
  // the four half-betas in LDS, read by index (a select chain over kernel arguments
  // compiles to branches that every wave with mixed beta indices runs in full)
  __shared__ double hbt[4];
  if (threadIdx.x < 4) hbt[threadIdx.x] = pick_half_beta(a, threadIdx.x);
  uint32_t w[TPB], bw[TPB];
  float sr[TPB];
  int sh[TPB];        // bit position of the block's beta index in its beta word
  int64_t ooff[TPB];
  // Rows of a multiple of 16 blocks written without a gap (ld_out = cols): block i of this
  // thread is block o + 256 i of the run, its beta word o / 16 + 16 i at bits 2 (o mod 16)
  // and its output 8 (o + 256 i) values on; only the row, for the scale, is stepped (with no
  // carry when nb divides 256).
  auto load = [&](auto flat, auto carry) {
    constexpr bool FLAT = decltype(flat)::value;
#pragma unroll
    for (int i = 0; i < TPB; ++i) {
      if (i > 0) {
        j += dj;
        r += dr;
        if constexpr (!FLAT) oo += ostep;
        if (decltype(carry)::value && j >= nb) {
          j -= nb;
          ++r;
          if constexpr (!FLAT) oo += owrap;
        }
      }
      const uint32_t ok = 256 * i < left ? 0u : OOB;
      // the code words of a run are consecutive: block i of this thread is word o + 256 i
      // (ok sets bit 31 only, above every in-range offset, so the constant can follow it)
      w[i] = __builtin_amdgcn_raw_buffer_load_b32(rc, ((4u * (uint32_t)o) | ok) + 1024u * i, 0, 0);
      uint32_t bo;
      if constexpr (FLAT) {
        sh[i] = 2 * (o & 15);
        bo = ((4u * (uint32_t)(o >> 4)) | ok) + 64u * i;
        ooff[i] = 8 * (int64_t)o + 2048 * i;
      } else {
        sh[i] = 2 * (j & 15);
        bo = (4u * (__umul24((uint32_t)r, (uint32_t)nbw) + (uint32_t)(j >> 4))) | ok;
        ooff[i] = oo;
      }
      bw[i] = __builtin_amdgcn_raw_buffer_load_b32(rb, bo, 0, 0);
      sr[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, (4u * (uint32_t)r) | ok, 0, 0));
    }
  };
  if ((nb & 15) == 0 && ld_out == 8 * (int64_t)nb) {
    if (dj == 0) {
      load(std::true_type{}, std::false_type{});
    } else {
      load(std::true_type{}, std::true_type{});
    }
  } else {
    load(std::false_type{}, std::true_type{});
  }
  __syncthreads();   // hbt
#pragma unroll
  for (int i = 0; i < TPB; ++i) {
    if (256 * i >= left) break;
    const uint32_t t = (bw[i] >> sh[i]) & 3u;
    const double sc = (double)sr[i] * hbt[t];
    // X2 of the block: xs holds coordinates 0-3 and 4-7 as bytes X2 + 128 (decode_word_b8),
    // or X2 + 32 for NestQuantM at q = 16 (decode_word_m16, coordinate 0 apart)
    uint32_t xs[2];
    int x0 = 0;
    if constexpr (DV == 2) {
      decode_word_m16(w[i], xs[0], xs[1], x0);
    } else {
      decode_word_b8<DV == 1>(w[i], a.q, a.m2q, xs[0], xs[1]);
    }
    auto x2 = [&](int l) {
      if constexpr (DV == 2) {
        return l == 0 ? x0 : (int)((xs[l >> 2] >> (8 * (l & 3))) & 0xFFu) - 32;
      }
      return (int)((xs[l >> 2] >> (8 * (l & 3))) & 0xFFu) - 128;
    };
    if constexpr (OUT == 0) {
      // fp32: each value rounded once from its fp64 product
      float v[8];
#pragma unroll
      for (int l = 0; l < 8; ++l) v[l] = (float)(sc * (double)x2(l));
      f32x4* o = reinterpret_cast<f32x4*>((float*)out + row0 * ld_out + ooff[i]);
      const f32x4 lo = {v[0], v[1], v[2], v[3]};
      const f32x4 hi = {v[4], v[5], v[6], v[7]};
      __builtin_nontemporal_store(lo, o);
      __builtin_nontemporal_store(hi, o + 1);
    } else {
      // 16-bit outputs: X2 (|X2| <= 32) times the fp32-rounded scale is within two fp32
      // roundings (relative 2^-23) of the exact value, far below half an fp16 / bf16 ulp,
      // so the final rounding lands on the nearest or the adjacent 16-bit value.  From the
      // biased byte b = X2 + 128 the fp32 product is one fma, b s - 128 s (128 s is exact),
      // the same rounding of the same exact value X2 s.
      const float s32 = (float)sc, off = -128.0f * s32;
      auto val = [&](int l) {
        if constexpr (DV == 2) return (float)x2(l) * s32;
        return __builtin_fmaf((float)((xs[l >> 2] >> (8 * (l & 3))) & 0xFFu), s32, off);
      };
      uint32_t pk[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if constexpr (OUT == 1) {
          // the fma and its rounding to fp16 in one mixed-precision instruction per half
          if constexpr (DV == 2) {
            pk[u] = fma_mix_pk_f16((float)x2(2 * u), (float)x2(2 * u + 1), s32, 0.0f);
          } else {
            const uint32_t x = xs[u >> 1];
            const float b0 = (float)((x >> (16 * (u & 1))) & 0xFFu);
            const float b1 = (float)((x >> (16 * (u & 1) + 8)) & 0xFFu);
            pk[u] = fma_mix_pk_f16(b0, b1, s32, off);
          }
        } else {
          // one two-value conversion (round to nearest even) per word
          typedef float f32x2 __attribute__((ext_vector_type(2)));
          typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
          pk[u] = __builtin_bit_cast(
              uint32_t, __builtin_convertvector((f32x2){val(2 * u), val(2 * u + 1)}, bf16x2));
        }
      }
      const u32x4 v = {pk[0], pk[1], pk[2], pk[3]};
      __builtin_nontemporal_store(
          v, reinterpret_cast<u32x4*>((uint16_t*)out + row0 * ld_out + ooff[i]));
    }
  }
}

hipError_t launch_decode(const uint32_t* codes, const uint32_t* beta, const float* scales,
                         int64_t rows, int cols, void* out, int out_dtype, int64_t ld_out,
                         const DecodeArgs& a, hipStream_t st) {
  const int nb = cols / 8;
  const int64_t total = rows * nb;
  const unsigned grid = (unsigned)((total + 256 * kDecodePerThread - 1) / (256 * kDecodePerThread));
  const float inv = 1.0f / (float)nb;
#define NQ_DEC(O, DV)                                                                       \
  hipLaunchKernelGGL((decode_kernel<O, DV>), dim3(grid), dim3(256), 0, st, codes, beta,     \
                     scales, rows, nb, inv, out, ld_out, a)
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
