// Coded matrix product for small M (decode-shaped layers: a few activation rows against a
// large coded weight), C = A_hat * W_hat^T, Alg. 4 of the NestQuant paper for every pair of
// rows.
//
// Here the weight decode dominates (the product is a few flops per decoded weight entry),
// so every block of W is decoded exactly once, straight into a matrix-core operand: for
// v_mfma_f32_16x16x32_bf16 the B operand of lane l is the 8 K-values of column l % 16 at
// K offset 8 (l / 16), i.e. exactly one decoded block (m * X2, exact in bf16; fp16 for beta
// sets whose multiples m exceed what bf16 holds), so each lane decodes its own block and no
// LDS staging is needed.  The activation (at most 64 rows) is
// decoded once beforehand into a bf16 tile (tiles_kernel) that stays in cache; its
// fragments are loaded per step for up to four 16-row M tiles.  A workgroup owns 16
// columns of C; its four waves split K and combine their partial sums through LDS before
// the epilogue C_ij = acc * r_Ai * r_Wj * base_A * base_W / 4.
#include <algorithm>
#include <type_traits>

#include "nq_device.hpp"
#include "nq_kernels.hpp"

namespace nq {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

template <int ET>
void launch_tiles(const MatmulOperand& X, int nb, int64_t rows_p, int nb_p, void* ws,
                  hipStream_t st);

// One workgroup per 16 columns of C; its NWV waves split K.  An MFMA sums over its K values
// in any order as long as both operands follow it, so K is dealt in chunks of 4 PD steps'
// worth of blocks (32 blocks for bf16, PD = 8) and lane (column l % 16, group g = l / 16)
// takes the g-th quarter of each chunk, one block (bf16, v_mfma_f32_16x16x32_bf16) or two
// (int8, v_mfma_i32_16x16x64_i8) per step.  A lane's code words of a chunk are then
// contiguous (two or four 16-byte loads) and share one beta word, and its A fragments are
// the matching 16-byte chunks of the decoded A tile ta ([16 * MT][kcb] chunks; rows at or
// past M are not read).  Buffer loads with 32-bit offsets and the hardware range check:
// words out of range read as 0 (a zero code word decodes to zero); a chunk that runs past
// the end of a row is read word by word, the words past the row made out of range.  The
// next chunk's words are loaded while the current one is decoded (two register sets in
// turn).  The host keeps W's code array below
// 2^31 bytes per launch.
//
// ADEC (one or two activation rows, the GEMV): each workgroup first decodes A's rows itself
// into LDS (the same tile layout, kcb chunks per row) and reads its fragments there, so the
// product is one launch instead of two; the extra decodes are A.rows * nbp per workgroup
// against 16 * nb of W's.
//
// DOT (with ADEC, when the sums fit 32 bits): no matrix cores.  A's rows go to LDS as int8
// X2 with their blocks' multiples m_A beside them; a lane decodes each of its W blocks to
// int8 X2, forms sum_l X2_W,l X2_A,l with two v_dot4_i32_i8 and adds m_W m_A times it to an
// exact int32 sum (Alg. 4's inner product of the lattice points, times the two multiples).
// The column's sum is the lanes' sum over the four K quarters and the waves.
template <int MT, int ET, int DVW, int NWV, bool ADEC = false, bool DOT = false>
__global__ __launch_bounds__(NWV * 64) void skinny_kernel(const u32x4* __restrict__ ta, int kcb,
                                                          MatmulOperand A, MatmulOperand W,
                                                          int nb, float* __restrict__ c,
                                                          int64_t ldc, float scale) {
  constexpr bool I8 = ET == ET_I8;
  using Acc = typename std::conditional<I8, i32x4, f32x4>::type;
  constexpr int BPL = I8 ? 2 : 1;        // blocks per lane per step
  constexpr int PD = MT <= 2 ? 8 : 4;    // steps per chunk
  constexpr int WPL = PD * BPL;          // code words per lane per chunk (8 or 16, or 4 / 8)
  constexpr int CB = 4 * WPL;            // blocks per chunk
  constexpr uint32_t OOB = 0x80000000u;  // beyond every range below
  __shared__ Acc part[NWV - 1][MT][64];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // uniform: scalar
  const int lane = threadIdx.x & 63;
  const int col = lane & 15, kg = lane >> 4;
  const int64_t n = (int64_t)blockIdx.x * 16 + col;
  const bool nok = n < W.rows;
  const int nbw = (nb + 15) >> 4;
  const __amdgpu_buffer_rsrc_t rc =
      __builtin_amdgcn_make_buffer_rsrc((void*)W.codes, (short)0, (int)(W.rows * nb * 4), 0x00020000);
  const __amdgpu_buffer_rsrc_t rb =
      __builtin_amdgcn_make_buffer_rsrc((void*)W.beta, (short)0, (int)(W.rows * nbw * 4), 0x00020000);
  const __amdgpu_buffer_rsrc_t ra =
      __builtin_amdgcn_make_buffer_rsrc((void*)ta, (short)0, 16 * MT * kcb * 16, 0x00020000);
  const uint32_t cbase = nok ? (uint32_t)(n * nb) * 4u : OOB;
  const uint32_t bbase = nok ? (uint32_t)(n * nbw) * 4u : OOB;

  // chunks of CB blocks; wave w takes a contiguous share of them
  const int nbp = kcb * 16 / (I8 ? 8 : 16);            // padded blocks per row of the A tile
  extern __shared__ __attribute__((aligned(16))) unsigned char alds[];   // ADEC: A's tile
  if constexpr (ADEC) {
    // A's blocks (padding columns read as the zero word, which decodes to zero)
    const int nbwa = (nb + 15) >> 4;
    const int na = (int)A.rows * nbp;
    const int dva = decoder_variant(A.decoder, A.q);
    for (int b = threadIdx.x; b < na; b += NWV * 64) {
      const int r = b >= nbp ? 1 : 0;                   // A.rows <= 2
      const int j = b - r * nbp;
      uint32_t wd = 0u, bw = 0u;
      if (j < nb) {
        wd = A.codes[(int64_t)r * nb + j];
        bw = A.beta[(int64_t)r * nbwa + (j >> 4)];
      }
      const int ma = beta_mult(A.mtab, (bw >> (2 * (j & 15))) & 3u);
      if constexpr (DOT) {
        // NestQuantM at q = 16 through the byte decoder too: its int8 form is one XOR a word
        const u32x2 v = dva == 0 ? decode_x2_i8<0>(wd, A.q, A.m2q)
                                 : decode_x2_i8<1>(wd, A.q, A.m2q);
        *reinterpret_cast<u32x2*>(alds + (r * nbp + j) * 8) = v;
        alds[(int)A.rows * nbp * 8 + r * nbp + j] = (unsigned char)ma;
      } else if constexpr (I8) {
        const u32x2 v = dva == 0 ? decode_tile_i8<0>(wd, ma, A.q, A.m2q)
                                 : (dva == 1 ? decode_tile_i8<1>(wd, ma, A.q, A.m2q)
                                             : decode_tile_i8<2>(wd, ma, A.q, A.m2q));
        *reinterpret_cast<u32x2*>(alds + r * kcb * 16 + j * 8) = v;
      } else {
        constexpr bool F16 = ET == ET_F16;
        const u32x4 v = dva == 0 ? decode_tile_16<0, F16>(wd, ma, A.q, A.m2q)
                                 : (dva == 1 ? decode_tile_16<1, F16>(wd, ma, A.q, A.m2q)
                                             : decode_tile_16<2, F16>(wd, ma, A.q, A.m2q));
        *reinterpret_cast<u32x4*>(alds + (r * kcb + j) * 16) = v;
      }
    }
    __syncthreads();
  }
  const int nch = (nbp + CB - 1) / CB;
  const int c0 = (int)((int64_t)nch * wave / NWV), c1 = (int)((int64_t)nch * (wave + 1) / NWV);

  struct Words {
    uint32_t w[WPL];
    uint32_t b;
  };
  // 16-byte loads when every row starts 16-byte aligned and the chunk lies inside the row;
  // otherwise one word at a time, blocks past the row read as out of range
  const bool rows16 = (nb & 3) == 0;
  auto load_w = [&](int ch, Words& x) {
    const int blk0 = ch * CB + kg * WPL;                 // first block of this lane's quarter
    const uint32_t past = ch < c1 ? 0u : OOB;           // beyond the wave's chunks: nothing
    if (rows16 && ch * CB + CB <= nb) {
#pragma unroll
      for (int v = 0; v < WPL / 4; ++v) {
        const u32x4 q = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                       rc, (cbase + 4u * (uint32_t)(blk0 + 4 * v)) | past, 0, 0));
        x.w[4 * v] = q.x; x.w[4 * v + 1] = q.y; x.w[4 * v + 2] = q.z; x.w[4 * v + 3] = q.w;
      }
    } else {
#pragma unroll
      for (int j = 0; j < WPL; ++j)
        x.w[j] = __builtin_amdgcn_raw_buffer_load_b32(
            rc, (blk0 + j < nb ? cbase + 4u * (uint32_t)(blk0 + j) : OOB) | past, 0, 0);
    }
    x.b = __builtin_amdgcn_raw_buffer_load_b32(rb, (bbase + 4u * (uint32_t)(blk0 >> 4)) | past, 0, 0);
  };

  Acc acc[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) acc[m] = Acc{};

  // A fragments of chunk ch: row 16 m + col, the 16-byte chunk holding the step's blocks
  u32x4 af[PD][MT];
  auto load_a = [&](int ch) {
    const int blk0 = ch * CB + kg * WPL;
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const bool row_ok = 16 * m + col < A.rows;
#pragma unroll
      for (int i = 0; i < PD; ++i) {
        const int blk = blk0 + i * BPL;
        const uint32_t off = (uint32_t)((16 * m + col) * kcb + blk / BPL) * 16u;
        if constexpr (ADEC) {
          af[i][m] = row_ok && blk < nbp ? *reinterpret_cast<const u32x4*>(alds + off)
                                         : u32x4{0u, 0u, 0u, 0u};
        } else {
          af[i][m] = row_ok && blk < nbp
                         ? __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(ra, off, 0, 0))
                         : u32x4{0u, 0u, 0u, 0u};
        }
      }
    }
  };
  int isum[2] = {0, 0};   // DOT: the exact sums of A's rows 0 and 1
  auto compute = [&](int ch, Words& x) {
    const int blk0 = ch * CB + kg * WPL;
    if constexpr (DOT) {
      const int ar = (int)A.rows;
      const unsigned char* mas = alds + ar * nbp * 8;   // m_A of each block
#pragma unroll
      for (int i = 0; i < PD; ++i) {
        const int blk = blk0 + i;
        const u32x2 xw = decode_x2_i8<DVW>(x.w[i], W.q, W.m2q);
        const int mw = beta_mult(W.mtab, (x.b >> (2 * (blk & 15))) & 3u);
        if (blk < nbp) {     // past the padded row: W's words read as 0, nothing to add
#pragma unroll
          for (int r = 0; r < 2; ++r) {
            if (r < ar) {
              const u32x2 xa = *reinterpret_cast<const u32x2*>(alds + (r * nbp + blk) * 8);
              int d = __builtin_amdgcn_sdot4((int)xa.x, (int)xw.x, 0, false);
              d = __builtin_amdgcn_sdot4((int)xa.y, (int)xw.y, d, false);
              isum[r] += __mul24(d, __mul24(mw, (int)mas[r * nbp + blk]));
            }
          }
        }
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < PD; ++i) {
      const int blk = blk0 + i * BPL;
      u32x4 b;
      if constexpr (I8) {
        const u32x2 lo = decode_tile_i8<DVW>(
            x.w[2 * i], beta_mult(W.mtab, (x.b >> (2 * (blk & 15))) & 3u), W.q, W.m2q);
        const u32x2 hi = decode_tile_i8<DVW>(
            x.w[2 * i + 1], beta_mult(W.mtab, (x.b >> (2 * ((blk + 1) & 15))) & 3u), W.q, W.m2q);
        b = u32x4{lo.x, lo.y, hi.x, hi.y};
      } else {
        b = decode_tile_16<DVW, ET == ET_F16>(
            x.w[i], beta_mult(W.mtab, (x.b >> (2 * (blk & 15))) & 3u), W.q, W.m2q);
      }
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        if constexpr (I8) {
          acc[m] = __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, af[i][m]),
                                                         __builtin_bit_cast(i32x4, b), acc[m], 0,
                                                         0, 0);
        } else if constexpr (ET == ET_F16) {
          acc[m] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, af[i][m]),
                                                          __builtin_bit_cast(f16x8, b), acc[m],
                                                          0, 0, 0);
        } else {
          acc[m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, af[i][m]),
                                                           __builtin_bit_cast(bf16x8, b), acc[m],
                                                           0, 0, 0);
        }
      }
    }
  };

  Words x0, x1;
  load_w(c0, x0);
  for (int ch = c0; ch < c1; ch += 2) {
    if constexpr (!DOT) load_a(ch);   // before the next W words: loads complete in order
    load_w(ch + 1, x1);
    compute(ch, x0);
    if (ch + 1 >= c1) break;
    if constexpr (!DOT) load_a(ch + 1);
    load_w(ch + 2, x0);
    compute(ch + 1, x1);
  }

  if constexpr (DOT) {
    // every lane's two sums through LDS; wave 0 adds the waves', then the four K quarters
    // (lanes col, col + 16, col + 32, col + 48), and scales once
    __shared__ int dpart[NWV][2][64];
    dpart[wave][0][lane] = isum[0];
    dpart[wave][1][lane] = isum[1];
    __syncthreads();
    if (wave == 0) {
      const float sw = nok ? W.scales[n] * scale : 0.0f;
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        int v = 0;
#pragma unroll
        for (int w = 0; w < NWV; ++w) v += dpart[w][r][lane];
        v += __shfl_xor(v, 16);
        v += __shfl_xor(v, 32);
        if (kg == 0 && nok && r < A.rows) c[r * ldc + n] = (float)v * (A.scales[r] * sw);
      }
    }
    return;
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
      for (int w = 0; w < NWV - 1; ++w) {
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

// The largest multiple m in an operand's table (its four bytes).
static uint32_t max_mult(uint32_t t) {
  return std::max(std::max(t & 0xFFu, (t >> 8) & 0xFFu), std::max((t >> 16) & 0xFFu, t >> 24));
}

template <int ET>
static hipError_t skinny_launch(const MatmulOperand& A, const MatmulOperand& W, const u32x4* ta,
                                int kcb, int nb, float* c, int64_t ldc, float scale,
                                bool adec, hipStream_t st) {
  const int64_t mp = (A.rows + 15) / 16 * 16;
  const unsigned grid = (unsigned)((W.rows + 15) / 16);
  // the integer-dot GEMV when a row's exact sum fits 32 bits: |X2| <= 2q per coordinate, so
  // |sum| <= nbp * 8 * (2 q_A)(2 q_W) * max m_A * max m_W
  const int nbp = kcb * 16 / (ET == ET_I8 ? 8 : 16);
  const bool dot = adec && ET != ET_I8 &&
                   (double)nbp * 8.0 * (2.0 * A.q) * (2.0 * W.q) * (double)max_mult(A.mtab) *
                           (double)max_mult(W.mtab) < 2147483647.0;
  if (dot) {
    const size_t lds = (size_t)A.rows * nbp * 9;      // int8 X2 (8 bytes) + m_A per block
#define NQ_SKD(DV)                                                                           \
  hipLaunchKernelGGL((skinny_kernel<1, ET, DV, 8, true, true>), dim3(grid), dim3(512), lds,  \
                     st, ta, kcb, A, W, nb, c, ldc, scale)
    // NestQuantM (variants 1 and 2) on the byte decoder: cheaper than decode_word_m16 here,
    // where the int8 form costs one XOR a word against three
    const int dv = decoder_variant(W.decoder, W.q);
    if (dv == 0) NQ_SKD(0); else NQ_SKD(1);
#undef NQ_SKD
    return hipGetLastError();
  }
  if (adec) {
    const size_t lds = (size_t)A.rows * kcb * 16;
#define NQ_SKA(DV)                                                                             \
  hipLaunchKernelGGL((skinny_kernel<1, ET, DV, 8, true>), dim3(grid), dim3(512), lds, st, ta,  \
                     kcb, A, W, nb, c, ldc, scale)
    const int dv = decoder_variant(W.decoder, W.q);
    if (dv == 0) NQ_SKA(0); else if (dv == 1) NQ_SKA(1); else NQ_SKA(2);
#undef NQ_SKA
    return hipGetLastError();
  }
#define NQ_SK(MT, DV)                                                                     \
  hipLaunchKernelGGL((skinny_kernel<MT, ET, DV, 8>), dim3(grid), dim3(512), 0, st, ta, kcb, A, \
                     W, nb, c, ldc, scale)
  const int dvw = decoder_variant(W.decoder, W.q);
#define NQ_SK2(MT) \
  if (dvw == 0) NQ_SK(MT, 0); else if (dvw == 1) NQ_SK(MT, 1); else NQ_SK(MT, 2)
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

template <int ET>
static hipError_t skinny(int stages, const MatmulOperand& A, const MatmulOperand& W, int64_t K,
                         float* c, int64_t ldc, float scale, void* ws, hipStream_t st) {
  const int nb = (int)(K / 8);
  const int64_t mp = (A.rows + 15) / 16 * 16;
  constexpr int EB = ET == ET_I8 ? 1 : 2;
  const int64_t kp = (K * EB + 127) / 128 * 128 / EB;
  const int nbp = (int)(kp / 8);
  const int kcb = (int)(kp * EB / 16);
  u32x4* ta = reinterpret_cast<u32x4*>(ws);
  // one or two activation rows whose tile fits 48 KiB of LDS: the product kernel decodes
  // them itself (no decode stage of its own)
  const bool adec = A.rows <= 2 && A.rows * (int64_t)kcb * 16 <= 49152;
  if ((stages & 1) && !adec) launch_tiles<ET>(A, nb, mp, nbp, (void*)ta, st);
  if (!(stages & 2)) return hipGetLastError();
  // W in column ranges whose code words stay below 2^31 bytes (buffer-load offsets)
  const int64_t max_rows = (((int64_t)1 << 31) - 1) / ((int64_t)nb * 4) / 16 * 16;
  for (int64_t r0 = 0; r0 < W.rows; r0 += max_rows) {
    MatmulOperand Wc = W;
    const int64_t rows = std::min(max_rows, W.rows - r0);
    Wc.codes = W.codes + r0 * nb;
    Wc.beta = W.beta + r0 * ((nb + 15) / 16);
    Wc.scales = W.scales + r0;
    Wc.rows = rows;
    const hipError_t e = skinny_launch<ET>(A, Wc, ta, kcb, nb, c + r0, ldc, scale, adec, st);
    if (e != hipSuccess) return e;
  }
  return hipGetLastError();
}

hipError_t launch_matmul_skinny(int stages, int et, const MatmulOperand& A,
                                const MatmulOperand& W, int64_t K, float* c, int64_t ldc,
                                float scale, void* ws, hipStream_t st) {
  switch (et) {
    case ET_I8: return skinny<ET_I8>(stages, A, W, K, c, ldc, scale, ws, st);
    case ET_F16: return skinny<ET_F16>(stages, A, W, K, c, ldc, scale, ws, st);
    default: return skinny<ET_BF16>(stages, A, W, K, c, ldc, scale, ws, st);
  }
}

}  // namespace nq
