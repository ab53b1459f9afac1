// Decode-once coded matrix product for large M (prefill shapes).
//
// The product C = A_hat W_hat^T is Alg. 4 of the NestQuant paper for every pair of rows.
// With M and N in the thousands, decoding inside every output tile would repeat each
// block's decode N/BN (resp. M/BM) times, and the decode (Alg. 2 + Alg. 5) costs far more
// vector-ALU work per block than the matrix cores spend on it.  So each block is decoded
// exactly once:
//
//   1. tiles_pair_kernel (both operands in one launch; tiles_kernel for one): Alg. 2 on
//      every code word; writes m * X2 (beta = m * base; with the uniform grid m = t and
//      |m X2| <= 128, exact in bf16) as 8 bf16 into a K-contiguous workspace tile,
//      zero-padded to the GEMM tile grid.  Beta sets with larger multiples
//      use fp16 tiles (exact to 2048) and fp16 matrix cores at the same rate.  The
//      workspace (a few tens of MB) stays in the 256 MB Infinity Cache.
//   2. gemm_kernel: bf16 MFMA GEMM (C = T_A T_W^T, fp32 accumulation) with the epilogue
//      C_ij = acc * r_Ai * r_Wj * base_A * base_W / 4.
//
// GEMM tiling (gfx950): a workgroup of NW = WM x WN waves owns a BM x BN tile of C; each
// wave owns (BM/WM) x (BN/WN) as v_mfma_f32_32x32x16_bf16 tiles.  K advances 64 or 32 bf16
// (SB = 128 or 64 B per row) per stage through NSTAGE LDS buffers filled by
// global_load_lds_dwordx4: each wave instruction moves 1 KiB of rows straight into LDS (no
// register staging).  The
// 16-byte chunk c of row r is stored at chunk c ^ swz(r) (see swz), so that the fragment
// reads (32 rows, one chunk) hit distinct LDS banks.  Stage k+NSTAGE-1 is loaded while stage k is
// multiplied.  Workgroups are mapped so that the tiles resident on one XCD (workgroup id
// mod 8) form a compact 4-row band of the tile grid and share their A and W rows in that
// XCD's L2.
#include <type_traits>

#include "nq_device.hpp"
#include "nq_gemm_common.hpp"
#include "nq_kernels.hpp"
#include "nq_tiles.hpp"

namespace nq {

namespace gemm {
constexpr int BK = 64;     // workspace rows are padded to 64 bf16 / 128 int8 ...
constexpr int BKB = kTileRowBytes;   // ... i.e. to whole 128-byte runs (the largest stage row)

// A tile configuration: BM x BN tile, WM x WN waves, NSTAGE LDS buffers of SB bytes of K per
// row (128: 64 bf16; 64: 32 bf16, twice the stages in the same LDS).
template <int BM_, int BN_, int WM_, int WN_, int NSTAGE_, int SB_ = BKB>
struct Cfg {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, NSTAGE = NSTAGE_, SB = SB_;
  static constexpr int NW = WM * WN;
  static constexpr int TM = BM / WM / 32;  // 32x32 MFMA tiles per wave along M
  static constexpr int TN = BN / WN / 32;
  static constexpr int CH = SB / 16;       // 16-byte chunks per row per stage
  static constexpr int STAGE_BYTES = (BM + BN) * SB;
  static constexpr int GROUP_ROWS = 1024 / SB;  // rows moved by one wave load instruction
  static constexpr int GROUPS = (BM + BN) / GROUP_ROWS;
  static constexpr int GROUPS_PER_WAVE = GROUPS / NW;
  static_assert(SB == 128 || SB == 64, "stage rows of 128 or 64 bytes");
  static_assert(GROUPS % NW == 0, "row groups must split evenly over the waves");
  static_assert(NSTAGE * STAGE_BYTES <= 160 * 1024, "LDS is 160 KB");
};

// 256 x 128 tiles (one per CU for the 8B prefill shapes) and 256 x 256 tiles (half the
// global->LDS traffic per flop, for products with at least one tile per CU).  LDS holds two
// stages of the big tile with 128 bytes of K per row, or four with 64 bytes; the deeper
// prefetch of the latter is faster (with two, waves waited on their loads 45% of the time).
// The int8 contraction (half the MFMA time per byte) keeps the two 128-byte stages, which
// measured faster for it.
using CfgMid = Cfg<256, 128, 4, 2, 3>;
using CfgBig = Cfg<256, 256, 4, 2, 4, 64>;
using CfgBigI8 = Cfg<256, 256, 4, 2, 2>;
}  // namespace gemm

// One workgroup per TB blocks of the tile (tiles_block).
template <int ET, int DV, bool FLAT, int TB>
__global__ __launch_bounds__(256) void tiles_kernel(const uint32_t* __restrict__ codes,
                                                    const uint32_t* __restrict__ beta,
                                                    int64_t rows, int nb, int64_t total,
                                                    int nb_p, float inv_nbp, int q,
                                                    uint32_t m2q, uint32_t mtab,
                                                    void* __restrict__ ws) {
  tiles_block<ET, DV, 256, FLAT, TB>(codes, beta, rows, nb, total, nb_p, inv_nbp, q, m2q,
                                     mtab, ws, (int64_t)blockIdx.x);
}

// Launch tiles_kernel for one operand with its decoder.
template <int ET>
void launch_tiles(const MatmulOperand& X, int nb, int64_t rows_p, int nb_p, void* ws,
                  hipStream_t st) {
  const int64_t total = rows_p * nb_p;
  const float inv = 1.0f / (float)nb_p;
  const bool flat = nb_p == nb && (nb & 15) == 0;
  // operands too small to fill the CUs at kTilesPerThread blocks per thread (the decode of a
  // decode-shaped activation) take one block per thread
  const bool small = total < (int64_t)256 * 256 * kTilesPerThread;
  const int64_t wgs = small ? (total + 255) / 256 : tile_workgroups(total);
#define NQ_TL1(DV, F, TB)                                                                    \
  hipLaunchKernelGGL((tiles_kernel<ET, DV, F, TB>), dim3((unsigned)wgs), dim3(256), 0, st,     \
                     X.codes, X.beta, X.rows, nb, total, nb_p, inv, X.q, X.m2q, X.mtab, ws)
#define NQ_TL(DV)                                                                            \
  if (small) {                                                                               \
    if (flat) NQ_TL1(DV, true, 256); else NQ_TL1(DV, false, 256);                            \
  } else {                                                                                   \
    if (flat) NQ_TL1(DV, true, 256 * kTilesPerThread);                                       \
    else NQ_TL1(DV, false, 256 * kTilesPerThread);                                           \
  }
  switch (decoder_variant(X.decoder, X.q)) {
    case 0: NQ_TL(0); break;
    case 1: NQ_TL(1); break;
    default: NQ_TL(2); break;
  }
#undef NQ_TL
#undef NQ_TL1
}
template void launch_tiles<ET_BF16>(const MatmulOperand&, int, int64_t, int, void*, hipStream_t);
template void launch_tiles<ET_F16>(const MatmulOperand&, int, int64_t, int, void*, hipStream_t);
template void launch_tiles<ET_I8>(const MatmulOperand&, int, int64_t, int, void*, hipStream_t);

// Both operands' tiles in one launch: workgroups below a.wgs decode A, the rest W (one
// launch boundary and one tail fewer than two launches).
__global__ __launch_bounds__(256) void tiles_pair_kernel(TileTask a, TileTask w, int et) {
  const int64_t b = blockIdx.x;
  if (b < a.wgs) {
    run_tile_task(a, et, b);
  } else {
    run_tile_task(w, et, b - a.wgs);
  }
}

// Zero blocks of a tile: the flat range [first, first + count) when cols == 0, else the
// blocks nb..nb_p-1 of rows 0..rows-1 (cols = nb_p - nb of them per row).
__global__ __launch_bounds__(256) void tiles_pad_kernel(void* __restrict__ ws, int eb,
                                                        int64_t first, int64_t count, int nb,
                                                        int nb_p, int cols) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= count) return;
  int64_t g = first + t;
  if (cols > 0) {
    const int64_t r = t / cols;
    g = r * nb_p + nb + (t - r * cols);
  }
  if (eb == 16) {
    reinterpret_cast<u32x4*>(ws)[g] = u32x4{0u, 0u, 0u, 0u};
  } else {
    reinterpret_cast<u32x2*>(ws)[g] = u32x2{0u, 0u};
  }
}

hipError_t launch_tiles_pad(int et, void* ws, int64_t rows, int nb, int64_t rows_p, int nb_p,
                            hipStream_t st) {
  const int eb = et == ET_I8 ? 8 : 16;
  if (rows_p > rows) {
    const int64_t count = (rows_p - rows) * nb_p;
    hipLaunchKernelGGL(tiles_pad_kernel, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, st,
                       ws, eb, rows * nb_p, count, nb, nb_p, 0);
  }
  if (nb_p > nb && rows > 0) {
    const int64_t count = rows * (nb_p - nb);
    hipLaunchKernelGGL(tiles_pad_kernel, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, st,
                       ws, eb, (int64_t)0, count, nb, nb_p, nb_p - nb);
  }
  return hipGetLastError();
}

// kc: row length of both tiles in 16-byte chunks (a multiple of 8).  ET: int8 tiles and
// v_mfma_i32_32x32x32_i8 (exact int32 sums), or bf16 / fp16 tiles and
// v_mfma_f32_32x32x16_bf16 / _f16.  All consume 16 B per lane per MFMA, so staging, swizzle
// and fragment reads are the same.
template <class C, int ET>
__global__ __launch_bounds__(C::NW * 64, 1) void gemm_kernel(
    const u32x4* __restrict__ ta, const u32x4* __restrict__ tw, int kc, int tm, int tn,
    const float* __restrict__ ra, const float* __restrict__ rw, int64_t M, int64_t N,
    float* __restrict__ c, int64_t ldc, float scale) {
  constexpr int BM = C::BM, BN = C::BN, WM = C::WM, WN = C::WN, NSTAGE = C::NSTAGE;
  constexpr int NW = C::NW, TM = C::TM, TN = C::TN, STAGE_BYTES = C::STAGE_BYTES;
  constexpr int GROUPS_PER_WAVE = C::GROUPS_PER_WAVE;
  constexpr int CH = C::CH, SB = C::SB, GR = C::GROUP_ROWS;
  constexpr bool I8 = ET == ET_I8;
  extern __shared__ __attribute__((aligned(1024))) unsigned char lds[];

  int pm, pn;
  tile_coords(blockIdx.x, tm, tn, pm, pn);
  const int tid = threadIdx.x;
  // the wave index as a uniform (scalar) value, so that LDS destinations stay scalar
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int wm = wave / WN, wn = wave % WN;

  // This lane's source for each of the wave's row groups: row lane / CH of the group,
  // stored at physical chunk lane % CH, i.e. logical chunk (lane % CH) ^ swz(row).
  const int lrow = lane / CH;
  const u32x4* src[GROUPS_PER_WAVE];
  int dst[GROUPS_PER_WAVE];
#pragma unroll
  for (int i = 0; i < GROUPS_PER_WAVE; ++i) {
    const int grp = wave + i * NW;              // 0 .. GROUPS-1; A groups first
    const int row = grp * GR + lrow;            // row within the stage (A rows, then W rows)
    const int lchunk = (lane % CH) ^ swz<CH>(row);
    if (grp < BM / GR) {
      src[i] = ta + ((int64_t)pm * BM + row) * kc + lchunk;
    } else {
      src[i] = tw + ((int64_t)pn * BN + (row - BM)) * kc + lchunk;
    }
    dst[i] = grp * 1024;                        // GR rows x SB bytes
  }
  auto load_stage = [&](int ks) {
    unsigned char* base = lds + (ks % NSTAGE) * STAGE_BYTES;
#pragma unroll
    for (int i = 0; i < GROUPS_PER_WAVE; ++i)
      __builtin_amdgcn_global_load_lds((const void*)(src[i] + ks * CH),
                                       (lds_void*)(base + dst[i]), 16, 0, 0);
  };

  using Acc = typename std::conditional<I8, i32x16, f32x16>::type;
  Acc acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = Acc{};

  // fragment reads: row (lane & 31) of a 32-row tile, logical chunk 2 kk + (lane >> 5).  The
  // swizzle depends only on the row modulo 32, and every 32-row tile starts at a multiple
  // of 32, so one offset per kk serves all of this lane's A and W tiles.
  const int frow = lane & 31;
  const int abase = (wm * (BM / WM) + frow) * SB;
  const int wbase = BM * SB + (wn * (BN / WN) + frow) * SB;
  int coff[CH / 2];
#pragma unroll
  for (int kk = 0; kk < CH / 2; ++kk) coff[kk] = ((2 * kk + (lane >> 5)) ^ swz<CH>(frow)) * 16;

  const int nks = kc / CH;
#pragma unroll
  for (int s = 0; s < NSTAGE - 1; ++s)
    if (s < nks) load_stage(s);

  // Row and column scales of this lane's outputs.  32x32 accumulator layout: lane l holds
  // column l % 32; register e holds row 8 (e / 4) + 4 (l / 32) + (e % 4).  Indices are
  // clamped into range (M, N >= 1).  The 256 x 128 tile fetches them before the main loop,
  // so that the epilogue issues only stores; the 256 x 256 tile's accumulators and
  // fragments leave no room to hold them through the loop (they were spilled to scratch and
  // reloaded in every stage), so it fetches them after the loop.
  constexpr bool EARLY_SCALES = BN <= 128;
  const int64_t m0 = (int64_t)pm * BM + wm * (BM / WM) + 4 * (lane >> 5);
  const int64_t n0 = (int64_t)pn * BN + wn * (BN / WN) + (lane & 31);
  float rs[TM][16], cs[TN];
  auto fetch_scales = [&]() {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int64_t row = m0 + i * 32 + 8 * (e >> 2) + (e & 3);
        rs[i][e] = ra[row < M ? row : M - 1];
      }
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int64_t col = n0 + j * 32;
      cs[j] = rw[col < N ? col : N - 1] * scale;
    }
  };
  if constexpr (EARLY_SCALES) fetch_scales();

  // One stage; PF: the loads of stage ks + NSTAGE - 1 are issued (every stage but the last
  // NSTAGE - 1), a compile-time flag so that the steady-state loop has no branches.
  auto stage = [&](int ks, auto pf) {
    constexpr bool PF = decltype(pf)::value;
    // stage ks has landed when at most the later stages' loads are outstanding
    if (PF || ks + NSTAGE - 2 < nks) {
      __builtin_amdgcn_s_waitcnt((GROUPS_PER_WAVE * (NSTAGE - 2)) | (0x7 << 4) | (0xF << 8));
    } else {
      __builtin_amdgcn_s_waitcnt(0 | (0x7 << 4) | (0xF << 8));
    }
    // Barrier without a memory fence: a fence would wait for every outstanding LDS DMA,
    // including the stages still being prefetched.  Each wave has waited for its own
    // loads of stage ks above, and its reads of the buffer reloaded below finished before
    // the MFMAs that consumed them.  The signal fences keep the compiler from moving LDS
    // accesses across the barrier.
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    constexpr bool prefetch = PF;
    unsigned char* nb = lds + ((ks + NSTAGE - 1) % NSTAGE) * STAGE_BYTES;
    const unsigned char* sb = lds + (ks % NSTAGE) * STAGE_BYTES;
    // Fragments are double-buffered in registers.  Within a step the MFMAs are interleaved
    // one by one with the LDS reads of the next step and with this wave's share of the
    // next stage's global loads, so that neither the LDS nor the texture path receives
    // its requests in one burst that would hold up the MFMA issue.
    u32x4 af[2][TM], bfr[2][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
      af[0][i] = *reinterpret_cast<const u32x4*>(sb + abase + i * 32 * SB + coff[0]);
#pragma unroll
    for (int j = 0; j < TN; ++j)
      bfr[0][j] = *reinterpret_cast<const u32x4*>(sb + wbase + j * 32 * SB + coff[0]);
    constexpr int KSTEPS = CH / 2;  // MFMAs per (i, j) per stage: 32 B of K each
    constexpr int LOADS_PER_STEP = (GROUPS_PER_WAVE + KSTEPS - 1) / KSTEPS;
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) {
      const int cur = kk & 1;
#pragma unroll
      for (int m = 0; m < TM * TN; ++m) {
        const int i = m / TN, j = m % TN;
        if constexpr (I8) {
          acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(
              __builtin_bit_cast(i32x4, af[cur][i]), __builtin_bit_cast(i32x4, bfr[cur][j]),
              acc[i][j], 0, 0, 0);
        } else if constexpr (ET == ET_F16) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(
              __builtin_bit_cast(f16x8, af[cur][i]), __builtin_bit_cast(f16x8, bfr[cur][j]),
              acc[i][j], 0, 0, 0);
        } else {
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8, af[cur][i]), __builtin_bit_cast(bf16x8, bfr[cur][j]),
              acc[i][j], 0, 0, 0);
        }
        if (kk + 1 < KSTEPS) {
          if (m < TM) {
            af[cur ^ 1][m] = *reinterpret_cast<const u32x4*>(sb + abase + m * 32 * SB + coff[kk + 1]);
          } else if (m < TM + TN) {
            bfr[cur ^ 1][m - TM] = *reinterpret_cast<const u32x4*>(sb + wbase + (m - TM) * 32 * SB + coff[kk + 1]);
          }
        }
        const int g = kk * LOADS_PER_STEP + m;
        if (prefetch && m < LOADS_PER_STEP && g < GROUPS_PER_WAVE)
          __builtin_amdgcn_global_load_lds((const void*)(src[g] + (ks + NSTAGE - 1) * CH),
                                           (lds_void*)(nb + dst[g]), 16, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
      // reads and loads left over when a step has fewer MFMAs than them
#pragma unroll
      for (int m = TM * TN; m < TM + TN || m < LOADS_PER_STEP; ++m) {
        if (kk + 1 < KSTEPS) {
          if (m < TM) {
            af[cur ^ 1][m] = *reinterpret_cast<const u32x4*>(sb + abase + m * 32 * SB + coff[kk + 1]);
          } else if (m < TM + TN) {
            bfr[cur ^ 1][m - TM] = *reinterpret_cast<const u32x4*>(sb + wbase + (m - TM) * 32 * SB + coff[kk + 1]);
          }
        }
        const int g = kk * LOADS_PER_STEP + m;
        if (prefetch && m < LOADS_PER_STEP && g < GROUPS_PER_WAVE)
          __builtin_amdgcn_global_load_lds((const void*)(src[g] + (ks + NSTAGE - 1) * CH),
                                           (lds_void*)(nb + dst[g]), 16, 0, 0);
      }
    }
  };
  int ks = 0;
  for (; ks < nks - (NSTAGE - 1); ++ks) stage(ks, std::true_type{});
  for (; ks < nks; ++ks) stage(ks, std::false_type{});

  if constexpr (!EARLY_SCALES) fetch_scales();

  // Epilogue: C = acc * r_A * (r_W * scale); whole tiles skip the bounds tests.  C is
  // written once and not read here, so its stores are nontemporal (streamed past the
  // caches: 2% off the contraction).
  float* cp = c + m0 * ldc + n0;
  const bool whole = m0 - 4 * (lane >> 5) + BM / WM <= M && n0 - (lane & 31) + BN / WN <= N;
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int r = i * 32 + 8 * (e >> 2) + (e & 3);
        if (whole || (m0 + r < M && n0 + j * 32 < N))
          __builtin_nontemporal_store((float)acc[i][j][e] * (rs[i][e] * cs[j]),
                                      &cp[r * ldc + j * 32]);
      }
}

template <class C, int ET>
static void launch_gemm(const u32x4* wa, const u32x4* ww, int kc, int64_t mp, int64_t np,
                        const MatmulOperand& A, const MatmulOperand& W, float* c, int64_t ldc,
                        float scale, hipStream_t st) {
  const int tm = (int)(mp / C::BM), tn = (int)(np / C::BN);
  hipLaunchKernelGGL((gemm_kernel<C, ET>), dim3((unsigned)(tm * tn)), dim3(C::NW * 64),
                     (size_t)C::NSTAGE * C::STAGE_BYTES, st, wa, ww, kc, tm, tn, A.scales,
                     W.scales, A.rows, W.rows, c, ldc, scale);
}

template <int ET>
static hipError_t decode_once(int stages, const MatmulOperand& A, const MatmulOperand& W,
                              int64_t K, float* c, int64_t ldc, float scale, void* ws,
                              hipStream_t st) {
  using namespace gemm;
  const int nb = (int)(K / 8);
  const int64_t mp = (A.rows + 255) / 256 * 256;
  int64_t w_offset, np;
  int nbp;
  decode_once_layout(ET, A.rows, W.rows, K, w_offset, np, nbp);
  constexpr int EB = ET == ET_I8 ? 1 : 2;              // bytes per element
  const int kc = nbp * 8 * EB / 16;
  u32x4* wa = reinterpret_cast<u32x4*>(ws);
  u32x4* ww = reinterpret_cast<u32x4*>(static_cast<unsigned char*>(ws) + w_offset);
  if (stages & 1) {
    const TileTask ta = tile_task(A, nb, mp, nbp, (void*)wa);
    const TileTask tw = tile_task(W, nb, np, nbp, (void*)ww);
    hipLaunchKernelGGL(tiles_pair_kernel, dim3((unsigned)(ta.wgs + tw.wgs)), dim3(256), 0, st,
                       ta, tw, ET);
  } else if (stages & kStageDecodeW) {
    launch_tiles<ET>(W, nb, np, nbp, (void*)ww, st);
  }
  if (!(stages & 2)) return hipGetLastError();
  // 256 x 256 tiles (half the global->LDS traffic per flop) unless they leave a partly
  // empty last round over the 256 CUs that 256 x 128 tiles (half the work each) avoid
  const int64_t big = (mp / 256) * (np / 256), mid = (mp / 256) * (np / 128);
  if (big >= 256 && 2 * ((big + 255) / 256) <= (mid + 255) / 256) {
    using Big = typename std::conditional<ET == ET_I8, CfgBigI8, CfgBig>::type;
    launch_gemm<Big, ET>(wa, ww, kc, mp, np, A, W, c, ldc, scale, st);
  } else {
    launch_gemm<CfgMid, ET>(wa, ww, kc, mp, np, A, W, c, ldc, scale, st);
  }
  return hipGetLastError();
}

hipError_t launch_matmul_decode_once(int stages, int et, const MatmulOperand& A,
                                     const MatmulOperand& W, int64_t K, float* c, int64_t ldc,
                                     float scale, void* ws, hipStream_t st) {
  switch (et) {
    case ET_I8: return decode_once<ET_I8>(stages, A, W, K, c, ldc, scale, ws, st);
    case ET_F16: return decode_once<ET_F16>(stages, A, W, K, c, ldc, scale, ws, st);
    default: return decode_once<ET_BF16>(stages, A, W, K, c, ldc, scale, ws, st);
  }
}

hipError_t gemm_set_attributes() {
  using namespace gemm;
  const void* k[6] = {(const void*)gemm_kernel<CfgMid, ET_BF16>, (const void*)gemm_kernel<CfgMid, ET_F16>,
                      (const void*)gemm_kernel<CfgMid, ET_I8>, (const void*)gemm_kernel<CfgBig, ET_BF16>,
                      (const void*)gemm_kernel<CfgBig, ET_F16>, (const void*)gemm_kernel<CfgBigI8, ET_I8>};
  constexpr int mid = CfgMid::NSTAGE * CfgMid::STAGE_BYTES, big = CfgBig::NSTAGE * CfgBig::STAGE_BYTES;
  constexpr int big8 = CfgBigI8::NSTAGE * CfgBigI8::STAGE_BYTES;
  const int bytes[6] = {mid, mid, mid, big, big, big8};
  for (int i = 0; i < 6; ++i) {
    const hipError_t e = hipFuncSetAttribute(k[i], hipFuncAttributeMaxDynamicSharedMemorySize, bytes[i]);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace nq
