// Decode of a coded operand into the product's integer tiles (m * X2 per block, Alg. 2 +
// Alg. 5 on every code word), one workgroup's share at a time.  tiles_kernel runs it as a
// launch of its own; the fused encode-and-multiply runs W's share as the last workgroups of
// the encoder's grid (TileTask), where they fill the CUs the encoder's last rows leave idle
// and save a launch.
#pragma once

#include <type_traits>

#include "nq_device.hpp"
#include "nq_kernels.hpp"

namespace nq {

// m * X2 of every block of a coded operand into ws[rows_p][nb_p blocks] (zero padding): 8
// bf16 or fp16 (16 B) per block, or 8 int8 (8 B) for the int8 contraction.  The workspace
// is one flat array of rows_p * nb_p blocks; workgroup w covers TB consecutive blocks of it
// with NT threads, thread t the blocks w TB + t + NT i (i < TPB = TB / NT), so each load
// and store instruction of a wave touches consecutive blocks.  A thread splits its first
// block's position into (row, column) once and steps the split by NT blocks for the next
// ones.  Every thread issues the loads of all its blocks before decoding any, which keeps
// TPB loads in flight per thread.  TB is 256 * kTilesPerThread, or 256 for an operand too
// small to fill the CUs (its launch is bound by the latency of one thread's decodes).
// FLAT: no padding columns (nb_p == nb) and nb a multiple of 16, so that the code words
// and beta words of a workgroup's blocks are consecutive and no block needs its (row,
// column); the callers pick it at run time.
template <int ET, int DV, int NT = 256, bool FLAT = false, int TB = 256 * kTilesPerThread>
__device__ __forceinline__ void tiles_block(const uint32_t* __restrict__ codes,
                                            const uint32_t* __restrict__ beta, int64_t rows,
                                            int nb, int64_t total, int nb_p, float inv_nbp,
                                            int q, uint32_t m2q, uint32_t mtab,
                                            void* __restrict__ ws, int64_t wg) {
  constexpr bool I8 = ET == ET_I8;
  constexpr int TPB = TB / NT;                // blocks per thread
  static_assert(TPB * NT == TB, "NT divides the workgroup's blocks");
  constexpr uint32_t OOB = 0x80000000u;   // past every buffer range below: reads 0
  using V = typename std::conditional<I8, u32x2, u32x4>::type;
  const int64_t g0 = wg * TB;
  if (g0 >= rows * (int64_t)nb_p) {
    // a workgroup of padding rows only (past the operand): zero tiles, nothing to read
#pragma unroll
    for (int i = 0; i < TPB; ++i) {
      const int64_t g = g0 + (int)threadIdx.x + NT * i;
      if (g < total) reinterpret_cast<V*>(ws)[g] = V{};
    }
    return;
  }
  // the workgroup's first block as (row0, j0); every other block is an offset
  // o < nb_p + TB <= 2^14 past (row0, 0).  Code and beta words are read through buffer
  // resources based at row0 (32-bit offsets; the range check makes rows past the operand
  // read as zero).
  const int64_t row0 = g0 / nb_p;
  const int j0 = (int)(g0 - row0 * nb_p);
  const int nbw = (nb + 15) >> 4;
  const int64_t rows_left = rows > row0 ? rows - row0 : 0;
  const int reach = (j0 + TB + nb_p - 1) / nb_p;            // rows this workgroup touches
  const int64_t span = rows_left < reach ? rows_left : reach;
  const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(codes + row0 * nb), (short)0, (int)(span * nb * 4), 0x00020000);
  const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(beta + row0 * nbw), (short)0, (int)(span * nbw * 4), 0x00020000);
  // the first block's (row, column) by a float division checked once in each direction;
  // each further block is NT blocks on: dr rows and dj columns more, with one carry
  const int o = j0 + (int)threadIdx.x;
  int r = (int)((float)o * inv_nbp);
  if ((int)__umul24((uint32_t)r, (uint32_t)nb_p) > o) --r;
  if ((int)__umul24((uint32_t)(r + 1), (uint32_t)nb_p) <= o) ++r;
  int j = o - (int)__umul24((uint32_t)r, (uint32_t)nb_p);
  const int dr = NT / nb_p, dj = NT - dr * nb_p;
  uint32_t w[TPB], bw[TPB];
  int sh[TPB];   // bit position of the block's beta index in its beta word
  if constexpr (FLAT) {
    // block i of this thread is code word o + NT i and beta word o / 16 + NT i / 16, at
    // bits 2 (o mod 16); blocks past the operand's rows lie past both buffer ranges
#pragma unroll
    for (int i = 0; i < TPB; ++i) {
      sh[i] = 2 * (o & 15);
      w[i] = __builtin_amdgcn_raw_buffer_load_b32(rc, 4u * (uint32_t)o + 4u * NT * i, 0, 0);
      bw[i] = __builtin_amdgcn_raw_buffer_load_b32(
          rb, 4u * (uint32_t)(o >> 4) + 4u * (NT / 16) * i, 0, 0);
    }
  } else {
    // Without padding columns (nb_p == nb) the code words are still consecutive (block i
    // of this thread is word o + NT i) and a block past the operand's rows lies past the
    // end of both buffer ranges, so no offset needs a select.
    auto load = [&](auto dense) {
#pragma unroll
      for (int i = 0; i < TPB; ++i) {
        if (i > 0) {
          j += dj;
          r += dr;
          if (j >= nb_p) {
            j -= nb_p;
            ++r;
          }
        }
        sh[i] = 2 * (j & 15);
        uint32_t co, bo;
        if constexpr (decltype(dense)::value) {
          co = 4u * (uint32_t)o + 4u * NT * i;
          bo = 4u * (__umul24((uint32_t)r, (uint32_t)nbw) + (uint32_t)(j >> 4));
        } else {
          const bool pad = j >= nb || r >= span;
          co = pad ? OOB : 4u * (__umul24((uint32_t)r, (uint32_t)nb) + (uint32_t)j);
          bo = pad ? OOB : 4u * (__umul24((uint32_t)r, (uint32_t)nbw) + (uint32_t)(j >> 4));
        }
        w[i] = __builtin_amdgcn_raw_buffer_load_b32(rc, co, 0, 0);
        bw[i] = __builtin_amdgcn_raw_buffer_load_b32(rb, bo, 0, 0);
      }
    };
    if (nb_p == nb) {
      load(std::true_type{});
    } else {
      load(std::false_type{});
    }
  }
  // blocks of this thread inside the workspace: block i exists iff NT i < left
  const int64_t left64 = total - g0 - (int64_t)threadIdx.x;
  const int left = left64 > TB ? TB : (int)left64;
  V* __restrict__ dst = reinterpret_cast<V*>(ws) + g0 + (int)threadIdx.x;
#pragma unroll
  for (int i = 0; i < TPB; ++i) {
    if (NT * i >= left) break;
    const int m = beta_mult(mtab, (bw[i] >> sh[i]) & 3u);
    V out;
    if constexpr (I8) {
      out = decode_tile_i8<DV>(w[i], m, q, m2q);
    } else {
      out = decode_tile_16<DV, ET == ET_F16>(w[i], m, q, m2q);
    }
    // padding past the operand's rows or columns read the word 0 (out of range), which
    // decodes to the zero point: its tile is zero
    dst[NT * i] = out;
  }
}

// Workgroup wg of a TileTask (NT threads), with the element type and decoder chosen at run
// time (uniform over the workgroup).
template <int NT = 256>
__device__ __forceinline__ void run_tile_task(const TileTask& t, int et, int64_t wg) {
  // the flat instantiation for the tile kernels' 256-thread workgroups only: in the
  // encoder's two-wave workgroups the general one measured faster (q_proj step 95.0-95.7
  // against 97.6-98.3 us on one box), and the encoder kernel keeps one instance per type
  const bool flat = NT == 256 && t.nb_p == t.nb && (t.nb & 15) == 0;
#define NQ_TB(ET, DV)                                                                     \
  if (flat)                                                                               \
    tiles_block<ET, DV, NT, NT == 256>(t.codes, t.beta, t.rows, t.nb, t.total, t.nb_p,    \
                                       t.inv_nbp, t.q, t.m2q, t.mtab, t.ws, wg);          \
  else                                                                                    \
    tiles_block<ET, DV, NT, false>(t.codes, t.beta, t.rows, t.nb, t.total, t.nb_p,        \
                                   t.inv_nbp, t.q, t.m2q, t.mtab, t.ws, wg)
  switch (et * 3 + t.dv) {
    case 0: NQ_TB(ET_BF16, 0); break;
    case 1: NQ_TB(ET_BF16, 1); break;
    case 2: NQ_TB(ET_BF16, 2); break;
    case 3: NQ_TB(ET_F16, 0); break;
    case 4: NQ_TB(ET_F16, 1); break;
    case 5: NQ_TB(ET_F16, 2); break;
    case 6: NQ_TB(ET_I8, 0); break;
    case 7: NQ_TB(ET_I8, 1); break;
    default: NQ_TB(ET_I8, 2); break;
  }
#undef NQ_TB
}

}  // namespace nq
