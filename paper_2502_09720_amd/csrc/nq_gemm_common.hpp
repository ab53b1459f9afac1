// Pieces shared by the matrix-core products (decode-once GEMM and the in-tile decode GEMM):
// fragment types, the XCD-aware tile order and the LDS swizzle of 16-byte chunks.
#pragma once

#include "nq_device.hpp"

namespace nq {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;

// Bands of this many tile rows share their operand rows in one XCD's L2 (tile_coords).
constexpr int kGroupM = 4;

// Tile (pm, pn) of workgroup bid in a tm x tn grid.  Workgroups bid, bid + 8, ... run on one
// XCD; they are numbered consecutively here and laid over bands of kGroupM tile rows, so that
// the tiles resident on one XCD share A and W rows in its L2.
__device__ __forceinline__ void tile_coords(int bid, int tm, int tn, int& pm, int& pn) {
  constexpr int GROUP_M = kGroupM;
  // XCD-contiguous numbering: workgroups bid, bid+8, ... run on one XCD
  const int total = tm * tn;
  int t = bid;
  if ((total & 7) == 0) t = (bid & 7) * (total >> 3) + (bid >> 3);
  const int width = GROUP_M * tn;
  const int g = t / width;
  const int first = g * GROUP_M;
  const int gm = min(tm - first, GROUP_M);
  const int r = t - g * width;
  pm = first + r % gm;
  pn = r / gm;
}


// LDS swizzle: chunk c of row r lives at chunk c ^ swz(r).  128-byte rows (8 chunks):
// swz(r) = (r mod 8) ^ ((r / 8) mod 4), a function of r mod 32 only (every 32-row MFMA tile
// starts at a multiple of 32); the 16-byte fragment reads of 32 consecutive rows at one
// logical chunk then fall in distinct bank groups whether the LDS serves 8, 16 or 32 lanes
// of a 128-bit read per cycle.  64-byte rows (4 chunks, four rows per 256-byte bank period):
// swz(r) = (r / 4) mod 4, so that any 16 consecutive rows cover all 64 banks.
template <int CH>
__device__ __forceinline__ int swz(int r) {
  if constexpr (CH == 8) {
    return (r ^ ((r >> 3) & 3)) & 7;
  } else {
    return (r >> 2) & 3;
  }
}

}  // namespace nq
