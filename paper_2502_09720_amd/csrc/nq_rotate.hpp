// Online Hadamard rotation of rows (Sec. 5 of the NestQuant paper), the part shared by
// nq_rotate and the encoder that rotates its rows in LDS before coding them (nq_rotate_encode):
// y = x U, with U = H_n / sqrt(n) (Sylvester) for n = 2^k and U = (H_28 kron H_{2^k}) / sqrt(n)
// for n = 28 * 2^k.  The row is read as X[i, j] = x[i 2^k + j] (i < m, m = 1 or 28).
//
// Arithmetic (the paper leaves it open; fixed here so that results are reproducible):
//   1. the fast Walsh-Hadamard transform along j in fp32: for h = 1, 2, 4, ..., every pair
//      (i, i + h) with i & h = 0 becomes (a + b, a - b);
//   2. for m = 28: output a = sum over i = 0..27, in that order, of H_28[i, a] X[i, :];
//   3. every entry times fl32(1 / sqrt(n)).
// Within a stage the butterflies are independent, so any parallel order gives the same
// numbers.
//
// A workgroup of 256 threads holds its rows in LDS as fp32.  Each thread first takes 8
// consecutive entries into registers and does the stages h = 1, 2, 4 there; the later stages
// run four at a time: a thread takes 16 entries whose indices differ in four consecutive
// bits, does those four stages in registers and writes them back (a barrier per four
// stages).  The H_28 signs are compile-time constants, so each term of the mix is one add or
// subtract.
#pragma once

#include "nq_device.hpp"

namespace nq {

// Paley's second construction at q = 13 (q = 1 mod 4): chi the quadratic character mod 13,
// C = [[0, 1^T], [1, Q]] with Q[i][j] = chi(j - i) (14 x 14, symmetric), and
// H_28 = C kron [[1, 1], [1, -1]] + I_14 kron [[1, -1], [-1, -1]].  neg[a] has bit i set
// where H_28[i][a] = -1.
struct H28Table {
  uint32_t neg[28];
};
constexpr H28Table make_h28() {
  H28Table s{};
  int chi[13] = {};
  for (int a = 1; a < 13; ++a) chi[a] = -1;
  for (int v = 1; v < 13; ++v) chi[(v * v) % 13] = 1;
  for (int i = 0; i < 28; ++i)
    for (int a = 0; a < 28; ++a) {
      const int bi = i / 2, ri = i % 2, ba = a / 2, ra = a % 2;
      const int c = (bi == 0 && ba == 0) ? 0
                    : (bi == 0 || ba == 0) ? 1
                    : chi[((ba - 1) - (bi - 1) + 13) % 13];
      const int k2 = (ri == 1 && ra == 1) ? -1 : 1;
      const int d2 = bi == ba ? ((ri == 0 && ra == 0) ? 1 : -1) : 0;
      if (c * k2 + d2 < 0) s.neg[a] |= 1u << i;
    }
  return s;
}
constexpr H28Table kH28 = make_h28();

template <typename T>
__device__ __forceinline__ void load8(const T* __restrict__ p, float (&v)[8]);
template <>
__device__ __forceinline__ void load8<float>(const float* __restrict__ p, float (&v)[8]) {
  const f32x4 a = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
  const f32x4 b = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p) + 1);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
template <>
__device__ __forceinline__ void load8<uint16_t>(const uint16_t* __restrict__ p, float (&v)[8]) {
  const u32x4 a = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(w[i] << 16);
    v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
template <>
__device__ __forceinline__ void load8<_Float16>(const _Float16* __restrict__ p, float (&v)[8]) {
  const u32x4 a = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w[i] & 0xffffu));
    v[2 * i + 1] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w[i] >> 16));
  }
}

// LDS position of entry e: bits 3..5 of e XOR bits 7..9.  The first four-stage pass (stride
// 8 entries) has the 64 lanes of a wave on 8 consecutive entries times 8 groups 128 entries
// apart, which would be 8 banks; the swizzle spreads them over all 64.  It permutes entries
// only within aligned runs of 64, keeps runs of 8 contiguous (the 8-entry loads and stores
// stay vector accesses) and leaves the other passes conflict-free.
__device__ __forceinline__ int lds_pos(int e) { return e ^ (((e >> 7) & 7) << 3); }

// Stages h = 2^b0 .. 2^(b0 + NB - 1) of every length-2^lp segment of buf (total entries):
// each thread takes groups of 2^NB entries whose indices differ only in bits b0 .. b0+NB-1.
template <int NB>
__device__ __forceinline__ void fwht_pass(float* buf, int total, int lp, int b0) {
  constexpr int G = 1 << NB;
  const int per_seg = 1 << (lp - NB);
  for (int g = threadIdx.x; g < (total >> NB); g += 256) {
    const int seg = g >> (lp - NB), lg = g & (per_seg - 1);
    const int base = (seg << lp) | ((lg >> b0) << (b0 + NB)) | (lg & ((1 << b0) - 1));
    float v[G];
#pragma unroll
    for (int r = 0; r < G; ++r) v[r] = buf[lds_pos(base + (r << b0))];
#pragma unroll
    for (int h = 1; h < G; h <<= 1) {
#pragma unroll
      for (int i = 0; i < G; ++i) {
        if ((i & h) == 0) {
          const float a = v[i], b = v[i + h];
          v[i] = a + b;
          v[i + h] = a - b;
        }
      }
    }
#pragma unroll
    for (int r = 0; r < G; ++r) buf[lds_pos(base + (r << b0))] = v[r];
  }
}

// Steps 1 and 2 for the rr consecutive rows at x (n entries each, row stride ld_x), held in
// buf: entry e (row e / n) ends at buf[lds_pos(e)], and its rotated value is that times
// fl32(1 / sqrt(n)).  p = n / m = 2^lp >= 8.  Every thread of the workgroup (256) must call
// it; it ends with a barrier.
template <typename T>
__device__ __forceinline__ void rotate_rows_lds(const T* __restrict__ x, int64_t ld_x, int rr,
                                                int n, int p, int lp, float* buf) {
  const int tid = threadIdx.x;
  const int total = rr * n;   // elements held
  const int m = n / p;
  // load 8 entries at a time, stages h = 1, 2, 4 in registers (p >= 8)
  for (int g = tid; g < total / 8; g += 256) {
    const int e = 8 * g;
    const int r = e / n, c = e - r * n;
    float v[8];
    load8<T>(x + r * ld_x + c, v);
#pragma unroll
    for (int h = 1; h < 8; h <<= 1) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        if ((i & h) == 0) {
          const float a = v[i], b = v[i + h];
          v[i] = a + b;
          v[i + h] = a - b;
        }
      }
    }
    float* d = buf + lds_pos(e);
#pragma unroll
    for (int i = 0; i < 8; ++i) d[i] = v[i];
  }
  // stages h = 8 .. p / 2 along each segment of length p, four at a time
  for (int b0 = 3; b0 < lp; b0 += 4) {
    __syncthreads();
    switch (lp - b0 < 4 ? lp - b0 : 4) {
      case 1: fwht_pass<1>(buf, total, lp, b0); break;
      case 2: fwht_pass<2>(buf, total, lp, b0); break;
      case 3: fwht_pass<3>(buf, total, lp, b0); break;
      default: fwht_pass<4>(buf, total, lp, b0); break;
    }
  }
  __syncthreads();
  if (m == 28) {
    // mix the 28 segments of each row column by column, sums in index order
    for (int q = tid; q < rr * p; q += 256) {
      const int r = q / p, b = q - r * p;
      const int col = r * n + b;
      float xi[28];
#pragma unroll
      for (int i = 0; i < 28; ++i) xi[i] = buf[lds_pos(col + i * p)];
#pragma unroll
      for (int a = 0; a < 28; ++a) {
        float acc = ((kH28.neg[a] & 1u) != 0) ? -xi[0] : xi[0];
#pragma unroll
        for (int i = 1; i < 28; ++i)
          acc = (((kH28.neg[a] >> i) & 1u) != 0) ? acc - xi[i] : acc + xi[i];
        buf[lds_pos(col + a * p)] = acc;
      }
    }
    __syncthreads();
  }
}

}  // namespace nq
