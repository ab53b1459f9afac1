// Online Hadamard rotation of rows (Sec. 5 of the NestQuant paper), the part shared by
// nq_rotate and the encoder that rotates its rows in LDS before coding them (nq_rotate_encode):
// y = x U, with U = H_n / sqrt(n) (Sylvester) for n = 2^k and U = (H_28 kron H_{2^k}) / sqrt(n)
// for n = 28 * 2^k.  The row is read as X[i, j] = x[i 2^k + j] (i < m, m = 1 or 28).
//
// Arithmetic (the paper leaves it open; fixed here so that results are reproducible):
//   1. the fast Walsh-Hadamard transform along j in fp32: for h = 1, 2, 4, ..., every pair
//      (i, i + h) with i & h = 0 becomes (a + b, a - b);
//   2. for m = 28, output segment a = the sum over i = 0..27, in increasing i, of
//      H_28[i][a] X_i (the plain product with the order-28 factor, one rounding per
//      addition, starting from H_28[0][a] X_0);
//   3. every entry times fl32(1 / sqrt(n)).
// Within a stage the butterflies are independent, so any parallel order gives the same
// numbers.
//
// A workgroup of NT threads holds its rows in LDS as fp32.  Each thread first takes 8
// consecutive entries into registers and does the stages h = 1, 2, 4 there; the later stages
// run four at a time: a thread takes 16 entries whose indices differ in four consecutive
// bits, does those four stages in registers and writes them back (a barrier per four
// stages).  The signs of H_28 are compile-time constants, so each term of the mix is one
// add or subtract.
#pragma once

#include "nq_device.hpp"

namespace nq {

// Paley's second construction at q = 13 (q = 1 mod 4): chi the quadratic character mod 13,
// the symmetric conference matrix C = [[0, 1^T], [1, Q]] with Q[i][j] = chi(j - i) (14 x 14,
// zero diagonal), and H_28 = C kron [[1, 1], [1, -1]] + I_14 kron [[1, -1], [-1, -1]].
// neg[a] has bit i set where H_28[i][a] = -1.
struct H28Table {
  uint32_t neg[28];
};
constexpr H28Table make_h28() {
  H28Table t{};
  int chi[13] = {};
  for (int a = 1; a < 13; ++a) chi[a] = -1;
  for (int v = 1; v < 13; ++v) chi[(v * v) % 13] = 1;
  int C[14][14] = {};
  for (int b = 0; b < 14; ++b)
    for (int c = 0; c < 14; ++c)
      C[b][c] = b == c ? 0 : (b == 0 || c == 0) ? 1 : chi[((c - 1) - (b - 1) + 13) % 13];
  const int H2[2][2] = {{1, 1}, {1, -1}}, K2[2][2] = {{1, -1}, {-1, -1}};
  for (int i = 0; i < 28; ++i)
    for (int a = 0; a < 28; ++a) {
      const int b = i / 2, r = i % 2, c = a / 2, s = a % 2;
      const int v = C[b][c] * H2[r][s] + (b == c ? K2[r][s] : 0);
      if (v < 0) t.neg[a] |= 1u << i;
    }
  return t;
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

// LDS position of entry e: bits 3..5 of e XOR bits 7..9, and bits 0..2 XOR (bit 5 ^ bit 8,
// bit 6, bit 7).  It permutes entries only within aligned runs of 64, and an aligned run of 8
// within itself (lds_pos(e + l) = lds_pos(e) ^ l for e a multiple of 8, l < 8).  Each access
// pattern below then puts the 64 lanes of a wave on 64 distinct banks, and each half-wave on
// 32 distinct banks modulo 32: a lane per 8-entry block, every lane on the same entry of its
// block (bits 3..8 from the lane; unswizzled, 8 lanes per bank); the first four-stage pass
// (bits 0..2 and 7..9 from the lane); the later passes and the H_28 mix (bits 0..5 from the
// lane).
__device__ __forceinline__ int lds_pos(int e) {
  return e ^ (((e >> 7) & 7) << 3) ^ (((e >> 5) ^ (e >> 8)) & 1) ^ (((e >> 6) & 3) << 1);
}

// lds_pos is linear over XOR: lds_pos(a ^ b) = lds_pos(a) ^ lds_pos(b).  So where an index is
// a base plus bits the base does not use, its position is the base's position XOR a
// constant, one instruction per access.

// Stages h = 2^B0 .. 2^(B0 + NB - 1) of every length-2^lp segment of buf (total entries):
// each thread takes groups of 2^NB entries whose indices differ only in bits B0 .. B0+NB-1.
template <int NB, int B0, int NT>
__device__ __forceinline__ void fwht_pass(float* buf, int total, int lp) {
  constexpr int G = 1 << NB;
  const int per_seg = 1 << (lp - NB);
  for (int g = threadIdx.x; g < (total >> NB); g += NT) {
    const int seg = g >> (lp - NB), lg = g & (per_seg - 1);
    const int base = (seg << lp) | ((lg >> B0) << (B0 + NB)) | (lg & ((1 << B0) - 1));
    const int pb = lds_pos(base);
    float v[G];
#pragma unroll
    for (int r = 0; r < G; ++r) v[r] = buf[pb ^ lds_pos(r << B0)];
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
    for (int r = 0; r < G; ++r) buf[pb ^ lds_pos(r << B0)] = v[r];
  }
}

// The pass over bits B0 .. min(B0 + 3, top - 1) of segments of length 2^lp, after a
// barrier, if top > B0.
template <int B0, int NT>
__device__ __forceinline__ void fwht_pass_at(float* buf, int total, int lp, int top) {
  if (top <= B0) return;
  __syncthreads();
  switch (top - B0 < 4 ? top - B0 : 4) {
    case 1: fwht_pass<1, B0, NT>(buf, total, lp); break;
    case 2: fwht_pass<2, B0, NT>(buf, total, lp); break;
    case 3: fwht_pass<3, B0, NT>(buf, total, lp); break;
    default: fwht_pass<4, B0, NT>(buf, total, lp); break;
  }
}

// The H_28 factor for column b (< p) of row r of buf: output segment a is the sum over
// i = 0..27, in increasing i, of H_28[i][a] X_i (27 additions per output).  Entry k of the
// column is r n + k p + b = (28 r + k) p | b.
__device__ __forceinline__ void mix28_column(float* buf, int b, int r, int p) {
  const int pb = lds_pos(b);
  auto at = [&](int k) -> float& { return buf[pb ^ lds_pos((28 * r + k) * p)]; };
  float x[28];
#pragma unroll
  for (int i = 0; i < 28; ++i) x[i] = at(i);
#pragma unroll
  for (int a = 0; a < 28; ++a) {
    float acc = (kH28.neg[a] & 1u) != 0 ? -x[0] : x[0];
#pragma unroll
    for (int i = 1; i < 28; ++i) acc = ((kH28.neg[a] >> i) & 1u) != 0 ? acc - x[i] : acc + x[i];
    at(a) = acc;
  }
}

// Steps 1 and 2 for the rr consecutive rows at x (n entries each, row stride ld_x), held in
// buf: entry e (row e / n) ends at buf[lds_pos(e)], and its rotated value is that times
// fl32(1 / sqrt(n)).  p = n / m = 2^lp >= 8.  Every thread of the workgroup (NT) must call
// it; it ends with a barrier.
//
// LAST_OUT (n = p = 2^lp with lp = 4, 8 or 12, where the last pass would hold a single
// stage): that stage, h = p / 2, is left to the caller, which applies it as it reads the
// entries out (rotate_last_stage); the function returns h then, else 0.
template <typename T, int NT = 256, bool LAST_OUT = false>
__device__ __forceinline__ int rotate_rows_lds(const T* __restrict__ x, int64_t ld_x, int rr,
                                               int n, int p, int lp, float* buf) {
  const int tid = threadIdx.x;
  const int total = rr * n;   // elements held
  const int m = n / p;
  // load 8 entries at a time, stages h = 1, 2, 4 in registers (p >= 8)
  auto first = [&](int e, int r, int c) {
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
    const int pe = lds_pos(e);
#pragma unroll
    for (int i = 0; i < 8; ++i) buf[pe ^ i] = v[i];
  };
  if (rr == 1) {
    for (int e = 8 * tid; e < n; e += 8 * NT) first(e, 0, e);
  } else {
    for (int e = 8 * tid; e < total; e += 8 * NT) {
      const int r = e / n;
      first(e, r, e - r * n);
    }
  }
  // stages h = 8 .. p / 2 along each segment of length p, four at a time (p <= 2^15)
  const bool defer = LAST_OUT && m == 1 && (lp == 4 || lp == 8 || lp == 12);
  const int top = defer ? lp - 1 : lp;   // stages below 2^top here
  fwht_pass_at<3, NT>(buf, total, lp, top);
  fwht_pass_at<7, NT>(buf, total, lp, top);
  fwht_pass_at<11, NT>(buf, total, lp, top);
  __syncthreads();
  if (defer) return p / 2;
  if (m == 28) {
    // the H_28 factor, column by column
    if (rr == 1) {
      for (int b = tid; b < p; b += NT) mix28_column(buf, b, 0, p);
    } else {
      for (int q = tid; q < rr * p; q += NT) {
        const int r = q / p;
        mix28_column(buf, q - r * p, r, p);
      }
    }
    __syncthreads();
  }
  return 0;
}

}  // namespace nq
