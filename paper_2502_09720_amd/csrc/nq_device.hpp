// Device primitives shared by the NestQuant kernels (gfx950).
//
// Lattice conventions (App. E of the NestQuant paper): E8 points are carried as integer
// vectors P = 2p in 2E8, and G is the generator of 2E8 whose rows give
//   X0 = c0, X1 = c0 + 2c2, X2 = c0 + 2c4, X3 = c0 + 2c6, X4 = c0 + 4c1 + 2(c2 + ... + c7),
//   X5 = c0 + 2c3, X6 = c0 + 2c5, X7 = c0 + 2c7.
// Its inverse is integral on 2E8:
//   c0 = P0, c2 = (P1-P0)/2, c4 = (P2-P0)/2, c6 = (P3-P0)/2, c3 = (P5-P0)/2,
//   c5 = (P6-P0)/2, c7 = (P7-P0)/2, c1 = (5P0 - P1 - P2 - P3 + P4 - P5 - P6 - P7)/4.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nq {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------------------
// Exact sign of a short sum of doubles (Shewchuk's grow-expansion with error-free
// TwoSum).  The expansion h is kept non-overlapping and increasing in magnitude, so the
// sign of the exact sum is the sign of its last non-zero component.  Round-to-nearest
// arithmetic without contraction is required (the library is built with
// -ffp-contract=off).
// ---------------------------------------------------------------------------------------
template <int N>
__device__ __forceinline__ int exact_sign_sum(const double (&t)[N]) {
  double h[N];
#pragma unroll
  for (int i = 0; i < N; ++i) {
    double Q = t[i];
#pragma unroll
    for (int j = 0; j < i; ++j) {
      const double s = Q + h[j];
      const double bv = s - Q;
      const double av = s - bv;
      const double err = (Q - av) + (h[j] - bv);
      Q = s;
      h[j] = err;
    }
    h[i] = Q;
  }
  int sgn = 0;
#pragma unroll
  for (int j = 0; j < N; ++j) sgn = (h[j] > 0.0) ? 1 : ((h[j] < 0.0) ? -1 : sgn);
  return sgn;
}

// ---------------------------------------------------------------------------------------
// Nearest point of E8 to an fp32 8-vector (App. C, Alg. 5, Conway-Sloane), in 2E8 units.
//
// Per coordinate: d = floor(y); g = [y > d + 1/2] (an exact half rounds down); the distance
// to the nearest integer e = |y - rint(y)| (exact for |y| < 2^23, also for tiny y).  The D8
// candidate is d + g with a parity fix at argmax e (lowest index) moving to the other
// neighbouring integer; the D8+1/2 candidate is d + 1/2 with a parity fix at argmin e
// (lowest index) moving towards y.  D8 wins iff the gap
//   sum e - 2 + odd1 (1 - 2 e_p) - odd2 2 e_r
// is negative; a zero gap returns D8+1/2.  The gap is evaluated in fp32 (about a dozen
// roundings, each below 2^-24 * 8, so the error is below 1e-5); when |gap| < 1e-5 its sign
// is recomputed exactly from the exact fp32 terms with exact_sign_sum.
//
// In 2E8 units every output is P_l = 2 d_l + delta_l with delta_l = 2 g_l (D8), 1 (D8+1/2);
// at the fixed coordinate delta = 2 - 2 g (D8) or 4 g - 1 (D8+1/2).
// ---------------------------------------------------------------------------------------
struct E8Cand {
  int d[8], g[8];
  float e[8];
  int odd1, odd2;
  float ep, er, gap;
};

__device__ __forceinline__ void e8_candidates(const float (&y)[8], E8Cand& k) {
#pragma unroll
  for (int l = 0; l < 8; ++l) {
    const float fl = floorf(y[l]);
    k.d[l] = (int)fl;
    k.g[l] = (y[l] > fl + 0.5f) ? 1 : 0;
    k.e[l] = fabsf(y[l] - rintf(y[l]));
  }
  const int sum_d = ((k.d[0] + k.d[1]) + (k.d[2] + k.d[3])) + ((k.d[4] + k.d[5]) + (k.d[6] + k.d[7]));
  const int sum_g = ((k.g[0] + k.g[1]) + (k.g[2] + k.g[3])) + ((k.g[4] + k.g[5]) + (k.g[6] + k.g[7]));
  // max e and min e (the coordinates that hold them are found in e8_point, for the one
  // candidate that is kept)
  k.ep = fmaxf(fmaxf(fmaxf(k.e[0], k.e[1]), fmaxf(k.e[2], k.e[3])),
               fmaxf(fmaxf(k.e[4], k.e[5]), fmaxf(k.e[6], k.e[7])));
  k.er = fminf(fminf(fminf(k.e[0], k.e[1]), fminf(k.e[2], k.e[3])),
               fminf(fminf(k.e[4], k.e[5]), fminf(k.e[6], k.e[7])));
  k.odd1 = (sum_d + sum_g) & 1;
  k.odd2 = sum_d & 1;
  float se = k.e[0];
#pragma unroll
  for (int l = 1; l < 8; ++l) se = se + k.e[l];
  float gap = se - 2.0f;
  if (k.odd1) gap = gap + (1.0f - 2.0f * k.ep);
  if (k.odd2) gap = gap - 2.0f * k.er;
  k.gap = gap;
}

// The exact sign of the gap from its exact fp32 terms (rare: |fp32 gap| < 1e-5).
__device__ __forceinline__ bool e8_gap_negative_exact(const E8Cand& k) {
  double t[12];
#pragma unroll
  for (int l = 0; l < 8; ++l) t[l] = (double)k.e[l];
  t[8] = -2.0;
  t[9] = k.odd1 ? 1.0 : 0.0;
  t[10] = k.odd1 ? -2.0 * (double)k.ep : 0.0;
  t[11] = k.odd2 ? -2.0 * (double)k.er : 0.0;
  return exact_sign_sum<12>(t) < 0;
}

__device__ __forceinline__ void e8_point(const E8Cand& k, bool d8, int (&P)[8]) {
  // delta for g = 0 / g = 1, off and on the fixed coordinate
  const int a_g0 = d8 ? 0 : 1, a_g1 = d8 ? 2 : 1;
  const int b_g0 = d8 ? 2 : -1, b_g1 = d8 ? 0 : 3;
  // the fixed coordinate: the lowest index holding max e (D8) or min e (D8+1/2), if that
  // candidate's parity needs a fix
  const float target = d8 ? k.ep : k.er;
  int idx = 7;
#pragma unroll
  for (int l = 6; l >= 0; --l) idx = (k.e[l] == target) ? l : idx;
  const int fix = (d8 ? k.odd1 : k.odd2) ? idx : 8;
#pragma unroll
  for (int l = 0; l < 8; ++l) {
    const int delta = (l == fix) ? (k.g[l] ? b_g1 : b_g0) : (k.g[l] ? a_g1 : a_g0);
    P[l] = 2 * k.d[l] + delta;
  }
}

__device__ __forceinline__ void nearest_e8(const float (&y)[8], int (&P)[8]) {
  E8Cand k;
  e8_candidates(y, k);
  bool d8 = k.gap < 0.0f;
  if (__builtin_expect(fabsf(k.gap) < 1.0e-5f, 0)) d8 = e8_gap_negative_exact(k);
  e8_point(k, d8, P);
}

// nearest_e8 without the exact fallback: false (P unset) when the fp32 gap cannot decide.
__device__ __forceinline__ bool nearest_e8_fast(const float (&y)[8], int (&P)[8]) {
  E8Cand k;
  e8_candidates(y, k);
  if (fabsf(k.gap) < 1.0e-5f) return false;
  e8_point(k, k.gap < 0.0f, P);
  return true;
}

// max over the 240 roots lambda of E8 of <P, lambda> for P in 2E8 units:
// max( |P|_(1) + |P|_(2),  (sum |P_i| - 2 [odd number of negative P_i] min |P_i|) / 2 ).
// P lies strictly inside the cell q V of q 2E8 iff the bound is < 2q, strictly outside iff
// it is > 2q; equality is the cell boundary.  amax = |P|_(1) comes with it.
__device__ __forceinline__ int e8_root_bound(const int (&P)[8], int& amax) {
  int a[8];
#pragma unroll
  for (int l = 0; l < 8; ++l) a[l] = abs(P[l]);
  int m1 = max(a[0], a[1]), m2 = min(a[0], a[1]);
#pragma unroll
  for (int l = 2; l < 8; ++l) {
    m2 = max(m2, min(m1, a[l]));  // the median of (m1, m2, a) since m2 <= m1
    m1 = max(m1, a[l]);
  }
  const int sa = ((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7]));
  const int mn = min(min(min(a[0], a[1]), min(a[2], a[3])), min(min(a[4], a[5]), min(a[6], a[7])));
  const int neg = (int)(((uint32_t)(P[0] ^ P[1] ^ P[2] ^ P[3] ^ P[4] ^ P[5] ^ P[6] ^ P[7])) >> 31);
  amax = m1;
  return max(m1 + m2, (sa - ((0 - neg) & (mn << 1))) >> 1);   // a select, not a multiply
}

__device__ __forceinline__ int e8_root_bound(const int (&P)[8]) {
  int amax;
  return e8_root_bound(P, amax);
}

// Root bound of a real 8-vector: max over the 240 roots lambda of <x, lambda>.  For the
// nearest point p of E8 to x, |max<2p, lambda> - 2 max<x, lambda>| <= 2 |p - x| |lambda|
// <= 2 sqrt(2), since the covering radius of E8 is 1 and roots have norm sqrt(2).
__device__ __forceinline__ float root_bound_f(const float (&x)[8]) {
  float a[8];
#pragma unroll
  for (int l = 0; l < 8; ++l) a[l] = fabsf(x[l]);
  float m1 = fmaxf(a[0], a[1]), m2 = fminf(a[0], a[1]);
#pragma unroll
  for (int l = 2; l < 8; ++l) {
    m2 = fmaxf(m2, fminf(m1, a[l]));
    m1 = fmaxf(m1, a[l]);
  }
  const float sa = ((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7]));
  const float mn = fminf(fminf(fminf(a[0], a[1]), fminf(a[2], a[3])),
                         fminf(fminf(a[4], a[5]), fminf(a[6], a[7])));
  int neg = 0;
#pragma unroll
  for (int l = 0; l < 8; ++l) neg ^= (x[l] < 0.0f) ? 1 : 0;
  return fmaxf(m1 + m2, 0.5f * (sa - (neg ? 2.0f * mn : 0.0f)));
}

// v mod q in [0, q): exact for |v| < 2^24 (fp32 reciprocal estimate and one correction).
__device__ __forceinline__ int mod_q_general(int v, int q, float rq) {
  const int n = (int)floorf((float)v * rq);
  int r = v - __mul24(n, q);
  r += (r < 0) ? q : 0;
  r -= (r >= q) ? q : 0;
  return r;
}

// Alg. 1 after the nearest-point step: the codes G^-1 P mod q, packed as nibbles.
// Fast path (|P_i| < 512, always true for points that do not overload, |P_i| <= 2q): add a
// bias of 1024 q to make v non-negative and divide with a 24-bit multiply,
// floor(u / q) = (u * mq) >> 20 with mq = ceil(2^20 / q), exact for u < 2^20 / q.
// encode_codes_amax takes max |P_i| when the caller already has it.
//
// umul24_v is the full-rate 24-bit multiply (low 32 bits of the product of the operands'
// low 24 bits), the same as __umul24; written out because the compiler turns some
// __umul24 of values it has range facts about into a quarter-rate 32-bit multiply.
__device__ __forceinline__ uint32_t umul24_v(uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_mul_u32_u24 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// fp16(fp32 fma(a0, b, c)) in the low and fp16(fp32 fma(a1, b, c)) in the high half: the
// mixed-precision fma with fp32 sources rounds its fp32 result to fp16 (the compiler selects
// the low-half form for fp16(a * b) itself; the high-half form saves the shift and OR).
__device__ __forceinline__ uint32_t fma_mix_pk_f16(float a0, float a1, float b, float c) {
  uint32_t d;
  asm("v_fma_mixlo_f16 %0, %1, %2, %3 op_sel_hi:[0,0,0]" : "=v"(d) : "v"(a0), "v"(b), "v"(c));
  asm("v_fma_mixhi_f16 %0, %1, %2, %3 op_sel_hi:[0,0,0]" : "+v"(d) : "v"(a1), "v"(b), "v"(c));
  return d;
}

// Low 16 bits of the products of the two 16-bit halves (full rate); a multiply of 16-bit
// vectors in C is split by the compiler into quarter-rate 32-bit multiplies.
__device__ __forceinline__ uint32_t pk_mul_lo_u16(uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_pk_mul_lo_u16 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// popcount(x) + acc in one instruction (the compiler adds a separate popcount to acc).
__device__ __forceinline__ uint32_t bcnt_add(uint32_t x, uint32_t acc) {
  uint32_t r;
  asm("v_bcnt_u32_b32 %0, %1, %2" : "=v"(r) : "v"(x), "v"(acc));
  return r;
}

__device__ __forceinline__ uint32_t encode_codes_amax(const int (&P)[8], int q, float rq,
                                                      uint32_t mq, int amax) {
  int v[8];
  v[0] = P[0];
  v[2] = (P[1] - P[0]) >> 1;
  v[4] = (P[2] - P[0]) >> 1;
  v[6] = (P[3] - P[0]) >> 1;
  v[3] = (P[5] - P[0]) >> 1;
  v[5] = (P[6] - P[0]) >> 1;
  v[7] = (P[7] - P[0]) >> 1;
  const int rest = -P[1] - P[2] - P[3] + P[4] - P[5] - P[6] - P[7];
  uint32_t w = 0;
  if (amax < 512) {
    // |v| <= 3 * 511 < 1024 q, so u = v + 1024 q lies in [0, 2048 q) and 2048 q < 2^20 / q.
    // Every product is a full-rate 24-bit multiply (u < 2^15, mq < 2^20, |P_0| < 512).
    v[1] = (__mul24(P[0], 5) + rest) >> 2;
    const uint32_t qq = (uint32_t)q, mm = mq;
    const int bias = q << 10;
#pragma unroll
    for (int l = 0; l < 8; ++l) {
      const uint32_t u = (uint32_t)(v[l] + bias);
      const uint32_t n = umul24_v(u, mm) >> 20;
      w |= (u - umul24_v(n, qq)) << (4 * l);
    }
  } else {
    v[1] = (5 * P[0] + rest) >> 2;
#pragma unroll
    for (int l = 0; l < 8; ++l) w |= (uint32_t)mod_q_general(v[l], q, rq) << (4 * l);
  }
  return w;
}

__device__ __forceinline__ uint32_t encode_codes(const int (&P)[8], int q, float rq, uint32_t mq) {
  int big = 0;
#pragma unroll
  for (int l = 0; l < 8; ++l) big |= abs(P[l]);
  return encode_codes_amax(P, q, rq, mq, big);
}

// ---------------------------------------------------------------------------------------
// Alg. 2 on one code word, four coordinates per 32-bit register (byte SIMD, nq_b8.hpp):
// X = G c, then X - q * 2 Q(X / 2q) in exact integers (all distances times 2q), Q = Alg. 5
// with the tie rules of nearest_e8, or (M) the NestQuantM oracle of App. D, whose parity
// fixes are at the first coordinate (no argmin / argmax).  m2q = ceil(2^16 / (2q)) gives
// floor(X / 2q) = (X * m2q) >> 16 exactly for 0 <= X < 2^11.
//
// Shifting X by 2q * v with v in D8 leaves the decode unchanged (Alg. 5 commutes with D8
// shifts), so only f = X mod 2q per coordinate and the parity pi of sum floor(X / 2q)
// matter.  With h = f - q: the D8+1/2 residual is h, the D8 residual is f - 2q [h > 0], the
// distance to the nearest integer (times 2q) is q - |h|, so argmax / argmin of it are
// argmin / argmax |h| (lowest index), and the gap of Alg. 5 times 2q is
//   4q - sum |h| + odd1 * 2 min|h| - pi * (2q - 2 max|h|),   odd1 = (pi + #[h > 0]) mod 2.
// ---------------------------------------------------------------------------------------
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

#include "nq_b8.hpp"

// ---------------------------------------------------------------------------------------
// NestQuantM decode at q = 16 with four coordinates per register (byte SIMD).  With 2q = 32
// every X = G c fits a byte (X4 <= 15 + 2 * 120 = 255, the others <= 45), floor(X / 32) and
// X mod 32 are a shift and a mask per byte, sum |X mod 32 - 16| is one v_sad_u8 per four
// coordinates, and without argmin / argmax only coordinate 0 is ever flipped.  Same
// arithmetic and tie rules as decode_word_b8<true> at q = 16.
//
// Outputs: x0 = X2_0 (the flipped coordinate, |x0| <= 32) and, in xa (coordinates 0-3) and
// xb (4-7), every coordinate before the flip as the unsigned byte X2_l + 32 (|X2_l| <= 16
// there): the D8 residual f - 32 g is f | (g << 5) as a 6-bit two's-complement field, the
// D8+1/2 residual f - 16 is f ^ 0x30 ^ ((f & 0x10) << 1), and flipping bit 5 of such a field
// adds 32.  Only OR / XOR / shifts, no carries between bytes.
// ---------------------------------------------------------------------------------------
__device__ __forceinline__ void decode_word_m16(uint32_t w, uint32_t& xa, uint32_t& xb, int& x0) {
  const uint32_t E = w & 0x0F0F0F0Fu;           // bytes c0 c2 c4 c6
  const uint32_t O = (w >> 4) & 0x0F0F0F0Fu;    // bytes c1 c3 c5 c7
  const uint32_t c0 = E & 0xFFu;
  const uint32_t sum_c = __builtin_amdgcn_sad_u8(E, 0u, __builtin_amdgcn_sad_u8(O, 0u, 0u));
  // (X0..X3) = c0 + 2 (0, c2, c4, c6); (X4..X7) = c0 + 2 (c1 + sum c - c0, c3, c5, c7)
  const uint32_t c0x4 = __builtin_amdgcn_perm(0u, c0, 0x00000000u);   // c0 in every byte
  const uint32_t Xa = c0x4 + ((E & 0xFFFFFF00u) << 1);
  const uint32_t Xb = c0x4 + (((O & 0xFFFFFF00u) | ((O & 0xFFu) + sum_c - c0)) << 1);
  const uint32_t Fa = Xa & 0x1F1F1F1Fu, Fb = Xb & 0x1F1F1F1Fu;              // X mod 32
  const uint32_t Da = (Xa >> 5) & 0x07070707u, Db = (Xb >> 5) & 0x07070707u;  // floor(X / 32)
  // g = [f > 16] (an exact half rounds down): bit 5 of f + 15
  const uint32_t Ga = ((Fa + 0x0F0F0F0Fu) >> 5) & 0x01010101u;
  const uint32_t Gb = ((Fb + 0x0F0F0F0Fu) >> 5) & 0x01010101u;
  const uint32_t sum_h = __builtin_amdgcn_sad_u8(Fa, 0x10101010u,
                                                 __builtin_amdgcn_sad_u8(Fb, 0x10101010u, 0u));
  const uint32_t pi = __builtin_amdgcn_sad_u8(Da, 0u, __builtin_amdgcn_sad_u8(Db, 0u, 0u)) & 1u;
  const uint32_t odd1 = (pi + __builtin_popcount(Ga | (Gb << 1))) & 1u;
  const int f0 = (int)(Fa & 0xFFu);
  const int h0 = abs(f0 - 16);
  // Alg. 5's gap times 2q with both fixes at coordinate 0: 4q - sum|h| + odd1 2|h0| - pi (2q - 2|h0|)
  const int gap = 64 - (int)sum_h + (odd1 ? 2 * h0 : 0) - (pi ? 32 - 2 * h0 : 0);
  const bool d8 = gap < 0;
  const uint32_t m = 0u - (uint32_t)d8;                       // all ones for D8
  const uint32_t ra = Fa ^ 0x30303030u ^ ((Fa & 0x10101010u) << 1);
  const uint32_t rb = Fb ^ 0x30303030u ^ ((Fb & 0x10101010u) << 1);
  xa = (ra ^ (((Fa | (Ga << 5)) ^ ra) & m)) ^ 0x20202020u;
  xb = (rb ^ (((Fb | (Gb << 5)) ^ rb) & m)) ^ 0x20202020u;
  // coordinate 0 moves by +32 s (D8) or -32 s (D8+1/2), s = 2 g0 - 1
  const bool g0 = (Ga & 1u) != 0;
  const int r0 = d8 ? (g0 ? f0 - 32 : f0) : f0 - 16;
  const bool fix = d8 ? (odd1 != 0) : (pi != 0);
  x0 = r0 + (fix ? ((g0 == d8) ? 32 : -32) : 0);
}

// One thread per block of a rows x nb grid of blocks, 256 threads per workgroup: rows
// shorter than 256 blocks are packed (a power-of-two group of lanes per row), longer rows
// are cut into 256-block segments.  lg = log2 of the group size (for nb <= 256) or -1.
// The workgroup's first row rb is uniform; the thread's row is rb + lr and its block j, so
// per-thread offsets inside the workgroup's rows fit 32 bits.
struct GridPos {
  int64_t rb;
  int lr, j;
};
__device__ __forceinline__ GridPos grid_block(int nb, int lg) {
  GridPos g;
  if (lg >= 0) {
    g.rb = (int64_t)blockIdx.x * (256 >> lg);
    g.lr = (int)(threadIdx.x >> lg);
    g.j = (int)(threadIdx.x & ((1u << lg) - 1u));
  } else {
    const uint32_t segs = ((uint32_t)nb + 255u) / 256u;
    const uint32_t row = blockIdx.x / segs;
    g.rb = row;
    g.lr = 0;
    g.j = (int)(blockIdx.x - row * segs) * 256 + (int)threadIdx.x;
  }
  return g;
}

// The multiple m of base for beta index idx (0..3): byte idx of the operand's table.
__device__ __forceinline__ int beta_mult(uint32_t mtab, uint32_t idx) {
  return (int)((mtab >> (8u * idx)) & 0xFFu);
}

// Two integer-valued floats as a 16-bit pair (lo in the low half): bf16 keeps the upper
// halves of the fp32 values, fp16 converts (toward zero; exact for the integers here).
template <bool F16>
__device__ __forceinline__ uint32_t pack16(float lo, float hi) {
  if constexpr (F16) {
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(lo, hi));
  } else {
    return __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), 0x07060302u);
  }
}

// m * X2 of one block as eight bf16 or fp16 values, coordinates 2i and 2i+1 in word i.
// |X2| <= 2q <= 32, so the values are exact integers in bf16 while |m X2| <= 256 (m <= 4
// for every q, the uniform beta grid) and in fp16 while |m X2| <= 2048 (m <= 64).  DV 0 and 1
// decode with decode_word_b8 (bytes biased by 128: value = m byte - 128 m, one exact fma);
// DV 2 (NestQuantM at q = 16) with decode_word_m16.
template <int DV = 0, bool F16 = false>
__device__ __forceinline__ u32x4 decode_tile_16(uint32_t w, int m, int q, uint32_t m2q) {
  if constexpr (DV == 2) {
    uint32_t xa, xb;
    int x0;
    decode_word_m16(w, xa, xb, x0);
    // bytes hold X2 + 32: m X2 = b m - 32 m is one fma (both terms exact, the result an
    // integer of at most 11 bits)
    const float fm = (float)m, off = -32.0f * fm;
    auto val = [&](uint32_t x, int b) {
      return __builtin_fmaf((float)((x >> (8 * b)) & 0xFFu), fm, off);
    };
    return u32x4{pack16<F16>((float)(x0 * m), val(xa, 1)), pack16<F16>(val(xa, 2), val(xa, 3)),
                 pack16<F16>(val(xb, 0), val(xb, 1)), pack16<F16>(val(xb, 2), val(xb, 3))};
  }
  uint32_t xa, xb;
  decode_word_b8<DV == 1>(w, q, m2q, xa, xb);
  const float fm = (float)m, off = -128.0f * fm;
  auto val = [&](uint32_t x, int b) {
    return __builtin_fmaf((float)((x >> (8 * b)) & 0xFFu), fm, off);   // m (byte - 128), exact
  };
  return u32x4{pack16<F16>(val(xa, 0), val(xa, 1)), pack16<F16>(val(xa, 2), val(xa, 3)),
               pack16<F16>(val(xb, 0), val(xb, 1)), pack16<F16>(val(xb, 2), val(xb, 3))};
}

// m * X2 of one block as eight int8 (exact when 2 q m <= 127: |X2| <= 2q), the
// coordinates in byte order.  The signed bytes X2 are multiplied in 16-bit lanes (even and
// odd bytes apart); each product keeps its low byte, the two's-complement int8 of a value
// in [-127, 127].
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
template <int DV = 0>
__device__ __forceinline__ u32x2 decode_tile_i8(uint32_t w, int m, int q, uint32_t m2q) {
  uint32_t xa, xb;
  decode_word_b8<DV != 0>(w, q, m2q, xa, xb);
  const uint32_t mm = (uint32_t)m | ((uint32_t)m << 16);   // m in both halves
  auto mul8 = [&](uint32_t x) {
    const uint32_t s = x ^ 0x80808080u;                  // X2 as signed bytes
    const uint32_t lo = pk_mul_lo_u16(s & 0x00FF00FFu, mm);
    const uint32_t hi = pk_mul_lo_u16((s >> 8) & 0x00FF00FFu, mm);
    return (lo & 0x00FF00FFu) | ((hi & 0x00FF00FFu) << 8);
  };
  return u32x2{mul8(xa), mul8(xb)};
}

// X2 of one block as eight int8 (|X2| <= 2q <= 32), the coordinates in byte order, with no
// multiple applied: the byte decoder's X2 + 128 with bit 7 of each byte flipped.  DV 0 is
// the full decoder, DV 1 NestQuantM (at q = 16 too: decode_word_m16's X2 + 32 would take
// three instructions a word to int8 instead of one).
template <int DV = 0>
__device__ __forceinline__ u32x2 decode_x2_i8(uint32_t w, int q, uint32_t m2q) {
  static_assert(DV == 0 || DV == 1, "the byte decoder's variants");
  uint32_t xa, xb;
  decode_word_b8<DV == 1>(w, q, m2q, xa, xb);
  return u32x2{xa ^ 0x80808080u, xb ^ 0x80808080u};
}

// The decoder's residual X - q * 2 Q(X / 2q) for integer X >= 0 (< 2^11), Q = Alg. 5 or
// (M) the NestQuantM oracle: the scalar form of decode_word_b8 without the generator step.
// Rounding half down, round(X / 2q) = floor((X + q - 1) / 2q).
template <bool M = false>
__device__ __forceinline__ void residual_from_X(const int (&X)[8], int q, uint32_t m2q,
                                                int (&X2)[8]) {
  const int den = 2 * q;
  const uint32_t half_off = (uint32_t)(q - 1) * m2q;
  int d[8], g[8], f[8], E[8];
#pragma unroll
  for (int l = 0; l < 8; ++l) {
    d[l] = (int)(__umul24((uint32_t)X[l], m2q) >> 16);
    const int x1 = (int)((__umul24((uint32_t)X[l], m2q) + half_off) >> 16);
    g[l] = x1 - d[l];
    f[l] = X[l] - __mul24(den, d[l]);
    E[l] = min(f[l], den - f[l]);
  }
  const int sum_d = ((d[0] + d[1]) + (d[2] + d[3])) + ((d[4] + d[5]) + (d[6] + d[7]));
  const int sum_g = ((g[0] + g[1]) + (g[2] + g[3])) + ((g[4] + g[5]) + (g[6] + g[7]));
  const int sE = ((E[0] + E[1]) + (E[2] + E[3])) + ((E[4] + E[5]) + (E[6] + E[7]));
  int p = 0, r = 0, Ep = E[0], Er = E[0];
  if constexpr (!M) {
    int kmax = (E[0] << 3) | 7, kmin = E[0] << 3;
#pragma unroll
    for (int l = 1; l < 8; ++l) {
      kmax = max(kmax, (E[l] << 3) | (7 - l));
      kmin = min(kmin, (E[l] << 3) | l);
    }
    p = 7 - (kmax & 7);
    Ep = kmax >> 3;
    r = kmin & 7;
    Er = kmin >> 3;
  }
  const int odd1 = (sum_d + sum_g) & 1, odd2 = sum_d & 1;
  const int gap = sE - 2 * den + (odd1 ? den - 2 * Ep : 0) - (odd2 ? 2 * Er : 0);
  const bool d8 = gap < 0;
  const int fix = d8 ? (odd1 ? p : 8) : (odd2 ? r : 8);
#pragma unroll
  for (int l = 0; l < 8; ++l) {
    const int v = d8 ? (g[l] ? f[l] - den : f[l]) : f[l] - q;
    const bool up = (g[l] != 0) == d8;
    X2[l] = (l == fix) ? (up ? v + den : v - den) : v;
  }
}

// First-beta overload test of one candidate point (Sec. 4.1): overloaded iff
// decode(encode(P)) != P.  The root bound settles every point off the cell boundary.  On the
// boundary (M(P) = 2q, where Alg. 5's tie rules decide) the literal test is evaluated
// without building the code word (boundary_overloaded; also the NestQuantM test): the
// decoder sees X = G (G^-1 P mod q) = P + 2q v with v in E8, and the residual of Alg. 2 is
// unchanged by D8 shifts of X / 2q (for both oracles), so it equals the residual of P
// (v in D8) or of P + q (1,...,1) (v in D8 + 1/2).  v lies in D8 + 1/2 exactly when
// floor(P_0 / q) is odd (column 0 of G is the only odd column).  An offset of 4q
// (= 2q * (2,...,2), in D8) keeps X non-negative for P_0 >= -2q.
template <bool M = false>
__device__ __forceinline__ bool boundary_overloaded(const int (&P)[8], int q, uint32_t mq,
                                                    uint32_t m2q) {
  const uint32_t u0 = (uint32_t)(P[0] + 4 * q);               // P_0 >= -2q on the boundary
  const int odd = (int)((__umul24(u0, mq) >> 20) & 1u);       // parity of floor(P_0 / q)
  const int off = 4 * q + (odd ? q : 0);
  int X[8], X2[8];
#pragma unroll
  for (int l = 0; l < 8; ++l) X[l] = P[l] + off;
  residual_from_X<M>(X, q, m2q, X2);
  bool diff = false;
#pragma unroll
  for (int l = 0; l < 8; ++l) diff |= (X2[l] != P[l]);
  return diff;
}

__device__ __forceinline__ bool overloaded(const int (&P)[8], int q, float rq, uint32_t mq,
                                           uint32_t m2q) {
  const int M = e8_root_bound(P);
  if (M != 2 * q) return M > 2 * q;
  return boundary_overloaded(P, q, mq, m2q);
}

// The same test for the NestQuantM decoder (App. D).  Every point that decoder returns lies
// in the box |P_0| <= 2q, |P_i| <= q (i > 0); outside it P surely overloads, and inside it
// (where P_0 >= -2q, as boundary_overloaded needs) the literal test decides.
__device__ __forceinline__ bool in_m_box(const int (&P)[8], int q) {
  int m = 0;
#pragma unroll
  for (int l = 1; l < 8; ++l) m = max(m, abs(P[l]));
  return m <= q && abs(P[0]) <= 2 * q;
}

__device__ __forceinline__ bool overloaded_m(const int (&P)[8], int q, uint32_t mq,
                                             uint32_t m2q) {
  if (!in_m_box(P, q)) return true;
  return boundary_overloaded<true>(P, q, mq, m2q);
}

}  // namespace nq
