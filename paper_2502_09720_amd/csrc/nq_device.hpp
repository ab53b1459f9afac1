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
__device__ __forceinline__ void nearest_e8(const float (&y)[8], int (&P)[8]) {
  float e[8];
  int d[8], g[8];
#pragma unroll
  for (int l = 0; l < 8; ++l) {
    const float fl = floorf(y[l]);
    d[l] = (int)fl;
    g[l] = (y[l] > fl + 0.5f) ? 1 : 0;
    e[l] = fabsf(y[l] - rintf(y[l]));
  }
  const int sum_d = ((d[0] + d[1]) + (d[2] + d[3])) + ((d[4] + d[5]) + (d[6] + d[7]));
  const int sum_g = ((g[0] + g[1]) + (g[2] + g[3])) + ((g[4] + g[5]) + (g[6] + g[7]));
  int p = 0, r = 0;
  float ep = e[0], er = e[0];
#pragma unroll
  for (int l = 1; l < 8; ++l) {
    const bool up = e[l] > ep;    // strict: the lowest index wins ties
    const bool dn = e[l] < er;
    p = up ? l : p;
    ep = up ? e[l] : ep;
    r = dn ? l : r;
    er = dn ? e[l] : er;
  }
  const int odd1 = (sum_d + sum_g) & 1;
  const int odd2 = sum_d & 1;
  float se = e[0];
#pragma unroll
  for (int l = 1; l < 8; ++l) se = se + e[l];
  float gap = se - 2.0f;
  if (odd1) gap = gap + (1.0f - 2.0f * ep);
  if (odd2) gap = gap - 2.0f * er;
  bool d8;
  if (fabsf(gap) >= 1.0e-5f) {
    d8 = gap < 0.0f;
  } else {
    double t[12];
#pragma unroll
    for (int l = 0; l < 8; ++l) t[l] = (double)e[l];
    t[8] = -2.0;
    t[9] = odd1 ? 1.0 : 0.0;
    t[10] = odd1 ? -2.0 * (double)ep : 0.0;
    t[11] = odd2 ? -2.0 * (double)er : 0.0;
    d8 = exact_sign_sum<12>(t) < 0;
  }
  // delta for g = 0 / g = 1, off and on the fixed coordinate
  const int a_g0 = d8 ? 0 : 1, a_g1 = d8 ? 2 : 1;
  const int b_g0 = d8 ? 2 : -1, b_g1 = d8 ? 0 : 3;
  const int fix = d8 ? (odd1 ? p : 8) : (odd2 ? r : 8);
#pragma unroll
  for (int l = 0; l < 8; ++l) {
    const int delta = (l == fix) ? (g[l] ? b_g1 : b_g0) : (g[l] ? a_g1 : a_g0);
    P[l] = 2 * d[l] + delta;
  }
}

// max over the 240 roots lambda of E8 of <P, lambda> for P in 2E8 units:
// max( |P|_(1) + |P|_(2),  (sum |P_i| - 2 [odd number of negative P_i] min |P_i|) / 2 ).
// P lies strictly inside the cell q V of q 2E8 iff the bound is < 2q, strictly outside iff
// it is > 2q; equality is the cell boundary.
__device__ __forceinline__ int e8_root_bound(const int (&P)[8]) {
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
  return max(m1 + m2, (sa - 2 * neg * mn) >> 1);
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
__device__ __forceinline__ uint32_t encode_codes(const int (&P)[8], int q, float rq, uint32_t mq) {
  int v[8];
  v[0] = P[0];
  v[2] = (P[1] - P[0]) >> 1;
  v[4] = (P[2] - P[0]) >> 1;
  v[6] = (P[3] - P[0]) >> 1;
  v[3] = (P[5] - P[0]) >> 1;
  v[5] = (P[6] - P[0]) >> 1;
  v[7] = (P[7] - P[0]) >> 1;
  v[1] = (5 * P[0] - P[1] - P[2] - P[3] + P[4] - P[5] - P[6] - P[7]) >> 2;
  int big = 0;
#pragma unroll
  for (int l = 0; l < 8; ++l) big |= abs(P[l]);
  uint32_t w = 0;
  if (big < 512) {
    // |v| <= 3 * 511 < 1024 q, so u = v + 1024 q lies in [0, 2048 q) and 2048 q < 2^20 / q
    const int bias = q << 10;
#pragma unroll
    for (int l = 0; l < 8; ++l) {
      const uint32_t u = (uint32_t)(v[l] + bias);
      const uint32_t n = __umul24(u, mq) >> 20;
      w |= (u - __umul24(n, (uint32_t)q)) << (4 * l);
    }
  } else {
#pragma unroll
    for (int l = 0; l < 8; ++l) w |= (uint32_t)mod_q_general(v[l], q, rq) << (4 * l);
  }
  return w;
}

// Alg. 2 on one packed code word: X = G c, then X - q * 2 Q_E8(X / 2q) with Alg. 5 in
// exact integers (all distances multiplied by 2q; same tie rules as nearest_e8).
// m2q = ceil(2^16 / (2q)) gives floor(X / 2q) = (X * m2q) >> 16 exactly for 0 <= X < 2^11,
// and X <= 15 + 60 + 180 = 255 here.  Rounding half down, round(X / 2q) = floor((X + q - 1)
// / 2q).  Outputs X2_l = X_l - 2q x1_l (D8) or X_l - q (2 d_l + 1) (D8+1/2); with f = X - 2q d
// these are f - 2q g and f - q.
__device__ __forceinline__ void decode_word(uint32_t w, int q, uint32_t m2q, int (&X2)[8]) {
  int c[8];
#pragma unroll
  for (int l = 0; l < 8; ++l) c[l] = (int)((w >> (4 * l)) & 15u);
  int X[8];
  X[0] = c[0];
  X[1] = c[0] + 2 * c[2];
  X[2] = c[0] + 2 * c[4];
  X[3] = c[0] + 2 * c[6];
  X[4] = c[0] + 4 * c[1] + 2 * ((c[2] + c[3]) + (c[4] + c[5]) + (c[6] + c[7]));
  X[5] = c[0] + 2 * c[3];
  X[6] = c[0] + 2 * c[5];
  X[7] = c[0] + 2 * c[7];
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
  // argmax E / argmin E with the lowest index on ties, through keys E*8 + index
  int kmax = (E[0] << 3) | 7, kmin = E[0] << 3;
#pragma unroll
  for (int l = 1; l < 8; ++l) {
    kmax = max(kmax, (E[l] << 3) | (7 - l));
    kmin = min(kmin, (E[l] << 3) | l);
  }
  const int p = 7 - (kmax & 7), Ep = kmax >> 3;
  const int r = kmin & 7, Er = kmin >> 3;
  const int odd1 = (sum_d + sum_g) & 1, odd2 = sum_d & 1;
  const int gap = sE - 2 * den + (odd1 ? den - 2 * Ep : 0) - (odd2 ? 2 * Er : 0);
  const bool d8 = gap < 0;
  // X2 = f - 2q g (D8) or f - q (D8+1/2); the fixed coordinate moves by +-2q:
  // D8: to f - 2q g + 2q (2 g - 1);  D8+1/2: to f - q - 2q (2 g - 1)
  const int fix = d8 ? (odd1 ? p : 8) : (odd2 ? r : 8);
#pragma unroll
  for (int l = 0; l < 8; ++l) {
    const int v = d8 ? (g[l] ? f[l] - den : f[l]) : f[l] - q;
    const bool up = (g[l] != 0) == d8;     // D8 moves by +2q s, D8+1/2 by -2q s, s = 2g - 1
    X2[l] = (l == fix) ? (up ? v + den : v - den) : v;
  }
}

// First-beta overload test of one candidate point (Sec. 4.1): overloaded iff
// decode(encode(P)) != P.  The root bound settles every point off the cell boundary; on
// the boundary the literal decode decides (Alg. 5's tie rules make it tie-dependent).
__device__ __forceinline__ bool overloaded(const int (&P)[8], int q, float rq, uint32_t mq,
                                           uint32_t m2q) {
  const int M = e8_root_bound(P);
  if (M != 2 * q) return M > 2 * q;
  int X2[8];
  decode_word(encode_codes(P, q, rq, mq), q, m2q, X2);
  bool diff = false;
#pragma unroll
  for (int l = 0; l < 8; ++l) diff |= (X2[l] != P[l]);
  return diff;
}

}  // namespace nq
