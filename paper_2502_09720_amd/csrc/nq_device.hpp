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
// Per coordinate: d = floor(y), f = y - d (exact for |y| < 2^23), e = distance to the
// nearest integer = min(f, 1 - f) (exact), g = [f > 1/2] (an exact half rounds down).
// The D8 candidate is d + g with a parity fix at argmax e (lowest index); the D8+1/2
// candidate is d + 1/2 with a parity fix at argmin e (lowest index) moving towards y.
// D8 wins iff the gap  sum e - 2 + odd1 (1 - 2 e_p) - odd2 2 e_r  is negative; a zero gap
// returns D8+1/2.  The gap is evaluated in fp32 (about a dozen roundings, each below
// 2^-24 * 8, so the error is below 1e-5); when |gap| < 1e-5 its sign is recomputed exactly
// from the exact fp32 terms with exact_sign_sum.
// ---------------------------------------------------------------------------------------
__device__ __forceinline__ void nearest_e8(const float (&y)[8], int (&P)[8]) {
  float e[8];
  int d[8];
  int g[8];
  int sum_x1 = 0, sum_d = 0;
#pragma unroll
  for (int l = 0; l < 8; ++l) {
    const float fl = floorf(y[l]);
    const float f = y[l] - fl;
    g[l] = f > 0.5f ? 1 : 0;
    e[l] = g[l] ? (1.0f - f) : f;
    d[l] = (int)fl;
    sum_d += d[l];
    sum_x1 += d[l] + g[l];
  }
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
  const int odd1 = sum_x1 & 1;
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
#pragma unroll
  for (int l = 0; l < 8; ++l) {
    const int s = 2 * g[l] - 1;
    const int a = 2 * (d[l] + g[l]) - ((odd1 && l == p) ? 2 * s : 0);
    const int b = 2 * d[l] + 1 + ((odd2 && l == r) ? 2 * s : 0);
    P[l] = d8 ? a : b;
  }
}

// max over the 240 roots lambda of E8 of <P, lambda> for P in 2E8 units:
// max( |P|_(1) + |P|_(2),  (sum |P_i| - 2 [odd number of negative P_i] min |P_i|) / 2 ).
// P lies strictly inside the cell q V of q 2E8 iff the bound is < 2q, strictly outside iff
// it is > 2q; equality is the cell boundary.
__device__ __forceinline__ int e8_root_bound(const int (&P)[8]) {
  int m1 = 0, m2 = 0, sa = 0, mn = 0x7fffffff, neg = 0;
#pragma unroll
  for (int l = 0; l < 8; ++l) {
    const int a = abs(P[l]);
    m2 = max(m2, min(m1, a));
    m1 = max(m1, a);
    sa += a;
    mn = min(mn, a);
    neg ^= (P[l] < 0) ? 1 : 0;
  }
  return max(m1 + m2, (sa - 2 * neg * mn) >> 1);
}

// v mod q in [0, q) for |v| < 2^24 using an fp32 reciprocal estimate and one correction.
__device__ __forceinline__ int mod_q(int v, int q, float rq) {
  const int n = (int)floorf((float)v * rq);
  int r = v - n * q;
  r += (r < 0) ? q : 0;
  r -= (r >= q) ? q : 0;
  return r;
}

// Alg. 1 after the nearest-point step: the codes G^-1 P mod q, packed as nibbles.
__device__ __forceinline__ uint32_t encode_codes(const int (&P)[8], int q, float rq) {
  int v[8];
  v[0] = P[0];
  v[2] = (P[1] - P[0]) >> 1;
  v[4] = (P[2] - P[0]) >> 1;
  v[6] = (P[3] - P[0]) >> 1;
  v[3] = (P[5] - P[0]) >> 1;
  v[5] = (P[6] - P[0]) >> 1;
  v[7] = (P[7] - P[0]) >> 1;
  v[1] = (5 * P[0] - P[1] - P[2] - P[3] + P[4] - P[5] - P[6] - P[7]) >> 2;
  uint32_t w = 0;
#pragma unroll
  for (int l = 0; l < 8; ++l) w |= (uint32_t)mod_q(v[l], q, rq) << (4 * l);
  return w;
}

// Alg. 2 on one packed code word: X = G c, then X - q * 2 Q_E8(X / 2q) with Alg. 5 in
// exact integers (all distances multiplied by 2q; same tie rules as nearest_e8).
// m2q = ceil(2^16 / (2q)) gives floor(X / 2q) = (X * m2q) >> 16 exactly for 0 <= X < 2^11.
__device__ __forceinline__ void decode_word(uint32_t w, int q, uint32_t m2q, int (&X2)[8]) {
  int c[8];
#pragma unroll
  for (int l = 0; l < 8; ++l) c[l] = (int)((w >> (4 * l)) & 15u);
  int X[8];
  X[0] = c[0];
  X[1] = c[0] + 2 * c[2];
  X[2] = c[0] + 2 * c[4];
  X[3] = c[0] + 2 * c[6];
  X[4] = c[0] + 4 * c[1] + 2 * (c[2] + c[3] + c[4] + c[5] + c[6] + c[7]);
  X[5] = c[0] + 2 * c[3];
  X[6] = c[0] + 2 * c[5];
  X[7] = c[0] + 2 * c[7];
  const int den = 2 * q;
  int d[8], g[8], E[8];
  int sx1 = 0, sd = 0, sE = 0;
#pragma unroll
  for (int l = 0; l < 8; ++l) {
    d[l] = (int)(((uint32_t)X[l] * m2q) >> 16);
    const int f = X[l] - den * d[l];
    g[l] = (2 * f > den) ? 1 : 0;
    E[l] = min(f, den - f);
    sx1 += d[l] + g[l];
    sd += d[l];
    sE += E[l];
  }
  int p = 0, r = 0;
  int Ep = E[0], Er = E[0];
#pragma unroll
  for (int l = 1; l < 8; ++l) {
    const bool up = E[l] > Ep;    // strict: the lowest index wins ties
    const bool dn = E[l] < Er;
    p = up ? l : p;
    Ep = up ? E[l] : Ep;
    r = dn ? l : r;
    Er = dn ? E[l] : Er;
  }
  const int odd1 = sx1 & 1, odd2 = sd & 1;
  const int gap = sE - 2 * den + (odd1 ? den - 2 * Ep : 0) - (odd2 ? 2 * Er : 0);
  const bool d8 = gap < 0;
#pragma unroll
  for (int l = 0; l < 8; ++l) {
    const int s = 2 * g[l] - 1;
    const int a = 2 * (d[l] + g[l]) - ((odd1 && l == p) ? 2 * s : 0);
    const int b = 2 * d[l] + 1 + ((odd2 && l == r) ? 2 * s : 0);
    X2[l] = X[l] - q * (d8 ? a : b);
  }
}

// First-beta overload test of one candidate point (Sec. 4.1): overloaded iff
// decode(encode(P)) != P.  The root bound settles every point off the cell boundary; on
// the boundary the literal decode decides (Alg. 5's tie rules make it tie-dependent).
__device__ __forceinline__ bool overloaded(const int (&P)[8], int q, float rq, uint32_t m2q) {
  const int M = e8_root_bound(P);
  if (M != 2 * q) return M > 2 * q;
  int X2[8];
  decode_word(encode_codes(P, q, rq), q, m2q, X2);
  bool diff = false;
#pragma unroll
  for (int l = 0; l < 8; ++l) diff |= (X2[l] != P[l]);
  return diff;
}

}  // namespace nq
