// NestQuant row encoder (Sec. 4.2, Alg. 3 with the First-beta or Opt-beta strategy of
// App. F).
//
// One lane per 8-entry block.  A row is handled by a group of LANES lanes (a power of two,
// 8 <= LANES <= 1024): several rows share a 256-thread workgroup when LANES <= 64, and a
// workgroup is exactly one row when LANES > 64.  Each lane keeps BPT blocks in registers, block
// j = lane + i * LANES, so the row is read from HBM exactly once and consecutive lanes read
// consecutive 8-entry blocks (16 B for bf16/fp16, 32 B for fp32).
//
// Row scale (Alg. 3, s / sqrt(n)): r is the fp32 number nearest to sqrt(sum x^2 / n).  The
// squares of fp32 values are exact in fp64; the fp64 sum is accepted when it cannot straddle
// an fp32 rounding boundary, otherwise the row is summed again as a double-double and the
// boundary comparison is made exactly.
#include "nq_device.hpp"
#include "nq_kernels.hpp"
#include "nq_rotate.hpp"
#include "nq_tiles.hpp"

namespace nq {

constexpr int a_max_k = 4;
constexpr float kRootMargin = 2.8284272f + 0.02f;  // 2 sqrt(2), rounded up, + slack

__device__ __forceinline__ float pick4(const float (&c)[4], int t) {
  return t == 0 ? c[0] : (t == 1 ? c[1] : (t == 2 ? c[2] : c[3]));
}

template <typename T>
__device__ __forceinline__ void load_block(const T* __restrict__ p, float (&v)[8]);

template <>
__device__ __forceinline__ void load_block<float>(const float* __restrict__ p, float (&v)[8]) {
  const f32x4 a = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
  const f32x4 b = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p) + 1);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

template <>
__device__ __forceinline__ void load_block<uint16_t>(const uint16_t* __restrict__ p,
                                                     float (&v)[8]) {
  // bf16: the value is the upper half of an fp32 word
  const u32x4 a = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(w[i] << 16);
    v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

template <>
__device__ __forceinline__ void load_block<_Float16>(const _Float16* __restrict__ p,
                                                     float (&v)[8]) {
  const u32x4 a = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint16_t lo = (uint16_t)(w[i] & 0xffffu), hi = (uint16_t)(w[i] >> 16);
    v[2 * i] = (float)__builtin_bit_cast(_Float16, lo);
    v[2 * i + 1] = (float)__builtin_bit_cast(_Float16, hi);
  }
}

// Sum over the LANES lanes of a row group.  LANES <= 64: within the wave by xor shuffles
// (every lane ends with the same, bit-identical sum).  LANES > 64: the workgroup is exactly
// one row (LANES threads); wave sums are combined through LDS in a fixed order.
template <int LANES>
__device__ __forceinline__ double group_sum(double v, double* red) {
#pragma unroll
  for (int m = 1; m < (LANES < 64 ? LANES : 64); m <<= 1) v += __shfl_xor(v, m, 64);
  if constexpr (LANES > 64) {
    const int wave = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[wave] = v;
    __syncthreads();
    v = red[0];
#pragma unroll
    for (int i = 1; i < LANES / 64; ++i) v += red[i];
  }
  return v;
}

// Double-double version of group_sum (error-free on the hi parts).
__device__ __forceinline__ void two_sum(double a, double b, double& s, double& e) {
  s = a + b;
  const double bv = s - a;
  const double av = s - bv;
  e = (a - av) + (b - bv);
}

template <int LANES>
__device__ __forceinline__ void group_sum_dd(double& hi, double& lo, double* red) {
#pragma unroll
  for (int m = 1; m < (LANES < 64 ? LANES : 64); m <<= 1) {
    const double oh = __shfl_xor(hi, m, 64), ol = __shfl_xor(lo, m, 64);
    double s, e;
    two_sum(hi, oh, s, e);
    hi = s;
    lo = lo + ol + e;
  }
  if constexpr (LANES > 64) {
    const int wave = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) {
      red[2 * wave] = hi;
      red[2 * wave + 1] = lo;
    }
    __syncthreads();
    hi = red[0];
    lo = red[1];
#pragma unroll
    for (int i = 1; i < LANES / 64; ++i) {
      double s, e;
      two_sum(hi, red[2 * i], s, e);
      hi = s;
      lo = lo + red[2 * i + 1] + e;
    }
  }
  double s, e;
  two_sum(hi, lo, s, e);
  hi = s;
  lo = e;
}

// sign of (hi + lo) - n * m^2, exactly (m has at most 25 significant bits, so m^2 is exact
// in fp64 and n * m^2 is exact as the pair (prod, err) of a fused multiply).
__device__ __forceinline__ int cmp_sum_square(double hi, double lo, double n, double m) {
  const double m2 = m * m;
  const double prod = n * m2;
  const double err = __builtin_fma(n, m2, -prod);
  const double t[4] = {hi, lo, -prod, -err};
  return exact_sign_sum<4>(t);
}

__device__ __forceinline__ float next_up(float v) { return __uint_as_float(__float_as_uint(v) + 1u); }
__device__ __forceinline__ float next_down(float v) { return __uint_as_float(__float_as_uint(v) - 1u); }

// NestQuantM (App. D): every point its decoder reproduces lies in |P_0| <= 2q, |P_i| <= q.
// The nearest point P of y has |P_i - 2 y_i| <= 2 (covering radius 1), so a block whose
// statistic s = max(2 max_{i>0} |x_i|, |x_0|) has s c > (q + 2)(1 + 2^-12) surely overloads
// at the multiplier c (the slack covers the rounding of y = fl32(x c)).
__device__ __forceinline__ float m_stat(const float (&x)[8]) {
  float m = fabsf(x[1]);
#pragma unroll
  for (int l = 2; l < 8; ++l) m = fmaxf(m, fabsf(x[l]));
  return fmaxf(2.0f * m, fabsf(x[0]));
}
__device__ __forceinline__ bool m_skip(float s, float c, int q) {
  return s * c > (float)(q + 2) * (1.0f + 0x1p-12f);
}

// First-beta search for one block (App. F): the smallest t whose nearest E8 point of
// y = fl32(x * c_t) survives decode(encode(.)); t = k when every beta overloads.
//
// The overload test of a candidate P_t compares its root bound M(P_t) with 2q.  Since
// |M(P_t) - 2 M(y_t)| <= 2 sqrt(2) and M(y_t) = c_t M(x) up to fp32 rounding, the bound
// u_t = 2 c_t M(x) settles most betas without computing P_t: u_t - margin > 2q means t
// surely overloads (it is skipped), u_t + margin < 2q means it surely does not (no test).
// The margin 2 sqrt(2) + 0.02 + 2^-12 u_t covers the covering-radius term and the fp32
// rounding of y_t, M and u_t (together below 2^-19 u_t).  Only betas in between are computed and tested.
__device__ __forceinline__ void encode_block(const float (&v)[8], const float (&c)[4],
                                             const EncodeArgs& a, uint32_t& word, int& tsel) {
  if (a.decoder) {
    // NestQuantM: skip the betas its box rules out, then test each with its decoder
    const float st = m_stat(v);
    int t = 0;
    while (t < a.k - 1 && m_skip(st, pick4(c, t), a.q)) ++t;
    int P[8];
    for (;;) {
      float y[8];
      const float ct = pick4(c, t);
#pragma unroll
      for (int l = 0; l < 8; ++l) y[l] = v[l] * ct;
      nearest_e8(y, P);
      if (t == a.k - 1 || !overloaded_m(P, a.q, a.mq, a.m2q)) break;
      ++t;
    }
    tsel = t;
    word = encode_codes(P, a.q, a.rq, a.mq);
    return;
  }
  const float mx = root_bound_f(v);
  const float two_q = (float)(2 * a.q);
  int t = a.k - 1;
  bool sure = false;
#pragma unroll
  for (int s = a_max_k - 1; s >= 0; --s) {
    if (s < a.k) {
      const float u = 2.0f * c[s] * mx;
      const float margin = kRootMargin + u * 0x1p-12f;
      if (u - margin <= two_q) {   // not surely overloaded: the first such beta is the start
        t = s;
        sure = (u + margin < two_q);
      }
    }
  }
  int P[8];
  for (;;) {
    float y[8];
    const float ct = pick4(c, t);
#pragma unroll
    for (int l = 0; l < 8; ++l) y[l] = v[l] * ct;
    nearest_e8(y, P);
    if (t == a.k - 1 || sure || !overloaded(P, a.q, a.rq, a.mq, a.m2q)) break;
    ++t;
    const float u = 2.0f * pick4(c, t) * mx;
    sure = (u + kRootMargin + u * 0x1p-12f < two_q);
  }
  tsel = t;
  word = encode_codes(P, a.q, a.rq, a.mq);
}

// Fused encode-and-multiply: the decoded tile m_t * X2 of block j of `row`, stored where
// the product's decode stage would put it.  X2 is the lattice point P itself when P is known
// to be reproduced by the decoder (tile_from_x2), else the decode of the code word
// (tile_decoded); rows that are not coded get zeros.  |X2_l| <= 2q for a point that is
// kept, so m X2 is a full-rate 24-bit product.
__device__ __forceinline__ void tile_from_x2(const EncodeArgs& a, int64_t row, int j,
                                             const int (&X2)[8], int t) {
  const int m = (int)((a.mtab >> (8 * t)) & 0xFFu);
  const int64_t idx = row * a.nb_p + j;
  if (a.tile_et == ET_I8) {
    uint32_t lo = 0u, hi = 0u;
#pragma unroll
    for (int l = 0; l < 4; ++l) {
      // the low byte of m X2 from the operands' low 24 bits
      lo |= (umul24_v((uint32_t)m, (uint32_t)X2[l]) & 0xFFu) << (8 * l);
      hi |= (umul24_v((uint32_t)m, (uint32_t)X2[4 + l]) & 0xFFu) << (8 * l);
    }
    reinterpret_cast<u32x2*>(a.tiles)[idx] = u32x2{lo, hi};
  } else {
    uint32_t o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float lo = (float)__mul24(m, X2[2 * i]), hi = (float)__mul24(m, X2[2 * i + 1]);
      o[i] = a.tile_et == ET_F16 ? pack16<true>(lo, hi) : pack16<false>(lo, hi);
    }
    reinterpret_cast<u32x4*>(a.tiles)[idx] = u32x4{o[0], o[1], o[2], o[3]};
  }
}

__device__ __forceinline__ void tile_decoded(const EncodeArgs& a, int64_t row, int j, uint32_t word,
                                          int t) {
  const int m = (int)((a.mtab >> (8 * t)) & 0xFFu);
  const int64_t idx = row * a.nb_p + j;
  const int dv = decoder_variant(a.decoder, a.q);
  if (a.tile_et == ET_I8) {
    reinterpret_cast<u32x2*>(a.tiles)[idx] =
        dv == 0 ? decode_tile_i8<0>(word, m, a.q, a.m2q) : decode_tile_i8<1>(word, m, a.q, a.m2q);
  } else if (a.tile_et == ET_F16) {
    reinterpret_cast<u32x4*>(a.tiles)[idx] =
        dv == 0 ? decode_tile_16<0, true>(word, m, a.q, a.m2q)
                : (dv == 1 ? decode_tile_16<1, true>(word, m, a.q, a.m2q)
                           : decode_tile_16<2, true>(word, m, a.q, a.m2q));
  } else {
    reinterpret_cast<u32x4*>(a.tiles)[idx] =
        dv == 0 ? decode_tile_16<0, false>(word, m, a.q, a.m2q)
                : (dv == 1 ? decode_tile_16<1, false>(word, m, a.q, a.m2q)
                           : decode_tile_16<2, false>(word, m, a.q, a.m2q));
  }
}

__device__ __forceinline__ void tile_zero(const EncodeArgs& a, int64_t row, int j) {
  const int64_t idx = row * a.nb_p + j;
  if (a.tile_et == ET_I8) {
    reinterpret_cast<u32x2*>(a.tiles)[idx] = u32x2{0u, 0u};
  } else {
    reinterpret_cast<u32x4*>(a.tiles)[idx] = u32x4{0u, 0u, 0u, 0u};
  }
}

// Opt-beta for one block (App. F): every beta is tried; the code of the nearest point of
// y_t = fl32(x c_t) is decoded (Alg. 2 with the code's decoder) to X2_t and compared with
// the normalized block x / r: err_t = sum over l = 0..7, in that order, of d_l^2 with
// d_l = fl64(beta_t X2_t,l) / 2 - fl64(x_l / r), each step rounded in fp64 (the library is
// built without contraction).  The first t of least error is kept.
__device__ __forceinline__ void opt_block(const float (&v)[8], const float (&c)[4], float r,
                                          const EncodeArgs& a, uint32_t& word, int& tsel) {
  double xn[8];
#pragma unroll
  for (int l = 0; l < 8; ++l) xn[l] = (double)v[l] / (double)r;
  double best = INFINITY;
  word = 0u;
  tsel = 0;
#pragma unroll 1
  for (int t = 0; t < a.k; ++t) {
    const float ct = pick4(c, t);
    float y[8];
#pragma unroll
    for (int l = 0; l < 8; ++l) y[l] = v[l] * ct;
    int P[8];
    nearest_e8(y, P);
    const uint32_t w = encode_codes(P, a.q, a.rq, a.mq);
    // the byte decoder: X2_l + 128 in byte l of xs (bit-exact with the 16-bit-pair one)
    uint32_t xs[2];
    if (a.decoder) {
      decode_word_b8<true>(w, a.q, a.m2q, xs[0], xs[1]);
    } else {
      decode_word_b8<false>(w, a.q, a.m2q, xs[0], xs[1]);
    }
    // a select chain, not an indexed read of the argument block (a memory load)
    const double bt = t == 0 ? a.beta[0] : (t == 1 ? a.beta[1] : (t == 2 ? a.beta[2] : a.beta[3]));
    double err = 0.0;
#pragma unroll
    for (int l = 0; l < 8; ++l) {
      const int x2 = (int)((xs[l >> 2] >> (8 * (l & 3))) & 0xFFu) - 128;
      const double d = bt * (double)x2 / 2.0 - xn[l];
      err = err + d * d;
    }
    if (err < best) {
      best = err;
      word = w;
      tsel = t;
    }
  }
}

// Exact RN32(sqrt(S / n)) from a double-double S and a candidate r within a few ulps.
__device__ __forceinline__ float exact_rms(double hi, double lo, double n, float r) {
  for (int it = 0; it < 4; ++it) {
    const float up = next_up(r), dn = next_down(r);
    const int cu = cmp_sum_square(hi, lo, n, 0.5 * ((double)r + (double)up));
    if (cu > 0) { r = up; continue; }
    if (cu == 0) return (__float_as_uint(r) & 1u) ? up : r;
    if (r > 0.0f) {
      const int cd = cmp_sum_square(hi, lo, n, 0.5 * ((double)r + (double)dn));
      if (cd < 0) { r = dn; continue; }
      if (cd == 0) return (__float_as_uint(r) & 1u) ? dn : r;
    }
    break;
  }
  return r;
}

// The fp32 RMS candidate from an fp64 sum, and whether it is certainly RN32(sqrt(S / n)):
// the fp64 sum has relative error below 2^-46 here, so S farther than 2^-40 S from both
// rounding-boundary squares n m^2 settles the rounding.
__device__ __forceinline__ float rms_candidate(double s, double n, bool& sure) {
  const float r = (float)__builtin_sqrt(s / n);
  sure = true;
  if (s > 0.0 && r > 0.0f && isfinite(r)) {
    const double m_hi = 0.5 * ((double)r + (double)next_up(r));
    const double m_lo = 0.5 * ((double)r + (double)next_down(r));
    const double tol = s * 0x1p-40;
    sure = (n * m_hi * m_hi - s > tol) && (s - n * m_lo * m_lo > tol);
  }
  return r;
}

__device__ __forceinline__ void dd_add_square(double& hi, double& lo, float x) {
  const double sq = (double)x * (double)x;
  double t, e;
  two_sum(hi, sq, t, e);
  hi = t;
  lo += e;
}

// BPT > 0: the row's blocks stay in registers (read once).  BPT == 0: long rows are
// streamed, reading each block once for the scale and once more for the codes.  OPT: the
// Opt-beta strategy (opt_block) instead of First-beta; a separate instantiation, since its
// registers would lower the occupancy of the First-beta kernel.  TILES: also write the
// decoded tiles of the fused encode-and-multiply (likewise a separate instantiation).
template <typename T, int LANES, int BPT, bool OPT, bool TILES>
__global__ __launch_bounds__(LANES > 64 ? LANES : 256) void encode_kernel(
    const T* __restrict__ x, int64_t rows, int cols, int64_t ld_x, EncodeArgs a,
    uint32_t* __restrict__ codes, uint32_t* __restrict__ beta, float* __restrict__ scales) {
  constexpr int WG = LANES > 64 ? LANES : 256;
  constexpr int ROWS_PER_WG = WG / LANES;
  constexpr int NV = BPT > 0 ? BPT : 1;
  __shared__ double red[2 * (WG / 64)];

  const int lane = threadIdx.x % LANES;
  const int64_t row = (int64_t)blockIdx.x * ROWS_PER_WG + threadIdx.x / LANES;
  const bool row_ok = row < rows;  // uniform per group; whole-WG uniform when LANES > 64
  const int nb = cols >> 3;
  const int nbw = (nb + 15) >> 4;
  const T* xr = x + (row_ok ? row : 0) * ld_x;

  float v[NV][8];
  double s = 0.0;
  if constexpr (BPT > 0) {
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
      const int j = lane + i * LANES;
      if (row_ok && j < nb) {
        load_block<T>(xr + 8 * j, v[i]);
      } else {
#pragma unroll
        for (int l = 0; l < 8; ++l) v[i][l] = 0.0f;
      }
#pragma unroll
      for (int l = 0; l < 8; ++l) s = __builtin_fma((double)v[i][l], (double)v[i][l], s);
    }
  } else {
    for (int j = lane; row_ok && j < nb; j += LANES) {
      load_block<T>(xr + 8 * j, v[0]);
#pragma unroll
      for (int l = 0; l < 8; ++l) s = __builtin_fma((double)v[0][l], (double)v[0][l], s);
    }
  }
  s = group_sum<LANES>(s, red);

  const double n = (double)cols;
  bool sure;
  float r = rms_candidate(s, n, sure);
  // With LANES > 64 there is one row per workgroup and every thread holds the same s, so
  // this branch (which synchronizes the workgroup) is uniform.
  if (!sure) {
    double hi = 0.0, lo = 0.0;
    if constexpr (BPT > 0) {
#pragma unroll
      for (int i = 0; i < BPT; ++i)
#pragma unroll
        for (int l = 0; l < 8; ++l) dd_add_square(hi, lo, v[i][l]);
    } else {
      for (int j = lane; row_ok && j < nb; j += LANES) {
        float w[8];
        load_block<T>(xr + 8 * j, w);
#pragma unroll
        for (int l = 0; l < 8; ++l) dd_add_square(hi, lo, w[l]);
      }
    }
    group_sum_dd<LANES>(hi, lo, red);
    r = exact_rms(hi, lo, n, r);
  }

  const bool coded = (r > 0.0f) && isfinite(r);
  float c[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) c[t] = coded ? (float)(1.0 / ((double)r * a.beta[t])) : 0.0f;

  uint32_t* crow = codes + (row_ok ? row : 0) * nb;
  uint32_t* brow = beta + (row_ok ? row : 0) * nbw;
  const int iters = BPT > 0 ? BPT : (nb + LANES - 1) / LANES;
  constexpr int UNROLL = BPT > 0 ? BPT : 1;
#pragma unroll UNROLL
  for (int i = 0; i < iters; ++i) {
    const int j = lane + i * LANES;
    const bool mine = row_ok && j < nb;
    float* vb = v[BPT > 0 ? i : 0];
    if constexpr (BPT == 0) {
      if (mine) load_block<T>(xr + 8 * j, v[0]);
    }
    uint32_t word = 0;
    int tsel = 0;
    if (mine && coded) {
      if constexpr (OPT) {
        opt_block(*reinterpret_cast<float(*)[8]>(vb), c, r, a, word, tsel);
      } else {
        encode_block(*reinterpret_cast<float(*)[8]>(vb), c, a, word, tsel);
      }
    }
    if (mine) crow[j] = word;
    if (TILES && mine) {
      if (coded) {
        tile_decoded(a, row, j, word, tsel);
      } else {
        tile_zero(a, row, j);
      }
    }
    // two-bit beta indices: OR over the 16 consecutive blocks of one word
    uint32_t bits = mine ? ((uint32_t)tsel << (2 * (j & 15))) : 0u;
    constexpr int W = LANES < 16 ? LANES : 16;
#pragma unroll
    for (int m = 1; m < W; m <<= 1) bits |= __shfl_xor(bits, m, 64);
    if (mine && (j & 15) == 0) brow[j >> 4] = bits;
  }
  if (row_ok && lane == 0) scales[row] = r;
}

// ---------------------------------------------------------------------------------------
// Slot-compacted encoder (rows of up to 2048 blocks).
//
// A workgroup of four waves (two with LANES = 128) owns 64 * BPT blocks per wave ("slots"):
// slot s = 64 i + l of wave w is
// block j of row row_w, with
//   LANES <  64: row_w = i * (64 / LANES) + l / LANES, j = l % LANES  (a row per lane group
//                and pass; 64 / LANES * BPT rows per wave)
//   LANES == 64: row_w = 0, j = l + 64 i                              (one row per wave)
//   LANES >  64: row_w = 0, j = 64 w + l + LANES i                   (one row per workgroup
//                of LANES / 64 waves)
// Phase 0 reads every slot from HBM once (all of a lane's loads in flight together), stages
// it in LDS and forms the row sums of squares; then one lane per row (one per beta, with one
// row per workgroup) turns its sum into the scale r, the multipliers c_t and the thresholds
// of skip_threshold.  Phase 1 evaluates every slot at the first beta the root bound of x
// does not rule out, with the fp32 nearest-point decision, and finishes it unless that
// decision was too close to call or the point's exact root bound says it overloads (both
// queued, at the same and at the next beta), or the point lies on the cell boundary (kept
// with its point in a boundary list).  Phase 2a runs the literal test on the boundary list;
// phase 2 then finishes the queued slots (8.6% of the blocks on heavy-tailed Student-t rows,
// fewer on Gaussian ones, plus the boundary points that overload) in rounds of one beta
// each, the slots still searching compacted after every round so that the lanes stay busy.
// With tiles, slots at the last beta whose point is not strictly inside the cell are queued
// too, so that phase 1 never runs the decoder (full decoder only).
// Two-bit beta indices are staged in LDS and packed into words at the end.
// ---------------------------------------------------------------------------------------
template <int LANES, int BPT>
struct SlotMap {
  static constexpr bool WGROW = LANES > 64;
  static constexpr int RPP = LANES < 64 ? 64 / LANES : 1;           // rows per pass
  static constexpr int ROWS_PER_WAVE = LANES < 64 ? RPP * BPT : 1;
  static constexpr int SLOTS = 64 * BPT;
  __device__ static int row_w(int i, int l) { return LANES < 64 ? i * RPP + l / LANES : 0; }
  // row_w(i, l) = row_step(i) + row_w(0, l), the first term the same for every lane
  __device__ static constexpr int row_step(int i) { return LANES < 64 ? i * RPP : 0; }
  __device__ static int j(int i, int l, int wave) {
    return LANES < 64 ? l % LANES : (LANES == 64 ? l + 64 * i : 64 * wave + l + LANES * i);
  }
  // inverse map for block j of row row_w: wave and slot
  __device__ static void slot_of(int row_w, int j, int wave_hint, int& w, int& s) {
    if constexpr (LANES < 64) {
      w = wave_hint;
      s = (row_w / RPP) * 64 + (row_w % RPP) * LANES + j;
    } else if constexpr (LANES == 64) {
      w = wave_hint;
      s = j;
    } else {
      const int rem = j % LANES;
      w = rem >> 6;
      s = (j / LANES) * 64 + (rem & 63);
    }
  }
};

// One evaluation of a queued block at beta t: its exact nearest point P, and whether the
// search stops there (the last beta, or a point that does not overload).  The root bound of
// x is not consulted: the integer root bound of P settles every point off the cell
// boundary, and a point it cannot settle is decided by the literal test.
__device__ __forceinline__ bool eval_block(const float (&v)[8], float ct, int t,
                                           const EncodeArgs& a, int (&P)[8]) {
  float y[8];
#pragma unroll
  for (int l = 0; l < 8; ++l) y[l] = v[l] * ct;
  nearest_e8(y, P);
  if (t == a.k - 1) return true;
  return a.decoder ? !overloaded_m(P, a.q, a.mq, a.m2q)
                   : !overloaded(P, a.q, a.rq, a.mq, a.m2q);
}

// Raw input of one block: 16 B for 16-bit types, 32 B for fp32.
template <typename T> struct RawBlock { u32x4 w; };
template <> struct RawBlock<float> { f32x4 a, b; };

template <typename T>
__device__ __forceinline__ void load_raw(const T* __restrict__ p, RawBlock<T>& r) {
  r.w = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
template <>
__device__ __forceinline__ void load_raw<float>(const float* __restrict__ p, RawBlock<float>& r) {
  r.a = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
  r.b = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p) + 1);
}
template <typename T>
__device__ __forceinline__ void zero_raw(RawBlock<T>& r) { r.w = u32x4{0u, 0u, 0u, 0u}; }
template <>
__device__ __forceinline__ void zero_raw<float>(RawBlock<float>& r) {
  r.a = f32x4{0.f, 0.f, 0.f, 0.f};
  r.b = r.a;
}
template <typename T>
__device__ __forceinline__ void unpack_raw(const RawBlock<T>& r, float (&v)[8]);
template <>
__device__ __forceinline__ void unpack_raw<float>(const RawBlock<float>& r, float (&v)[8]) {
  v[0] = r.a.x; v[1] = r.a.y; v[2] = r.a.z; v[3] = r.a.w;
  v[4] = r.b.x; v[5] = r.b.y; v[6] = r.b.z; v[7] = r.b.w;
}
template <>
__device__ __forceinline__ void unpack_raw<uint16_t>(const RawBlock<uint16_t>& r, float (&v)[8]) {
  const uint32_t w[4] = {r.w.x, r.w.y, r.w.z, r.w.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(w[i] << 16);
    v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
template <>
__device__ __forceinline__ void unpack_raw<_Float16>(const RawBlock<_Float16>& r, float (&v)[8]) {
  const uint32_t w[4] = {r.w.x, r.w.y, r.w.z, r.w.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w[i] & 0xffffu));
    v[2 * i + 1] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w[i] >> 16));
  }
}

// Threshold on the root bound M(x) of a block above which beta t surely overloads: for the
// nearest point P of y = fl32(c x), M(P) >= 2 M(y) - 2 sqrt(2) (covering radius 1, roots of
// norm sqrt(2)) and M(y) = c M(x) up to relative rounding errors below 2^-19 (y, and the
// fp32 evaluation of M), so M(x) > (2q + 2 sqrt(2) + 0.02) / (2 c (1 - 2^-12)) implies
// M(P) > 2q.  With rb = fl64(r beta_t) and c = fl32(fl64(1 / rb)), 1 / c <= rb (1 + 2^-23),
// so the threshold is evaluated from rb with products only (no division), inflated by 2^-20
// to cover their roundings, and rounded up.  A threshold a little above the exact one only
// lets a block try a beta that overloads; the search still ends at the same beta.
// The NestQuantM counterpart for the statistic m_stat: (q + 2)(1 + 2^-12) / c.
__device__ __forceinline__ float round_up_f32(double v) {
  float f = (float)v;
  if ((double)f < v) f = next_up(f);
  return f;
}

__device__ __forceinline__ float skip_threshold_m(double rb, int q) {
  return round_up_f32((double)(q + 2) * (1.0 + 0x1p-12) * rb * (1.0 + 0x1p-20));
}

__device__ __forceinline__ float skip_threshold(double rb, int q) {
  return round_up_f32((2.0 * q + (double)kRootMargin) * (0.5 / (1.0 - 0x1p-12)) * rb *
                      (1.0 + 0x1p-20));
}

// ROT (one row per workgroup only): the row is first rotated in LDS (rotate_rows_lds, the
// arithmetic of nq_rotate) and the encoder reads its blocks from there, times a.rot_s.
template <typename T, int LANES, int BPT, bool TILES, bool ROT>
// Workgroups of a row (LANES 128 and 256) are held to 96 VGPRs, five waves per SIMD: the
// fused launch (W's tile decode beside the coding of A) measured 94.9-95.1 against
// 96.2-96.4 us per q_proj step at 97 VGPRs (four waves, no spills), and the 70B MLP step
// 976-982 against 991-997 us (two dwords of scratch in its fused instantiation).  The
// 64-lane instantiation with one block per thread (rows of at most 64 blocks) gets the same
// bound: its fused instantiation fits it without scratch.
__global__ __launch_bounds__(LANES > 64 ? LANES : 256)
__attribute__((amdgpu_waves_per_eu(LANES >= 128 || (LANES == 64 && BPT == 1) ? 5 : 1))) void encode_wave_kernel(
    const T* __restrict__ x, int64_t rows, int cols, int64_t ld_x, EncodeArgs a,
    uint32_t* __restrict__ codes, uint32_t* __restrict__ beta, float* __restrict__ scales) {
  using SM = SlotMap<LANES, BPT>;
  constexpr int SLOTS = SM::SLOTS;
  constexpr int RW = SM::ROWS_PER_WAVE;
  constexpr int CW = SM::WGROW ? 1 : 4;          // row tables: per wave, or one per workgroup
  constexpr int NW = (LANES > 64 ? LANES : 256) / 64;   // waves per workgroup: 4, or 2
  static_assert(NW == 4 || NW == 2, "four or two waves per workgroup");
  static_assert(!ROT || LANES == 256, "rotation in LDS needs one row per 256-lane workgroup");
  __shared__ RawBlock<T> rawl[NW][ROT ? 1 : SLOTS];
  __shared__ __attribute__((aligned(16))) float rbuf[ROT ? 8 * 4 * SLOTS : 1];
  constexpr int BQ = SLOTS < 256 ? SLOTS : 256;   // room in the boundary list
  __shared__ uint16_t queue[NW][SLOTS];
  __shared__ uint16_t qnext[NW * SLOTS];
  __shared__ int qcnt[4];
  __shared__ uint16_t bq[BQ];                      // boundary slots: w << 11 | sl << 2 | t
  __shared__ uint2 bp[BQ];                         // and their points, as signed bytes
  __shared__ int bcnt;
  __shared__ uint8_t tsl[NW][SLOTS];
  __shared__ float crow[CW][RW][4];
  __shared__ __attribute__((aligned(16))) float chi[CW][RW][4];
  __shared__ float rrow[CW][RW];
  __shared__ double rsum[NW][RW];
  __shared__ int qlen[NW];

  // A TileTask's a.task.wgs workgroups come last in the grid for rows of up to 1024 blocks:
  // dispatched once every row has started, they fill the CUs that the encoder's last rows
  // leave idle.  For longer rows (8 blocks per lane, many rounds of encoder workgroups) they
  // come first.  Measured on the fused step: q_proj 98 (last) against 102.6 us (first),
  // down_proj 546 (last) against 529 us (first), the 70B MLP 988 against 992 us; spreading
  // them among the encoder's workgroups was slower in every case.
  constexpr bool TASK_FIRST = BPT == 8;
  int64_t bid = blockIdx.x;
  if constexpr (TILES && SM::WGROW) {
    if constexpr (TASK_FIRST) {
      if (bid < a.task.wgs) {
        run_tile_task<NW * 64>(a.task, a.tile_et, bid);
        return;
      }
      bid -= a.task.wgs;
    } else {
      const int64_t first = (int64_t)gridDim.x - a.task.wgs;
      if (bid >= first) {
        run_tile_task<NW * 64>(a.task, a.tile_et, bid - first);
        return;
      }
    }
  }
  // the wave index is uniform over the wave: held in a scalar register, so that row offsets
  // derived from it are scalar arithmetic
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int lane = threadIdx.x & 63;
  const int cw = SM::WGROW ? 0 : wave;
  const int nb = cols >> 3;
  const int nbw = (nb + 15) >> 4;
  auto row_base = [&](int w) -> int64_t {
    return SM::WGROW ? bid : (bid * 4 + w) * RW;
  };
  const int64_t row0 = row_base(wave);
  const double n = (double)cols;
  // index of block j of row row_base(w) + rw in the code words: rows of more than 64 blocks
  // have rw = 0, shorter rows w RW + rw < 2^12 and nb <= 64, a 24-bit product
  auto code_at = [&](int w, int rw, int j) -> int64_t {
    if constexpr (SM::WGROW) return row_base(w) * nb + j;
    return (bid * 4 * RW) * (int64_t)nb + __mul24(w * RW + rw, nb) + j;
  };
  // block of slot sl of wave w, as fp32
  auto slot_block = [&](int w, int sl, float (&v)[8]) {
    if constexpr (ROT) {
      const int pe = lds_pos(8 * SM::j(sl >> 6, sl & 63, w));
#pragma unroll
      for (int l = 0; l < 8; ++l) v[l] = rbuf[pe ^ l] * a.rot_s;
    } else {
      unpack_raw<T>(rawl[w][sl], v);
    }
  };

  if (threadIdx.x < 4) qcnt[threadIdx.x] = 0;   // phase 2's list lengths, one per round
  if (threadIdx.x == 0) bcnt = 0;

  // ---- phase 0: stage the slots in LDS, row sums of squares ----
  if constexpr (ROT) {
    // the whole workgroup rotates its row (uniform: one row per workgroup)
    if (row0 < rows) rotate_rows_lds<T>(x + row0 * ld_x, ld_x, 1, cols, a.rot_p, a.rot_lp, rbuf);
    double part = 0.0;
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
      const int j = SM::j(i, lane, wave);
      if (row0 < rows && j < nb) {
        float v[8];
        slot_block(wave, i * 64 + lane, v);
        double s = 0.0;
#pragma unroll
        for (int l = 0; l < 8; ++l) s = __builtin_fma((double)v[l], (double)v[l], s);
        part += s;
      }
    }
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) part += __shfl_xor(part, m, 64);
    if (lane == 0) rsum[wave][0] = part;
  } else {
    RawBlock<T> raw[BPT];
    // one 64-bit row offset per lane; the rest of each block's address is uniform
    const T* __restrict__ x_lane = x + (row0 + SM::row_w(0, lane)) * ld_x;
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
      const int rw = SM::row_w(i, lane), j = SM::j(i, lane, wave);
      const int64_t row = row0 + rw;
      if (row < rows && j < nb) {
        load_raw<T>(x_lane + SM::row_step(i) * ld_x + 8 * j, raw[i]);
      } else {
        zero_raw<T>(raw[i]);
      }
    }
    double part = 0.0;
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
      rawl[wave][i * 64 + lane] = raw[i];
      float v[8];
      unpack_raw<T>(raw[i], v);
      double s = 0.0;
#pragma unroll
      for (int l = 0; l < 8; ++l) s = __builtin_fma((double)v[l], (double)v[l], s);
      if constexpr (LANES < 64) {
#pragma unroll
        for (int m = 1; m < LANES; m <<= 1) s += __shfl_xor(s, m, 64);
        if (lane % LANES == 0) rsum[wave][SM::row_w(i, lane)] = s;
      } else {
        part += s;
      }
    }
    if constexpr (LANES >= 64) {
#pragma unroll
      for (int m = 1; m < 64; m <<= 1) part += __shfl_xor(part, m, 64);
      if (lane == 0) rsum[wave][0] = part;
    }
  }
  __syncthreads();

  // ---- row scales and multipliers ----
  // One lane per row; with one row per workgroup, lanes 0-3 of wave 0 all find the scale
  // (the same instructions) and then each the multiplier and threshold of its own beta.
  {
    constexpr int TL = SM::WGROW ? 4 : 1;   // lanes per row
    const bool mine = SM::WGROW ? threadIdx.x < TL : lane < RW;
    const int rw = SM::WGROW ? 0 : lane;
    const int64_t row = row0 + rw;
    if (mine && row < rows) {
      double s = rsum[wave][rw];
      if constexpr (SM::WGROW) {
        s = rsum[0][0];
#pragma unroll
        for (int w = 1; w < NW; ++w) s += rsum[w][0];
      }
      bool sure;
      float r = rms_candidate(s, n, sure);
      if (!sure) {
        // rare: the double-double sum of the row, block by block from LDS
        double hi = 0.0, lo = 0.0;
        for (int j = 0; j < nb; ++j) {
          int w, sl;
          SM::slot_of(rw, j, wave, w, sl);
          float v[8];
          slot_block(w, sl, v);
#pragma unroll
          for (int l = 0; l < 8; ++l) dd_add_square(hi, lo, v[l]);
        }
        double t, e;
        two_sum(hi, lo, t, e);
        r = exact_rms(t, e, n, r);
      }
      const bool coded = (r > 0.0f) && isfinite(r);
      auto set_beta = [&](int t) {
        const double rb = (double)r * a.beta[t];
        crow[cw][rw][t] = coded ? (float)(1.0 / rb) : 0.0f;
        chi[cw][rw][t] = (coded && t < a.k - 1)
                             ? (a.decoder ? skip_threshold_m(rb, a.q) : skip_threshold(rb, a.q))
                             : INFINITY;
      };
      if constexpr (SM::WGROW) {
        set_beta((int)threadIdx.x);
      } else {
#pragma unroll
        for (int t = 0; t < 4; ++t) set_beta(t);
      }
      if (SM::WGROW ? threadIdx.x == 0 : true) {
        rrow[cw][rw] = coded ? r : 0.0f;
        scales[row] = r;
      }
    }
  }
  __syncthreads();

  // ---- phase 1: every slot at its predicted beta ----
  uint32_t* __restrict__ codes_w = codes + row0 * nb;   // this wave's rows
  int qn = 0;   // queue length, uniform over the wave
#pragma unroll 1
  for (int i = 0; i < BPT; ++i) {
    const int sl = i * 64 + lane;
    const int rw = SM::row_w(i, lane), j = SM::j(i, lane, wave);
    const int64_t row = row0 + rw;
    const bool valid = row < rows && j < nb;
    const bool coded = valid && rrow[cw][rw] != 0.0f;
    bool queued = false, bnd = false;
    int start = 0, t0 = 0, amax = 0;
    int P[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (coded) {
      float v[8];
      slot_block(wave, sl, v);
      // first beta whose point is not surely overloaded: one threshold test per beta
      const float mx = a.decoder ? m_stat(v) : root_bound_f(v);
      const f32x4 hi = *reinterpret_cast<const f32x4*>(chi[cw][rw]);
      t0 = mx > hi.x ? (mx > hi.y ? (mx > hi.z ? 3 : 2) : 1) : 0;
      const float ct = crow[cw][rw][t0];
      float y[8];
#pragma unroll
      for (int l = 0; l < 8; ++l) y[l] = v[l] * ct;
      if (!nearest_e8_fast(y, P)) {
        queued = true;                 // decision too close for fp32: redo exactly
        start = t0;
      } else if (a.decoder) {
        amax = 1 << 30;                // not known: encode_codes finds it
        if (t0 < a.k - 1 && overloaded_m(P, a.q, a.mq, a.m2q)) {   // its decoder decides
          queued = true;
          start = t0 + 1;
        }
      } else {
        const int M = e8_root_bound(P, amax);
        if (t0 < a.k - 1) {
          if (M > 2 * a.q) {           // overloads: the next beta, later
            queued = true;
            start = t0 + 1;
          } else if (M == 2 * a.q) {   // on the boundary: the literal test decides, later
            bnd = true;
          }
        } else if (TILES && M >= 2 * a.q) {
          // the last beta, where a point may overload: only a point strictly inside the
          // cell is its own decode; the others take the decoder's tile in phase 2
          queued = true;
          start = t0;
        }
      }
    }
    // boundary points go to the boundary list with P (|P_l| <= 2q), while it has room, and
    // to the queue at the same beta otherwise
    const uint64_t lanes_below = (1ull << lane) - 1ull;
    bool listed = false;
    const uint64_t bmask = __ballot(bnd);
    if (bmask != 0) {
      int b0 = 0;
      if (lane == 0) b0 = atomicAdd(&bcnt, __popcll(bmask));
      b0 = __shfl(b0, 0, 64);
      if (bnd) {
        const int bi = b0 + __popcll(bmask & lanes_below);
        if (bi < BQ) {
          listed = true;
          bq[bi] = (uint16_t)((wave << 11) | (sl << 2) | t0);
          // low bytes of P_0..P_3 and P_4..P_7 (byte selects 0 and 4 of each pair; 12 = zero)
          auto pack4 = [](int p0, int p1, int p2, int p3) {
            return __builtin_amdgcn_perm((uint32_t)p1, (uint32_t)p0, 0x0C0C0400u) |
                   __builtin_amdgcn_perm((uint32_t)p3, (uint32_t)p2, 0x04000C0Cu);
          };
          bp[bi] = uint2{pack4(P[0], P[1], P[2], P[3]), pack4(P[4], P[5], P[6], P[7])};
        } else {
          queued = true;
          start = t0;
        }
      }
    }
    const uint64_t mask = __ballot(queued);
    if (queued) {
      const int pos = qn + __popcll(mask & lanes_below);
      queue[wave][pos] = (uint16_t)((sl << 2) | start);
    } else if (valid && !listed) {
      uint32_t word = 0u;
      if (coded) {
        word = amax < (1 << 30) ? encode_codes_amax(P, a.q, a.rq, a.mq, amax)
                                : encode_codes(P, a.q, a.rq, a.mq);
      }
      codes_w[__mul24(rw, nb) + j] = word;   // rw = 0 or nb <= 64
      tsl[wave][sl] = (uint8_t)t0;
      if constexpr (TILES) {
        // a point kept here passed the overload test or lies strictly inside the cell, so
        // X2 = P (zero for rows that are not coded); the NestQuantM decoder has no such
        // bound at the last beta, where its tile is decoded
        if (coded && a.decoder && t0 == a.k - 1) {
          tile_decoded(a, row, j, word, t0);
        } else {
          tile_from_x2(a, row, j, P, t0);
        }
      }
    }
    qn += __popcll(mask);
  }
  if (lane == 0) qlen[wave] = qn;
  __syncthreads();

  // ---- phase 2a: the boundary list, where P is known: the literal test alone ----
  // A point that passes is coded at its beta; the others join their wave's queue at the
  // next beta (each slot is in one list only, so the queues have room).
  {
    const int nbq = min(bcnt, BQ);
    if (nbq > 0) {
      for (int idx = threadIdx.x; idx < nbq; idx += NW * 64) {
        const uint32_t e = bq[idx];
        const int w = (int)(e >> 11), sl = (int)((e >> 2) & 511u), t = (int)(e & 3u);
        const uint2 pb = bp[idx];
        int P[8];
#pragma unroll
        for (int l = 0; l < 4; ++l) {
          P[l] = (int)(int8_t)(uint8_t)(pb.x >> (8 * l));
          P[4 + l] = (int)(int8_t)(uint8_t)(pb.y >> (8 * l));
        }
        if (!boundary_overloaded(P, a.q, a.mq, a.m2q)) {
          const int i = sl >> 6, l = sl & 63;
          const int rw = SM::row_w(i, l), j = SM::j(i, l, w);
          const int64_t row = row_base(w) + rw;
          const uint32_t word = encode_codes_amax(P, a.q, a.rq, a.mq, 2 * a.q);  // |P_l| <= 2q
          codes[code_at(w, rw, j)] = word;
          tsl[w][sl] = (uint8_t)t;
          if constexpr (TILES) tile_from_x2(a, row, j, P, t);
        } else {
          const int pos = atomicAdd(&qlen[w], 1);
          queue[w][pos] = (uint16_t)((sl << 2) | (t + 1));
        }
      }
      __syncthreads();
    }
  }

  // ---- phase 2: the queued slots of the whole workgroup, one beta per round ----
  // Round 0 takes the four wave queues; a slot whose point overloads goes on to the next
  // beta in the next round, through a compacted list (entries w << 11 | sl << 2 | t), so
  // that every round keeps its lanes busy instead of each wave looping until its slowest
  // lane is done.  There are at most k rounds (t grows by one per round, and t = k - 1
  // always stops).
  {
    int qs[NW + 1];   // starts of the wave queues in round 0's index space
    qs[0] = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) qs[w + 1] = qs[w] + qlen[w];
    int n = qs[NW];
#pragma unroll 1
    for (int rd = 0; n > 0; ++rd) {
      uint16_t* __restrict__ out_q = (rd & 1) ? &queue[0][0] : qnext;
      const uint16_t* __restrict__ in_q = (rd & 1) ? qnext : &queue[0][0];
#pragma unroll 1
      for (int base = 0; base < n; base += NW * 64) {
        const int idx = base + (int)threadIdx.x;
        bool more = false;
        uint32_t next = 0;
        if (idx < n) {
          int w, sl, t;
          if (rd == 0) {
            int off;
            if constexpr (NW == 4) {
              w = (idx >= qs[1]) + (idx >= qs[2]) + (idx >= qs[3]);
              off = w == 0 ? 0 : (w == 1 ? qs[1] : (w == 2 ? qs[2] : qs[3]));
            } else {
              w = idx >= qs[1];
              off = w ? qs[1] : 0;
            }
            const uint32_t e = queue[w][idx - off];
            sl = (int)(e >> 2);
            t = (int)(e & 3u);
          } else {
            const uint32_t e = in_q[idx];
            w = (int)(e >> 11);
            sl = (int)((e >> 2) & 511u);
            t = (int)(e & 3u);
          }
          const int i = sl >> 6, l = sl & 63;
          const int rw = SM::row_w(i, l), j = SM::j(i, l, w);
          const int64_t row = row_base(w) + rw;
          const int c2 = SM::WGROW ? 0 : w;
          float v[8];
          slot_block(w, sl, v);
          int P[8];
          if (eval_block(v, crow[c2][rw][t], t, a, P)) {
            const uint32_t word = encode_codes(P, a.q, a.rq, a.mq);
            codes[code_at(w, rw, j)] = word;
            tsl[w][sl] = (uint8_t)t;
            if constexpr (TILES) {
              if (t < a.k - 1) {
                tile_from_x2(a, row, j, P, t);
              } else {
                tile_decoded(a, row, j, word, t);
              }
            }
          } else {
            more = true;
            next = ((uint32_t)w << 11) | ((uint32_t)sl << 2) | (uint32_t)(t + 1);
          }
        }
        // wave-aggregated append to the next round's list
        const uint64_t mask = __ballot(more);
        if (mask != 0) {
          int pos0 = 0;
          if (lane == 0) pos0 = atomicAdd(&qcnt[rd], __popcll(mask));
          pos0 = __shfl(pos0, 0, 64);
          if (more) out_q[pos0 + __popcll(mask & ((1ull << lane) - 1ull))] = (uint16_t)next;
        }
      }
      __syncthreads();
      n = qcnt[rd];
    }
  }

  // ---- beta words: 16 two-bit indices of consecutive blocks (consecutive lanes) ----
  // Block j sits in lane j mod 16 of its group of 16 lanes (j mod 8 of 8 when rows have 8
  // blocks): each lane shifts its own index into place and an OR across the group forms the
  // word, which the group's first lane stores.
  constexpr int G = LANES < 16 ? LANES : 16;
  uint32_t* __restrict__ beta_w = beta + row0 * nbw;   // this wave's rows
#pragma unroll
  for (int i = 0; i < BPT; ++i) {
    const int rw = SM::row_w(i, lane), j = SM::j(i, lane, wave);
    const int64_t row = row0 + rw;
    const bool ok = row < rows && j < nb;
    uint32_t bits = ok ? (uint32_t)tsl[wave][i * 64 + lane] << (2 * (j & 15)) : 0u;
#pragma unroll
    for (int m = 1; m < G; m <<= 1) bits |= (uint32_t)__shfl_xor((int)bits, m, 64);
    if (ok && (j & 15) == 0) beta_w[__mul24(rw, nbw) + (j >> 4)] = bits;   // rw = 0 or nbw <= 4
  }
}

// ---------------------------------------------------------------------------------------
// launch
// ---------------------------------------------------------------------------------------
template <typename T, int LANES, int BPT, bool OPT, bool TILES>
static hipError_t launch_t(const void* x, int64_t rows, int cols, int64_t ld_x,
                           const EncodeArgs& a, uint32_t* codes, uint32_t* beta, float* scales,
                           hipStream_t st) {
  constexpr int WG = LANES > 64 ? LANES : 256;
  constexpr int RPW = WG / LANES;
  const int64_t grid = (rows + RPW - 1) / RPW;
  hipLaunchKernelGGL((encode_kernel<T, LANES, BPT, OPT, TILES>), dim3((unsigned)grid), dim3(WG), 0, st,
                     (const T*)x, rows, cols, ld_x, a, codes, beta, scales);
  return hipGetLastError();
}

template <typename T, int LANES, int BPT, bool TILES, bool ROT = false>
static hipError_t launch_w(const void* x, int64_t rows, int cols, int64_t ld_x,
                           const EncodeArgs& a, uint32_t* codes, uint32_t* beta, float* scales,
                           hipStream_t st) {
  using SM = SlotMap<LANES, BPT>;
  constexpr int WG = LANES > 64 ? LANES : 256;
  const int64_t rows_per_wg = SM::WGROW ? 1 : 4 * SM::ROWS_PER_WAVE;
  int64_t grid = (rows + rows_per_wg - 1) / rows_per_wg;
  if (TILES && SM::WGROW) grid += a.task.wgs;
  hipLaunchKernelGGL((encode_wave_kernel<T, LANES, BPT, TILES, ROT>), dim3((unsigned)grid), dim3(WG), 0, st,
                     (const T*)x, rows, cols, ld_x, a, codes, beta, scales);
  return hipGetLastError();
}

template <typename T, bool TILES>
static hipError_t launch_dtype(const void* x, int64_t rows, int cols, int64_t ld_x,
                               const EncodeArgs& a, uint32_t* codes, uint32_t* beta,
                               float* scales, hipStream_t st) {
  const int nb = cols / 8;
  if (a.rot_p) {
    // rows rotated in LDS first: one row per workgroup
#define NQ_R(B) return launch_w<T, 256, B, TILES, true>(x, rows, cols, ld_x, a, codes, beta, scales, st)
    if (!encode_rotates(cols, a.strategy)) return hipErrorInvalidValue;
    if (nb <= 512) NQ_R(2);
    if (nb <= 1024) NQ_R(4);
    NQ_R(8);
#undef NQ_R
  }
  if (a.strategy) {
    // Opt-beta: a lane group of up to 64 holds short rows in registers; longer rows stream
#define NQ_O(L, B) return launch_t<T, L, B, true, TILES>(x, rows, cols, ld_x, a, codes, beta, scales, st)
    if (nb <= 8) NQ_O(8, 1);
    if (nb <= 16) NQ_O(16, 1);
    if (nb <= 32) NQ_O(32, 1);
    if (nb <= 64) NQ_O(64, 1);
    if (nb <= 2048) NQ_O(256, 0);
    NQ_O(1024, 0);
#undef NQ_O
  }
#define NQ_W(L, B) return launch_w<T, L, B, TILES>(x, rows, cols, ld_x, a, codes, beta, scales, st)
#define NQ_L(L, B) return launch_t<T, L, B, false, TILES>(x, rows, cols, ld_x, a, codes, beta, scales, st)
  // short rows: several rows per lane group, 256 blocks per wave when there are enough rows
  // (with 512 the staged blocks took 51 KB of LDS per workgroup of fp16 rows, three
  // workgroups per CU: the 2^21 x 128 fp16 matrix 555 against 509-511 us); rows of 33-64
  // blocks have one row per wave, one block per lane
  if (nb <= 8) { if (rows >= 2048) NQ_W(8, 4); NQ_W(8, 1); }
  if (nb <= 16) { if (rows >= 1024) NQ_W(16, 4); NQ_W(16, 1); }
  if (nb <= 32) { if (rows >= 512) NQ_W(32, 4); NQ_W(32, 1); }
  if (nb <= 64) NQ_W(64, 1);
  if (nb <= 128) NQ_W(64, 2);
  if (nb <= 256) NQ_W(64, 4);
  // 257..512 blocks: with many rows, one row per two waves keeps the launch to a single wave
  // of workgroups over the CUs; with few rows, four waves per row finish each row sooner
  if (nb <= 512) { if (rows > 1024) NQ_W(128, 4); NQ_W(256, 2); }
  if (nb <= 1024) NQ_W(256, 4);
  if (nb <= 2048) NQ_W(256, 8);
  if (nb <= 4096) NQ_L(512, 8);
  NQ_L(1024, 0);
#undef NQ_W
#undef NQ_L
}

hipError_t launch_encode(const void* x, int dtype, int64_t rows, int cols, int64_t ld_x,
                         const EncodeArgs& a, uint32_t* codes, uint32_t* beta, float* scales,
                         hipStream_t st) {
  if (a.task.wgs > 0 && !(a.tiles && encode_carries_task(cols, a.strategy)))
    return hipErrorInvalidValue;
  if (a.tiles) {
    switch (dtype) {
      case 0: return launch_dtype<float, true>(x, rows, cols, ld_x, a, codes, beta, scales, st);
      case 1: return launch_dtype<_Float16, true>(x, rows, cols, ld_x, a, codes, beta, scales, st);
      default: return launch_dtype<uint16_t, true>(x, rows, cols, ld_x, a, codes, beta, scales, st);
    }
  }
  switch (dtype) {
    case 0: return launch_dtype<float, false>(x, rows, cols, ld_x, a, codes, beta, scales, st);
    case 1: return launch_dtype<_Float16, false>(x, rows, cols, ld_x, a, codes, beta, scales, st);
    default: return launch_dtype<uint16_t, false>(x, rows, cols, ld_x, a, codes, beta, scales, st);
  }
}

}  // namespace nq
