// Alg. 2 (Voronoi decode, with the Gosset oracle of Alg. 5 or NestQuantM's of App. D) on one
// code word, four coordinates per 32-bit register (byte SIMD), for every q <= 16.  Included
// by nq_device.hpp inside namespace nq (it needs u16x2, bcnt_add and the amdgcn byte builtins).
//
// The arithmetic and tie rules of Alg. 5 (nq_device.hpp): X = G c, then X - q * 2 Q(X / 2q)
// in exact integers, every distance times 2q.  Why bytes suffice:
//   * every X = G c fits a byte: X4 = c0 + 4 c1 + 2 (c2 + ... + c7) <= 255 and the others
//     are below 3q <= 48;
//   * f = X mod 2q and d = floor(X / 2q) (in {0, 1} except for X4): with 128 - 2q added to
//     every byte (no carry: all sums stay below 256), bit 7 of a byte says X >= 2q, and then
//     the byte's low seven bits are X - 2q.  X4 alone is divided (a 24-bit multiply);
//   * g = [f > q] (an exact half rounds down) is bit 7 of f + 127 - q;
//   * the distance to the nearest integer, times 2q, is E = min(f, 2q - f) = g ? 2q - f : f
//     (2q - f never borrows since f < 2q).  Alg. 5's D8 fix goes to argmax E and its D8+1/2
//     fix to argmin E, lowest index on ties: the keys 256 E + 7 - l (max) and 256 E + l (min)
//     are reduced in 16-bit lanes;
//   * the gap of Alg. 5 times 2q is sum E - 4q + odd1 (2q - 2 E_p) - odd2 2 E_r, with
//     odd2 = sum d mod 2 (popcounts of the bit-7 masks plus floor(X4 / 2q)) and
//     odd1 = (odd2 + #g) mod 2; D8 iff it is negative;
//   * the residuals D8: f - 2q g and D8+1/2: f - q, and the fix of +-2q at one coordinate,
//     are formed on values biased by 128 (every byte then lies in [80, 176]), so that no byte
//     borrows from or carries into its neighbour.
// NestQuantM (M): both fixes at coordinate 0, no argmin / argmax.
//
// Output: xa holds coordinates 0-3 and xb coordinates 4-7, byte l = X2_l + 128.
#pragma once

template <bool M = false>
__device__ __forceinline__ void decode_word_b8(uint32_t w, int q, uint32_t m2q, uint32_t& xa,
                                               uint32_t& xb) {
  const uint32_t den = 2u * (uint32_t)q;
  // per-byte constants (q is uniform): scalar multiplies, except qb, a select operand (which
  // must be a vector register) broadcast once by v_perm
  const uint32_t q2 = den * 0x01010101u;                      // 2q
  const uint32_t c1 = (128u - den) * 0x01010101u;             // 128 - 2q
  const uint32_t c2 = (127u - (uint32_t)q) * 0x01010101u;     // 127 - q
  const uint32_t qb = __builtin_amdgcn_perm(0u, (uint32_t)q, 0x00000000u);   // q

  // X = G c: (X0..X3) = c0 + 2 (0, c2, c4, c6); (X4..X7) = c0 + 2 (c1 + sum c - c0, c3, c5, c7)
  const uint32_t E = w & 0x0F0F0F0Fu;           // bytes c0 c2 c4 c6
  const uint32_t O = (w >> 4) & 0x0F0F0F0Fu;    // bytes c1 c3 c5 c7
  const uint32_t c0 = E & 0xFFu;
  // c1 + sum c - c0, with c1 - c0 as the sums' accumulator (modulo 2^32)
  const uint32_t x4h =
      __builtin_amdgcn_sad_u8(E, 0u, __builtin_amdgcn_sad_u8(O, 0u, (O & 0xFFu) - c0));
  const uint32_t c0x4 = __builtin_amdgcn_perm(0u, E, 0x00000000u);     // c0 in every byte
  const uint32_t Xa = c0x4 + ((E ^ c0) << 1);                          // E ^ c0: byte 0 cleared
  const uint32_t Xb = c0x4 + (((O & 0xFFFFFF00u) | x4h) << 1);

  // f = X mod 2q; bit 7 of (X + 128 - 2q) is [X >= 2q], and then f is its low seven bits
  const uint32_t tA = Xa + c1;
  const uint32_t mA = tA & 0x80808080u;
  const uint32_t kA = mA - (mA >> 7);                  // 0x7F in the bytes with X >= 2q
  const uint32_t fA = (kA & tA) | (~kA & Xa);
  const uint32_t Xb0 = Xb & 0xFFFFFF00u;               // X4 apart
  const uint32_t tB = Xb0 + c1;
  const uint32_t mB = tB & 0x80808080u;
  const uint32_t kB = mB - (mB >> 7);
  const uint32_t X4 = Xb & 0xFFu;
  const uint32_t d4 = __umul24(X4, m2q) >> 16;         // floor(X4 / 2q), X4 < 2^11
  const uint32_t f4 = X4 - __umul24(d4, den);
  const uint32_t fB = ((kB & tB) | (~kB & Xb0)) | f4;
  const uint32_t pis = bcnt_add(mB, bcnt_add(mA, d4));

  // g = [f > q]; E = g ? 2q - f : f.  gf is 0xFF in the bytes with g: v_perm's selectors 8-11
  // repeat bit 7 of bytes 1 and 3 of either source, so with the sources (t, t << 8) every
  // byte of t has its bit 7 spread over its own byte.  popcount(gf) = 8 #g.
  const uint32_t tgA = fA + c2, tgB = fB + c2;
  const uint32_t gfA = __builtin_amdgcn_perm(tgA, tgA << 8, 0x0B090A08u);
  const uint32_t gfB = __builtin_amdgcn_perm(tgB, tgB << 8, 0x0B090A08u);
  const uint32_t nA = q2 - fA, nB = q2 - fB;
  const uint32_t EA = (gfA & nA) | (~gfA & fA);
  const uint32_t EB = (gfB & nB) | (~gfB & fB);
  // parity masks (all ones when odd): odd2 = sum d mod 2, odd1 = (odd2 + #g) mod 2
  const uint32_t pim = 0u - (pis & 1u);
  const uint32_t o1m = 0u - ((bcnt_add(gfB, bcnt_add(gfA, pis << 3)) >> 3) & 1u);
  // sum E - 4q (the sums' accumulator starts at -4q, modulo 2^32)
  const int sumE4 =
      (int)__builtin_amdgcn_sad_u8(EA, 0u, __builtin_amdgcn_sad_u8(EB, 0u, 0u - 2u * den));

  int p = 0, r = 0, Ep2, Er2;   // 2 E_p, 2 E_r
  if constexpr (M) {
    Ep2 = Er2 = (int)((EA & 0xFFu) << 1);
  } else {
    // 16-bit keys 256 E + 7 - l (max) and 256 E + l (min): E_l is the high byte of a lane,
    // the index tag the low byte, taken from a constant word (tag byte i belongs to byte i)
    const uint32_t s01 = 0x05010400u, s23 = 0x07030602u;   // lanes (byte 0, 1), (byte 2, 3)
    const u16x2 a0 = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(EA, 0x04050607u, s01));
    const u16x2 a1 = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(EA, 0x04050607u, s23));
    const u16x2 a2 = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(EB, 0x00010203u, s01));
    const u16x2 a3 = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(EB, 0x00010203u, s23));
    const u16x2 b0 = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(EA, 0x03020100u, s01));
    const u16x2 b1 = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(EA, 0x03020100u, s23));
    const u16x2 b2 = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(EB, 0x07060504u, s01));
    const u16x2 b3 = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(EB, 0x07060504u, s23));
    const u16x2 mx = __builtin_elementwise_max(__builtin_elementwise_max(a0, a1),
                                               __builtin_elementwise_max(a2, a3));
    const u16x2 mn = __builtin_elementwise_min(__builtin_elementwise_min(b0, b1),
                                               __builtin_elementwise_min(b2, b3));
    const uint32_t kmax = mx.x > mx.y ? (uint32_t)mx.x : (uint32_t)mx.y;
    const uint32_t kmin = mn.x < mn.y ? (uint32_t)mn.x : (uint32_t)mn.y;
    p = 7 - (int)(kmax & 7u);
    Ep2 = (int)(kmax >> 7);   // the tag is below 128
    r = (int)(kmin & 7u);
    Er2 = (int)(kmin >> 7);
  }
  const int gap = sumE4 + (int)(o1m & (den - (uint32_t)Ep2)) - (int)(pim & (uint32_t)Er2);
  const bool d8 = gap < 0;

  // residuals biased by 128: D8 f - 2q g, D8+1/2 f - q, i.e. (f | 128) minus 2q in the bytes
  // with g (D8) or minus q in every byte (D8+1/2), chosen with a mask (a branch would diverge)
  const uint32_t dm = 0u - (uint32_t)d8;               // all ones for D8
  const uint32_t rA = (fA | 0x80808080u) - (d8 ? (gfA & q2) : qb);
  const uint32_t rB = (fB | 0x80808080u) - (d8 ? (gfB & q2) : qb);
  // the fixed coordinate moves by 2q towards the other rounding: +2q where [g] == d8 (a D8
  // coordinate rounded up, a D8+1/2 coordinate below its half-integer), else -2q.  With dl the
  // move's size at its byte of the pair (xa, xb), the fixed pair is (rA, rB) - dl + 2 (dl
  // where [g] == d8); (rA, rB) - dl stays at least 80 in every byte, so nothing borrows.
  const uint32_t idx = (uint32_t)(d8 ? p : r);
  const uint32_t fd = (d8 ? o1m : pim) & den;
  const uint64_t dl = (uint64_t)fd << (8u * idx);
  const uint32_t dlA = (uint32_t)dl, dlB = (uint32_t)(dl >> 32);
  xa = rA - dlA + 2u * (dlA & ~(gfA ^ dm));
  xb = rB - dlB + 2u * (dlB & ~(gfB ^ dm));
}
