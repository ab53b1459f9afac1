// Alg. 2 (Voronoi decode, with the Gosset oracle of Alg. 5 or NestQuantM's of App. D) on one
// code word, four coordinates per 32-bit register (byte SIMD), for every q <= 16.  Included
// by nq_device.hpp inside namespace nq (it needs u16x2 and the amdgcn byte builtins).
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
//     fix to argmin E, lowest index on ties: keys 8 E + 7 - l (max) and 8 E + l (min) fit a
//     byte (E <= q <= 16) and are reduced in 16-bit lanes;
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
  // per-byte constants (q is uniform, so the compiler keeps them out of the block loops)
  const uint32_t q2 = __builtin_amdgcn_perm(0u, den, 0x00000000u);            // 2q
  const uint32_t c1 = __builtin_amdgcn_perm(0u, 128u - den, 0x00000000u);     // 128 - 2q
  const uint32_t c2 = __builtin_amdgcn_perm(0u, 127u - (uint32_t)q, 0x00000000u);  // 127 - q
  const uint32_t c3 = __builtin_amdgcn_perm(0u, 128u - (uint32_t)q, 0x00000000u);  // 128 - q

  // X = G c: (X0..X3) = c0 + 2 (0, c2, c4, c6); (X4..X7) = c0 + 2 (c1 + sum c - c0, c3, c5, c7)
  const uint32_t E = w & 0x0F0F0F0Fu;           // bytes c0 c2 c4 c6
  const uint32_t O = (w >> 4) & 0x0F0F0F0Fu;    // bytes c1 c3 c5 c7
  const uint32_t c0 = E & 0xFFu;
  const uint32_t sum_c = __builtin_amdgcn_sad_u8(E, 0u, __builtin_amdgcn_sad_u8(O, 0u, 0u));
  const uint32_t c0x4 = __builtin_amdgcn_perm(0u, E, 0x00000000u);     // c0 in every byte
  const uint32_t Xa = c0x4 + ((E & 0xFFFFFF00u) << 1);
  const uint32_t Xb = c0x4 + (((O & 0xFFFFFF00u) | ((O & 0xFFu) + sum_c - c0)) << 1);

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
  const uint32_t pis = (uint32_t)__builtin_popcount(mA) + (uint32_t)__builtin_popcount(mB) + d4;

  // g = [f > q]; E = g ? 2q - f : f
  const uint32_t gA = (fA + c2) & 0x80808080u, gB = (fB + c2) & 0x80808080u;
  const uint32_t gkA = gA - (gA >> 7), gkB = gB - (gB >> 7);
  const uint32_t nA = q2 - fA, nB = q2 - fB;
  const uint32_t EA = (gkA & nA) | (~gkA & fA);
  const uint32_t EB = (gkB & nB) | (~gkB & fB);
  const uint32_t pi = pis & 1u;
  const uint32_t odd1 =
      (pis + (uint32_t)__builtin_popcount(gA) + (uint32_t)__builtin_popcount(gB)) & 1u;
  const int sumE = (int)__builtin_amdgcn_sad_u8(EA, 0u, __builtin_amdgcn_sad_u8(EB, 0u, 0u));

  int p = 0, r = 0, Ep, Er;
  if constexpr (M) {
    Ep = Er = (int)(EA & 0xFFu);
  } else {
    // byte l of a word: coordinate l (A) or 4 + l (B)
    const uint32_t xA = (EA << 3) | 0x04050607u, xB = (EB << 3) | 0x00010203u;  // 8E + 7 - l
    const uint32_t nA8 = (EA << 3) | 0x03020100u, nB8 = (EB << 3) | 0x07060504u;  // 8E + l
    // 16-bit lanes (byte i of A, byte i of B) for i = 0..3
    const u16x2 a0 = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(xB, xA, 0x0C040C00u));
    const u16x2 a1 = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(xB, xA, 0x0C050C01u));
    const u16x2 a2 = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(xB, xA, 0x0C060C02u));
    const u16x2 a3 = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(xB, xA, 0x0C070C03u));
    const u16x2 b0 = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(nB8, nA8, 0x0C040C00u));
    const u16x2 b1 = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(nB8, nA8, 0x0C050C01u));
    const u16x2 b2 = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(nB8, nA8, 0x0C060C02u));
    const u16x2 b3 = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(nB8, nA8, 0x0C070C03u));
    const u16x2 mx = __builtin_elementwise_max(__builtin_elementwise_max(a0, a1),
                                               __builtin_elementwise_max(a2, a3));
    const u16x2 mn = __builtin_elementwise_min(__builtin_elementwise_min(b0, b1),
                                               __builtin_elementwise_min(b2, b3));
    const uint32_t kmax = mx.x > mx.y ? (uint32_t)mx.x : (uint32_t)mx.y;
    const uint32_t kmin = mn.x < mn.y ? (uint32_t)mn.x : (uint32_t)mn.y;
    p = 7 - (int)(kmax & 7u);
    Ep = (int)(kmax >> 3);
    r = (int)(kmin & 7u);
    Er = (int)(kmin >> 3);
  }
  const int gap = sumE - 2 * (int)den + (odd1 ? (int)den - 2 * Ep : 0) - (pi ? 2 * Er : 0);
  const bool d8 = gap < 0;

  // residuals biased by 128: D8 f - 2q g (g ? 128 - (2q - f) : 128 + f); D8+1/2 f - q + 128;
  // chosen with a mask (both are cheap, and a branch would diverge)
  const uint32_t dm = 0u - (uint32_t)d8;               // all ones for D8
  const uint32_t gfA = gkA + gA, gfB = gkB + gB;       // 0xFF in the bytes with g
  const uint32_t dA = (gfA & (0x80808080u - nA)) | (~gfA & (fA | 0x80808080u));
  const uint32_t dB = (gfB & (0x80808080u - nB)) | (~gfB & (fB | 0x80808080u));
  const uint32_t rA = (dm & dA) | (~dm & (fA + c3));
  const uint32_t rB = (dm & dB) | (~dm & (fB + c3));
  // the fixed coordinate moves by +2q s (D8) or -2q s (D8+1/2), s = 2 g - 1
  const int idx = d8 ? p : r;
  const uint32_t fix = d8 ? odd1 : pi;
  const int sh = 8 * (idx & 3);
  const uint32_t gw = idx < 4 ? gA : gB;
  const uint32_t gi = (gw >> (sh + 7)) & 1u;
  const uint32_t dl = (0u - fix) & (den << sh);
  const uint32_t sdl = (gi ^ (uint32_t)d8) ? 0u - dl : dl;   // +dl when g_idx == d8
  const uint32_t lo = idx < 4 ? 0xFFFFFFFFu : 0u;
  xa = rA + (lo & sdl);
  xb = rB + (~lo & sdl);
}
