// The byte-SIMD Voronoi decoder (decode_word_b8, nq_b8.hpp) compiled for the host: every
// AMDGCN instruction it uses is replaced by a plain C++ function written from that
// instruction's definition in the CDNA3 ISA reference (v_perm_b32 byte select, v_sad_u8,
// v_bcnt_u32_b32, v_mul_u32_u24), so that its byte arithmetic can be checked against the
// oracle over every code word of small q.  Test infrastructure; built by
// tests/test_decoder_host.py with clang++ (ext_vector_type and __builtin_elementwise_*).
#include <cstdint>

#define __device__
#define __forceinline__ inline __attribute__((always_inline))
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// v_perm_b32: byte i of the result is selected by byte i of sel from the eight bytes of
// {s0, s1} (s1 the low word): 0-7 a byte, 8-11 bit 7 of byte 1, 3, 5, 7 repeated, 12 zero,
// 13 and above 0xFF.
static inline uint32_t host_perm(uint32_t s0, uint32_t s1, uint32_t sel) {
  const uint64_t v = ((uint64_t)s0 << 32) | s1;
  uint32_t d = 0;
  for (int i = 0; i < 4; ++i) {
    const uint32_t s = (sel >> (8 * i)) & 0xFFu;
    uint32_t b;
    if (s < 8) b = (uint32_t)(v >> (8 * s)) & 0xFFu;
    else if (s < 12) b = ((v >> (8 * (2 * (s - 8) + 1) + 7)) & 1u) ? 0xFFu : 0u;
    else if (s == 12) b = 0u;
    else b = 0xFFu;
    d |= b << (8 * i);
  }
  return d;
}
// v_sad_u8: sum over the four bytes of |a_i - b_i|, plus c
static inline uint32_t host_sad_u8(uint32_t a, uint32_t b, uint32_t c) {
  uint32_t s = c;
  for (int i = 0; i < 4; ++i) {
    const int x = (int)((a >> (8 * i)) & 0xFFu), y = (int)((b >> (8 * i)) & 0xFFu);
    s += (uint32_t)(x > y ? x - y : y - x);
  }
  return s;
}
// v_mul_u32_u24: low 32 bits of the product of the operands' low 24 bits
static inline uint32_t host_mul24(uint32_t a, uint32_t b) {
  return (uint32_t)((uint64_t)(a & 0xFFFFFFu) * (b & 0xFFFFFFu));
}
#define __builtin_amdgcn_perm host_perm
#define __builtin_amdgcn_sad_u8 host_sad_u8
#define __umul24 host_mul24

namespace nq {
// v_bcnt_u32_b32: popcount(x) + acc
static inline uint32_t bcnt_add(uint32_t x, uint32_t acc) {
  return acc + (uint32_t)__builtin_popcount(x);
}
#include "nq_b8.hpp"
}  // namespace nq

// n code words -> 8 n values X2 (the decoded point in 2E8 units), M = NestQuantM decoder
extern "C" void nq_b8_host_decode(const uint32_t* words, int64_t n, int q, int M,
                                  int32_t* out) {
  const uint32_t m2q = (65536u + 2u * (uint32_t)q - 1u) / (2u * (uint32_t)q);   // magic_2q
  for (int64_t i = 0; i < n; ++i) {
    uint32_t xa, xb;
    if (M) nq::decode_word_b8<true>(words[i], q, m2q, xa, xb);
    else nq::decode_word_b8<false>(words[i], q, m2q, xa, xb);
    for (int l = 0; l < 4; ++l) {
      out[8 * i + l] = (int32_t)((xa >> (8 * l)) & 0xFFu) - 128;
      out[8 * i + 4 + l] = (int32_t)((xb >> (8 * l)) & 0xFFu) - 128;
    }
  }
}
