// reassemble.h - bit-plane words -> int8 MFMA operand bytes on gfx950.
//
// The packed format stores b bit-planes of a row (APT-LLM, arXiv 2508.19087,
// Sec. IV-A).  The int8 MFMA routes rebuild the b-bit bipolar word of every
// element from its planes before the multiply: because
//     sum_{i,j} 2^(i+j) W_i A_j = (sum_i 2^i W_i)(sum_j 2^j A_j),
// recombining the planes before the product gives the same sum as the
// paper's recovery after the 1-bit products (Sec. III-B), with one int8
// multiply-accumulate per element pair instead of p*q 1-bit ones.
//
// One 32-bit word per plane covers 32 elements; they become 8 output dwords
// (32 bytes).  Output dword t, byte j holds the element at bit 8j + t of the
// word.  The same order is used for every bit width and for both operands, and
// a dot product is unchanged by a permutation of k applied to both sides, so
// the order never shows in the result.
//
// The rebuild is a 3-level merge tree: pairs of planes -> 2-bit fields
// (elements at even / odd bit positions), pairs of those -> nibbles, then
// nibbles -> bytes.  Each merge is a shift plus a bit-field select
// (v_bfi_b32).  With b <= 4 the top level only splits nibbles into bytes.
// Missing planes (i >= b) are zero and fold away at compile time.
#pragma once

#include <stdint.h>

namespace apt {

// (a & mask) | (b & ~mask) as one v_bfi_b32.  Written as an instruction so
// that the compiler keeps one select per merge instead of distributing the
// masks over the tree, which costs about twice the instructions.
__device__ __forceinline__ uint32_t bsel(uint32_t mask, uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(r) : "s"(mask), "v"(a), "v"(b));
  return r;
}

// The tree in two halves, so that a caller can spread one word's work over
// two scheduling slots: reassemble_lo builds the level-1/2 merges (kept in
// mid[]) and output dwords 0..3, reassemble_hi output dwords 4..7 from mid[].
template <int B>
__device__ __forceinline__ void reassemble_lo(const uint32_t* pw, uint32_t mid[8], uint32_t out[4]) {
  if (B == 1) {
    mid[0] = pw[0];
#pragma unroll
    for (int t = 0; t < 4; ++t) out[t] = (pw[0] >> t) & 0x01010101u;
    return;
  }
  auto PL = [&](int i) -> uint32_t { return i < B ? pw[i] : 0u; };
  // level 1: 2-bit fields; e: elements at bits 2f, o: elements at bits 2f+1
  const uint32_t m1 = 0x55555555u;
  uint32_t e01 = bsel(m1, PL(0), PL(1) << 1), o01 = bsel(m1, PL(0) >> 1, PL(1));
  uint32_t e23 = bsel(m1, PL(2), PL(3) << 1), o23 = bsel(m1, PL(2) >> 1, PL(3));
  // level 2: nibbles; ee: elements 4f, eo: 4f+2, oe: 4f+1, oo: 4f+3
  const uint32_t m2 = 0x33333333u;
  mid[0] = bsel(m2, e01, e23 << 2);  // ee
  mid[1] = bsel(m2, o01, o23 << 2);  // oe
  mid[2] = bsel(m2, e01 >> 2, e23);  // eo
  mid[3] = bsel(m2, o01 >> 2, o23);  // oo
  const uint32_t m3 = 0x0F0F0F0Fu;
  if (B <= 4) {
    // level 3: nibble 2j -> byte j (element 8j + s), nibble 2j+1 -> element 8j + 4 + s
#pragma unroll
    for (int t = 0; t < 4; ++t) out[t] = mid[t] & m3;
  } else {
    uint32_t e45 = bsel(m1, PL(4), PL(5) << 1), o45 = bsel(m1, PL(4) >> 1, PL(5));
    uint32_t e67 = bsel(m1, PL(6), PL(7) << 1), o67 = bsel(m1, PL(6) >> 1, PL(7));
    mid[4] = bsel(m2, e45, e67 << 2);
    mid[5] = bsel(m2, o45, o67 << 2);
    mid[6] = bsel(m2, e45 >> 2, e67);
    mid[7] = bsel(m2, o45 >> 2, o67);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      out[t] = bsel(m3, mid[t], mid[4 + t] << 4);
      if (B == 8) out[t] ^= 0x80808080u;
    }
  }
}

template <int B>
__device__ __forceinline__ void reassemble_hi(const uint32_t mid[8], uint32_t out[4]) {
  if (B == 1) {
#pragma unroll
    for (int t = 0; t < 4; ++t) out[t] = (mid[0] >> (4 + t)) & 0x01010101u;
    return;
  }
  const uint32_t m3 = 0x0F0F0F0Fu;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if (B <= 4) {
      out[t] = (mid[t] >> 4) & m3;
    } else {
      out[t] = bsel(m3, mid[t] >> 4, mid[4 + t]);
      if (B == 8) out[t] ^= 0x80808080u;
    }
  }
}

// Bytes of the unsigned b-bit words u (B <= 7), or of u XOR 0x80 = the signed
// code (B == 8), for the 32 elements of plane words pw[0..B-1].
template <int B>
__device__ __forceinline__ void reassemble_word(const uint32_t* pw, uint32_t out[8]) {
  uint32_t mid[8];
  reassemble_lo<B>(pw, mid, out);
  reassemble_hi<B>(mid, out + 4);
}

// FP4 operand nibbles (OCP E2M1: sign bit 3, exponent bits 2..1 with bias
// 1, mantissa bit 0) of the 32 elements of plane words pw[0..B-1], B <= 2.
// Every bipolar value of up to 2 bits is exact in E2M1: +-1 = e 01 m 0,
// +-3 = e 10 m 1.
//   B = 1: v = 2u - 1,  nibble = (~u) << 3 | 0b0010;
//   B = 2: v = 2u - 3 with u = 2h + l: negative when h = 0, |v| = 3 when
//          h == l; nibble = (~h) << 3 | x << 2 | (~x) << 1 | x, x = ~(h ^ l).
// The four nibble bit-planes are merged as the first two levels of the byte
// tree: output dword t, nibble f holds element 4f + t (t = 0..3).
template <int B>
__device__ __forceinline__ void fp4_word(const uint32_t* pw, uint32_t out[4]) {
  static_assert(B == 1 || B == 2, "E2M1 holds bipolar values of up to 2 bits");
  uint32_t n0, n1, n2, n3;  // nibble bit-planes, bit 0 .. bit 3
  if (B == 1) {
    n0 = 0u;
    n1 = ~0u;
    n2 = 0u;
    n3 = ~pw[0];
  } else {
    const uint32_t x = ~(pw[0] ^ pw[1]);
    n0 = x;
    n1 = ~x;
    n2 = x;
    n3 = ~pw[1];
  }
  const uint32_t m1 = 0x55555555u, m2 = 0x33333333u;
  const uint32_t e01 = bsel(m1, n0, n1 << 1), o01 = bsel(m1, n0 >> 1, n1);
  const uint32_t e23 = bsel(m1, n2, n3 << 1), o23 = bsel(m1, n2 >> 1, n3);
  out[0] = bsel(m2, e01, e23 << 2);  // elements 4f
  out[1] = bsel(m2, o01, o23 << 2);  // elements 4f + 1
  out[2] = bsel(m2, e01 >> 2, e23);  // elements 4f + 2
  out[3] = bsel(m2, o01 >> 2, o23);  // elements 4f + 3
}

// FP6 operand fields (OCP E2M3: sign bit 5, exponent bits 4..3 with bias 1,
// mantissa bits 2..0) of the 32 elements of plane words pw[0..B-1], B <= 3.
// Every bipolar value of up to 3 bits is exact in E2M3: +-1 = e 01 m 000,
// +-3 = e 10 m 100, +-5 = e 11 m 010, +-7 = e 11 m 110.  The words u are
// rebuilt as bytes (the int8 tree), mapped to their E2M3 codes with one byte
// permute per dword (the 8-entry table of v = 2u - (2^B - 1)), and the 32
// six-bit codes are packed without gaps into out[0..5] (a 192-bit operand):
// field s (bits 6s .. 6s+5) holds element 8 (s mod 4) + s / 4.  Weights and
// activations use the same order, and a dot product is unchanged by a common
// permutation of k, so the order never shows in the result.
template <int B>
__host__ __device__ constexpr uint32_t e2m3_of_word(uint32_t u) {
  // |v| = 1, 3, 5, 7 -> 8, 20, 26, 30; sign bit 32
  const int v = 2 * (int)u - ((1 << B) - 1);
  const int a = v < 0 ? -v : v;
  const uint32_t mag = a == 1 ? 8u : a == 3 ? 20u : a == 5 ? 26u : 30u;
  return v < 0 ? mag | 32u : mag;
}

template <int B>
__host__ __device__ constexpr uint32_t e2m3_table(int half) {
  // bytes 4 half .. 4 half + 3 of the table indexed by u (entries past 2^B unused)
  uint32_t t = 0u;
  for (int j = 0; j < 4; ++j) {
    const int u = 4 * half + j;
    t |= (u < (1 << B) ? e2m3_of_word<B>((uint32_t)u) : 0u) << (8 * j);
  }
  return t;
}

template <int B>
__device__ __forceinline__ void fp6_word(const uint32_t* pw, uint32_t out[6]) {
  static_assert(B >= 1 && B <= 3, "E2M3 holds bipolar values of up to 3 bits");
  uint32_t by[8];
  reassemble_word<B>(pw, by);  // byte j of by[t]: u of element 8 j + t
  constexpr uint32_t lo = e2m3_table<B>(0), hi = e2m3_table<B>(1);
  uint32_t y[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    const uint32_t c = __builtin_amdgcn_perm(hi, lo, by[t]);  // byte j <- table[u_j]
    // four 6-bit codes (one per byte) -> 24 contiguous bits
    const uint32_t c01 = bsel(0x3Fu, c, c >> 2);      // bits 0..11: codes 0, 1
    const uint32_t c012 = bsel(0xFFFu, c01, c >> 4);  // bits 0..17: codes 0..2
    y[t] = bsel(0x3FFFFu, c012, c >> 6);               // bits 0..23: codes 0..3
  }
  out[0] = y[0] | (y[1] << 24);
  out[1] = (y[1] >> 8) | (y[2] << 16);
  out[2] = (y[2] >> 16) | (y[3] << 8);
  out[3] = y[4] | (y[5] << 24);
  out[4] = (y[5] >> 8) | (y[6] << 16);
  out[5] = (y[6] >> 16) | (y[7] << 8);
}

// FP8 operand bytes (OCP E4M3: sign bit 7, exponent bits 6..3 with bias 7,
// mantissa bits 2..0) of the 32 elements of plane words pw[0..B-1], B <= 4.
// Every bipolar value of up to 4 bits (odd, |v| <= 15) is exact in E4M3.  The
// words u are rebuilt as bytes (the int8 tree, same element order) and each
// byte becomes the E4M3 code of v = 2u - (2^B - 1) through a byte permute over
// the 8-entry table of u mod 8, plus, for B = 4, a second table for u >= 8
// chosen by bit 3 of the byte.
template <int B>
__host__ __device__ constexpr uint32_t e4m3_of_word(uint32_t u) {
  const int v = 2 * (int)u - ((1 << B) - 1);
  const int a = v < 0 ? -v : v;
  // |v| = 1, 3, ..., 15: exponent field 7 + floor(log2 |v|), 3 mantissa bits
  const int e = a >= 8 ? 3 : a >= 4 ? 2 : a >= 2 ? 1 : 0;
  const uint32_t bits = (uint32_t)(((e + 7) << 3) | (((a << 3) >> e) & 7));
  return v < 0 ? bits | 0x80u : bits;
}

template <int B>
__host__ __device__ constexpr uint32_t e4m3_table(int quarter) {
  // bytes 4 quarter .. 4 quarter + 3 of the table indexed by u (entries past 2^B unused)
  uint32_t t = 0u;
  for (int j = 0; j < 4; ++j) {
    const int u = 4 * quarter + j;
    t |= (u < (1 << B) ? e4m3_of_word<B>((uint32_t)u) : 0u) << (8 * j);
  }
  return t;
}

template <int B>
__device__ __forceinline__ uint32_t e4m3_dword(uint32_t by) {
  static_assert(B >= 1 && B <= 4, "E4M3 holds bipolar values of up to 4 bits");
  if (B <= 3) return __builtin_amdgcn_perm(e4m3_table<B>(1), e4m3_table<B>(0), by);
  const uint32_t lo = by & 0x07070707u;
  const uint32_t c0 = __builtin_amdgcn_perm(e4m3_table<B>(1), e4m3_table<B>(0), lo);
  const uint32_t c1 = __builtin_amdgcn_perm(e4m3_table<B>(3), e4m3_table<B>(2), lo);
  const uint32_t hi = ((by >> 3) & 0x01010101u) * 0xFFu;  // 0xFF in the bytes with u >= 8
  return (c1 & hi) | (c0 & ~hi);  // (a per-lane mask: one v_bfi_b32)
}

template <int B>
__device__ __forceinline__ void fp8_word(const uint32_t* pw, uint32_t out[8]) {
  reassemble_word<B>(pw, out);  // byte j of out[t]: u of element 8 j + t
#pragma unroll
  for (int t = 0; t < 8; ++t) out[t] = e4m3_dword<B>(out[t]);
}

// Operand offset of the reassembled byte y: bipolar value v = 2 y + c.
//   B <= 7: y = u,        v = 2u - (2^B - 1)  ->  c = 1 - 2^B
//   B == 8: y = u - 128,  v = 2u - 255        ->  c = 1
template <int B>
__host__ __device__ constexpr int operand_offset() { return B == 8 ? 1 : 1 - (1 << B); }

// Operand byte of a padding element (all plane bits zero).
template <int B>
__host__ __device__ constexpr int operand_pad() { return B == 8 ? -128 : 0; }

}  // namespace apt
