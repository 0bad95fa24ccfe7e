// rowcode.h - one lane's share of a row of activation codes or fp16
// activations, turned into bipolar words and bit-planes on gfx950 (APT-LLM,
// arXiv 2508.19087: Sec. III-A conversion and the bipolar form of a linear
// quantizer; Sec. IV-A decomposition into bit-planes).  Shared by the packer
// (pack.hip), which stores the plane words in the packed layout, and by the
// XOR route's fused decode form (gemm_xor.h), which stores them in LDS.
//
// A lane takes 16 consecutive elements of a row.  CodeRow reads signed b-bit
// codes (one byte each) and HalfRow fp16 values, which it quantizes with the
// row's bipolar scale (see row_scale).  words() gives the 16 bipolar words u,
// one per byte; transpose8x8 leaves plane i of 8 elements in byte i; and
// plane_word gives, for a pair of planes, the 32-bit plane word that this lane
// and its neighbour (lanes 2m, 2m + 1, 32 consecutive elements) hold between
// them: the even lane gets plane i, the odd lane plane i + 1.
#pragma once

#include "apt_internal.h"

namespace apt {
namespace rowcode {

constexpr int kLaneElems = 16;
constexpr uint32_t kRawBufferFlags = 0x00020000u;

typedef unsigned short ushort2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Signed b-bit codes, one byte each.
template <bool kVec, int B>
struct CodeRow {
  static constexpr int kDwords = kLaneElems / 4;
  static constexpr int kElemBytes = 1;
  static constexpr bool kVector = kVec;
  static constexpr bool kScaled = false;

  // The lane's 16 codes from element k0 on.
  __device__ static void load(__amdgpu_buffer_rsrc_t rsrc, int k0, uint32_t d[kDwords]) {
    if (kVector) {
      // K % 16 == 0: the lane's 16 codes are all in the row or all past it.
      const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(rsrc, (uint32_t)k0, 0, 0);
#pragma unroll
      for (int t = 0; t < 4; ++t) d[t] = v[t];
    } else {
#pragma unroll
      for (int t = 0; t < kDwords; ++t) {
        uint32_t w = 0u;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          w |= (uint32_t)__builtin_amdgcn_raw_buffer_load_b8(rsrc, (uint32_t)(k0 + 4 * t + q), 0, 0)
               << (8 * q);
        d[t] = w;
      }
    }
  }
  // Bipolar words u = (x mod 2^b) XOR 2^(b-1), one per byte (Sec. III-A).
  __device__ static void words(const uint32_t d[kDwords], float, float, uint32_t u[4]) {
    constexpr uint32_t field = ((1u << B) - 1u) * 0x01010101u;
    constexpr uint32_t flip = (1u << (B - 1)) * 0x01010101u;
#pragma unroll
    for (int t = 0; t < 4; ++t) u[t] = (d[t] & field) ^ flip;
  }
};

// fp16 activations, quantized with the row's scale.
template <bool kVec, int B>
struct HalfRow {
  static constexpr int kDwords = kLaneElems / 2;
  static constexpr int kElemBytes = 2;
  static constexpr bool kVector = kVec;
  static constexpr bool kScaled = true;

  // The lane's 16 values from element k0 on (fp16 bits, two per dword).
  __device__ static void load(__amdgpu_buffer_rsrc_t rsrc, int k0, uint32_t d[kDwords]) {
    const uint32_t off = (uint32_t)k0 * 2u;
    if (kVector) {
      const u32x4_t v0 = __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, 0);
      const u32x4_t v1 = __builtin_amdgcn_raw_buffer_load_b128(rsrc, off + 16u, 0, 0);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        d[t] = v0[t];
        d[4 + t] = v1[t];
      }
    } else {
#pragma unroll
      for (int t = 0; t < kDwords; ++t) {
        const uint32_t h0 = __builtin_amdgcn_raw_buffer_load_b16(rsrc, off + 4u * t, 0, 0);
        const uint32_t h1 = __builtin_amdgcn_raw_buffer_load_b16(rsrc, off + 4u * t + 2u, 0, 0);
        d[t] = (h0 & 0xFFFFu) | (h1 << 16);
      }
    }
  }
  // Largest |x| of the lane's values as fp16 bits, one maximum per 16-bit
  // half: for finite values the order of |x| is the integer order of the bits
  // without the sign.
  __device__ static ushort2_t fold_max(ushort2_t m, const uint32_t d[kDwords]) {
#pragma unroll
    for (int t = 0; t < kDwords; ++t)
      m = __builtin_elementwise_max(m, __builtin_bit_cast(ushort2_t, d[t] & 0x7FFF7FFFu));
    return m;
  }
  // Bipolar words of the lane's 16 values, one per byte (element 4t + q in
  // byte q of u[t]).  The signed code c = floor(h) clamped to the b-bit range
  // goes into a byte as two's complement; the word is then
  // (c mod 2^b) XOR 2^(b-1) = c + 2^(b-1), four bytes at once.  A zero's sign
  // in h0 does not change floor(h).
  __device__ static void words(const uint32_t d[kDwords], float rh, float s2, uint32_t u[4]) {
#pragma clang fp contract(off)
    constexpr int clo = -(1 << (B - 1)), chi = (1 << (B - 1)) - 1;
    constexpr uint32_t field = ((1u << B) - 1u) * 0x01010101u;
    constexpr uint32_t flip = (1u << (B - 1)) * 0x01010101u;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      uint32_t acc = 0u;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int j = 4 * t + q;
        const uint32_t bits = (d[j / 2] >> (16 * (j % 2))) & 0xFFFFu;
        const float x = __half2float(__ushort_as_half((unsigned short)bits));
        const float h0 = __builtin_fmaf(x, rh, 0.0f);
        const float e = __builtin_fmaf(-h0, s2, x);
        const float h = __builtin_fmaf(e, rh, h0);  // RN(x / s) / 2
        int c;  // floor(h) as int32 in one instruction (saturating)
        asm("v_cvt_flr_i32_f32 %0, %1" : "=v"(c) : "v"(h));
        c = min(max(c, clo), chi);
        // byte q of acc <- low byte of c; the other bytes stay
        const uint32_t sel = q == 1 ? 0x03020400u : q == 2 ? 0x03040100u : 0x04020100u;
        acc = q == 0 ? (uint32_t)c : __builtin_amdgcn_perm((uint32_t)c, acc, sel);
      }
      u[t] = (acc & field) ^ flip;
    }
  }
};

// Delta swaps of an 8x8 bit-matrix transpose (bit 8r + c <-> bit 8c + r of a
// 64-bit value, rows r = bytes): distance 7 and 14 stay inside each dword,
// distance 28 moves nibbles between the dwords.  The three commute.
__device__ __forceinline__ uint32_t swap7(uint32_t x) {
  const uint32_t t = (x ^ (x >> 7)) & 0x00AA00AAu;
  return x ^ t ^ (t << 7);
}
__device__ __forceinline__ uint32_t swap14(uint32_t x) {
  const uint32_t t = (x ^ (x >> 14)) & 0x0000CCCCu;
  return x ^ t ^ (t << 14);
}

// Transposes the bytes lo (rows 0..3) and hi (rows 4..7): afterwards bit j of
// byte i is bit i of the former byte j.  With b <= 4 every byte is below 16:
// the distance-28 swap just moves hi's low nibbles up into lo (hi becomes 0).
template <int B>
__device__ __forceinline__ void transpose8x8(uint32_t& lo, uint32_t& hi) {
  if (B <= 4) {
    lo = swap14(swap7(lo | (hi << 4)));
    hi = 0u;
  } else {
    lo = swap14(swap7(lo));
    hi = swap14(swap7(hi));
    const uint32_t t = (lo ^ (hi << 4)) & 0xF0F0F0F0u;
    lo ^= t;
    hi ^= t >> 4;
  }
}

// The rows' bipolar scale and the two constants of the exact half quotient
// (HalfRow::words) from the largest magnitude's fp16 bits:
// s = fp16(absmax / (2^B - 1)) with an IEEE fp32 divide, rh = RN(1 / s) / 2
// (0 when s = 0, so that every quotient is 0), s2 = 2 s.  Returns the fp16 bits
// of s.
template <int B>
__device__ __forceinline__ uint16_t row_scale(uint32_t absmax_bits, float& rh, float& s2) {
  const float absmax = __half2float(__ushort_as_half((unsigned short)absmax_bits));
  const __half s16 = __float2half_rn(__fdiv_rn(absmax, (float)((1 << B) - 1)));
  const float s = __half2float(s16);
  rh = s > 0.0f ? __fdiv_rn(1.0f, s) * 0.5f : 0.0f;
  s2 = s * 2.0f;
  return __half_as_ushort(s16);
}

// This lane's word of plane pair (i, i + 1) after transpose8x8 of its two
// 8-element groups (lo/hi of elements 0..7 in sa, of 8..15 in sb): the even
// lane of a pair gets the 32 bits of plane i, the odd lane those of plane i + 1
// (one DPP swap between neighbours).
__device__ __forceinline__ uint32_t plane_word(uint32_t sa, uint32_t sb, int bi, bool odd) {
  // y = [a_i, b_i, a_i+1, b_i+1]: this lane's 16 bits of plane i, then of plane i+1
  const uint32_t y = __builtin_amdgcn_perm(
      sb, sa, (uint32_t)(bi | (4 + bi) << 8 | (bi + 1) << 16 | (5 + bi) << 24));
  const uint32_t z = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)y, 0xB1, 0xF, 0xF, false);  // lane ^ 1
  return __builtin_amdgcn_perm(z, y, odd ? 0x03020706u : 0x05040100u);
}

}  // namespace rowcode
}  // namespace apt
