// quantize.hip - fp16 activations -> per-row (token) b-bit bipolar-INT codes
// -> bit-planes, in one kernel for gfx950 (APT-LLM, arXiv 2508.19087: the
// bipolar form of a linear quantizer, Sec. III-A; the packed layout,
// Sec. IV-A steps 1-3).
//
// Quantizer of row m (the rounding is this library's choice; the paper fixes
// none): s = fp16(absmax_k |x[m][k]| / (2^b - 1)) with an IEEE fp32 divide,
// so the largest magnitude lands on the outermost odd level; element x goes
// to the odd level 2 floor(t / 2) + 1 of t = x / s clamped to +-(2^b - 1),
// i.e. to the signed code floor(t / 2) clamped to [-2^(b-1), 2^(b-1) - 1],
// whose bipolar word is code + 2^(b-1).  A row with s = 0 gets t = 0.
//
// One workgroup per row, the padding rows of the last 8-row group included
// (they write zero words).  The row is split over the workgroup's nw waves in
// steps of 1024 elements: wave w takes steps w, w + nw, ...; lane l of a step
// takes elements [16 l, 16 l + 16) (two 16-byte buffer loads; the buffer's
// size is the row's, so reads past K return 0 and a padding row reads only
// zeros).  When every wave has at most 4 steps (K <= 32768) the loaded values
// stay in registers and the row is read once: pass 1 folds the largest
// magnitude, reduced over the workgroup through LDS, pass 2 quantizes and
// packs from registers.  Longer rows load their steps again in pass 2.
//
// Packing: the 16 bipolar words of a lane (one byte each) go through an 8x8
// bit-matrix transpose per 8 elements, which leaves plane i of those elements
// in byte i; for b <= 4 the high nibbles are zero and the transpose reduces to
// two delta swaps on one dword.  Lanes 2m and 2m+1 hold the two 16-bit halves
// of one plane word; per pair of planes they swap halves with a DPP move.
//
// Workgroups are dispatched to the 8 XCDs round robin; rows are assigned so
// that consecutive workgroups on one XCD take consecutive rows, and the 8 rows
// of a packed row group, which share every 128-byte plane segment (16 bytes
// each), meet in that XCD's L2.
//
// Division: instead of a correctly rounded fp32 divide per element, each row
// computes r = RN(1 / s) once and each element
//     h0 = RN(x r / 2),  e = fma(-h0, 2 s, x),  h = fma(e, r / 2, h0),
// the quotient correction of Markstein's division with a correctly rounded
// reciprocal, applied to the half quotient.  h equals RN(x / s) / 2 for every
// finite fp16 x and positive finite fp16 s; the test suite checks all of
// those pairs on the CPU.
#include <algorithm>

#include "apt_internal.h"

namespace apt {
namespace {

constexpr int kWave = 64;
constexpr int kMaxWaves = 8;
constexpr int kLaneElems = 16;
constexpr int kStep = kWave * kLaneElems;  // 1024 elements = 8 chunks
constexpr int kMaxCachedSteps = 4;
constexpr int kTargetWaves = 4096;  // 16 per CU
constexpr int kXcds = 8;
constexpr int kDwords = kLaneElems / 2;  // fp16 pairs per lane and step

typedef unsigned short ushort2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// The lane's 16 values from element k0 on (fp16 bits, two per dword).
template <bool kVector>
__device__ __forceinline__ void load_lane(__amdgpu_buffer_rsrc_t rsrc, int k0,
                                          uint32_t d[kDwords]) {
  const uint32_t off = (uint32_t)k0 * 2u;
  if (kVector) {
    // K % 16 == 0: the lane's 16 values are all in the row or all past it.
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

// Largest |x| of the lane's values as fp16 bits, one maximum per 16-bit half:
// for finite values the order of |x| is the integer order of the bits without
// the sign.
__device__ __forceinline__ ushort2_t fold_max(ushort2_t m, const uint32_t d[kDwords]) {
#pragma unroll
  for (int t = 0; t < kDwords; ++t)
    m = __builtin_elementwise_max(m, __builtin_bit_cast(ushort2_t, d[t] & 0x7FFF7FFFu));
  return m;
}

// Bipolar words of the lane's 16 values, one per byte (element 4t + q in byte
// q of u[t]).  The signed code c = floor(h) clamped to [-2^(b-1), 2^(b-1) - 1]
// goes into a byte as two's complement; the word is then
// (c mod 2^b) XOR 2^(b-1) = c + 2^(b-1), applied to four bytes at once.
// h0 = fma(x, r/2, +0) differs from RN(x r/2) at most in the sign of a zero,
// which floor(h) does not see.
template <int B>
__device__ __forceinline__ void quantize_lane(const uint32_t d[kDwords], float rh, float s2,
                                              uint32_t u[4]) {
#pragma clang fp contract(off)
  constexpr int clo = -(1 << (B - 1)), chi = (1 << (B - 1)) - 1;
  constexpr uint32_t field = ((1u << B) - 1u) * 0x01010101u, flip = (1u << (B - 1)) * 0x01010101u;
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

// kSteps: steps each wave keeps in registers (1, 2 or 4), or 0 for rows too
// long for that, which are loaded twice.
template <bool kVector, int B, int kSteps>
__global__ __launch_bounds__(kWave* kMaxWaves) void quantize_pack_kernel(
    const uint16_t* __restrict__ x, int rows, int K, int nchunks, int groups,
    uint32_t* __restrict__ packed, int32_t* __restrict__ rowsum, uint16_t* __restrict__ scale) {
  constexpr int kHeld = kSteps > 0 ? kSteps : kMaxCachedSteps;
  __shared__ uint32_t lds_red[kMaxWaves];
  const int nw = blockDim.x / kWave;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x % kWave;
  const int row = (blockIdx.x % kXcds) * groups + blockIdx.x / kXcds;  // < padded row count
  const bool real = row < rows;
  const int kpad = nchunks * kChunk;
  const int nsteps = (kpad + kStep - 1) / kStep;
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(real ? x + (int64_t)row * K : x), 0,
                                        real ? 2 * K : 0, 0x00020000);

  // Pass 1: the row's largest magnitude.
  uint32_t d[kHeld][kDwords];
  ushort2_t mm = {0, 0};
  for (int j0 = wave; j0 < nsteps; j0 += kHeld * nw) {
#pragma unroll
    for (int t = 0; t < kHeld; ++t) load_lane<kVector>(rsrc, (j0 + t * nw) * kStep + lane * kLaneElems, d[t]);
#pragma unroll
    for (int t = 0; t < kHeld; ++t) mm = fold_max(mm, d[t]);
    if (kSteps > 0) break;  // one trip covers all steps
  }
  uint32_t m = max((uint32_t)mm.x, (uint32_t)mm.y);
  for (int off = kWave / 2; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
  if (lane == 0) lds_red[wave] = m;
  __syncthreads();
  m = 0u;
  for (int w = 0; w < nw; ++w) m = max(m, lds_red[w]);
  __syncthreads();  // lds_red is reused for the row sum

  const float absmax = __half2float(__ushort_as_half((unsigned short)m));
  const __half s16 = __float2half_rn(__fdiv_rn(absmax, (float)((1 << B) - 1)));
  const float s = __half2float(s16);
  const float rh = s > 0.0f ? __fdiv_rn(1.0f, s) * 0.5f : 0.0f;  // s = 0: every h is 0
  const float s2 = s * 2.0f;
  if (real && threadIdx.x == 0) scale[row] = __half_as_ushort(s16);

  // Pass 2: quantize, convert and pack.
  uint32_t usum = 0u;
  const bool odd = (lane & 1) != 0;
  const uint32_t join = odd ? 0x03020706u : 0x05040100u;
  auto process = [&](int j, const uint32_t* dd) __attribute__((always_inline)) {
    const int k0 = j * kStep + lane * kLaneElems;
    uint32_t u[4];
    quantize_lane<B>(dd, rh, s2, u);
    // padding elements and rows: all-zero words
    if (kVector) {
      const uint32_t valid = (real && k0 < K) ? 0xFFFFFFFFu : 0u;
#pragma unroll
      for (int t = 0; t < 4; ++t) u[t] &= valid;
    } else {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int n_valid = real ? K - (k0 + 4 * t) : 0;
        u[t] &= n_valid >= 4 ? 0xFFFFFFFFu : (n_valid <= 0 ? 0u : ((1u << (8 * n_valid)) - 1u));
      }
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) usum = __builtin_amdgcn_sad_u8(u[t], 0u, usum);
    // Planes of elements 0..7 (a) and 8..15 (b): byte i = plane i (i < 4 in lo).
    uint32_t alo = u[0], ahi = u[1], blo = u[2], bhi = u[3];
    transpose8x8<B>(alo, ahi);
    transpose8x8<B>(blo, bhi);
    if (k0 >= kpad) return;
    uint32_t* dst = packed + plane_words(row, k0 / kChunk, 0, nchunks, B) + (k0 % kChunk) / 32;
#pragma unroll
    for (int i = 0; i < B; i += 2) {
      const uint32_t sa = i < 4 ? alo : ahi, sb = i < 4 ? blo : bhi;
      const int bi = i % 4;
      // y = [a_i, b_i, a_i+1, b_i+1]: this lane's 16 bits of plane i, then of plane i+1
      const uint32_t y =
          __builtin_amdgcn_perm(sb, sa, (uint32_t)(bi | (4 + bi) << 8 | (bi + 1) << 16 | (5 + bi) << 24));
      const uint32_t z = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)y, 0xB1, 0xF, 0xF, false);  // lane ^ 1
      const uint32_t wv = __builtin_amdgcn_perm(z, y, join);  // even: plane i, odd: plane i+1
      if (!odd || i + 1 < B) dst[(i + (odd ? 1 : 0)) * kPlaneStride] = wv;
    }
  };
  if (kSteps > 0) {
#pragma unroll
    for (int t = 0; t < kHeld; ++t) {
      const int j = wave + t * nw;
      if (j < nsteps) process(j, d[t]);
    }
  } else {
    for (int j0 = wave; j0 < nsteps; j0 += kHeld * nw) {
#pragma unroll
      for (int t = 0; t < kHeld; ++t) load_lane<kVector>(rsrc, (j0 + t * nw) * kStep + lane * kLaneElems, d[t]);
#pragma unroll
      for (int t = 0; t < kHeld; ++t)
        if (j0 + t * nw < nsteps) process(j0 + t * nw, d[t]);
    }
  }

  if (rowsum != nullptr) {
    for (int off = kWave / 2; off > 0; off >>= 1) usum += __shfl_xor(usum, off);
    if (lane == 0) lds_red[wave] = usum;
    __syncthreads();
    if (real && threadIdx.x == 0) {
      uint32_t total = 0u;
      for (int w = 0; w < nw; ++w) total += lds_red[w];
      // sum_k (2 u - (2^b - 1)) over the K real elements
      rowsum[row] = (int32_t)(2u * total - ((1u << B) - 1u) * (uint32_t)K);
    }
  }
}

template <bool kVector, int B, int kSteps>
void launch_kernel(dim3 grid, dim3 block, hipStream_t stream, const uint16_t* x, int rows, int K,
                   int nchunks, int groups, uint32_t* packed, int32_t* rowsum, uint16_t* scale) {
  hipLaunchKernelGGL((quantize_pack_kernel<kVector, B, kSteps>), grid, block, 0, stream, x, rows,
                     K, nchunks, groups, packed, rowsum, scale);
}

template <bool kVector, int B>
hipError_t launch_vec_bits(const uint16_t* x, int rows, int K, uint32_t* packed, int32_t* rowsum,
                           uint16_t* scale, hipStream_t stream) {
  const int nchunks = num_chunks(K);
  const int nsteps = (nchunks * kChunk + kStep - 1) / kStep;
  // Fewest waves per row that hold the row in registers (the per-row
  // reductions and scale cost the same for every wave), but more while the
  // whole grid has fewer than kTargetWaves waves.
  const int max_nw = nsteps < kMaxWaves ? nsteps : kMaxWaves;
  int nw = std::min((nsteps + kMaxCachedSteps - 1) / kMaxCachedSteps, max_nw);
  while (nw < max_nw && (int64_t)padded_rows(rows) * nw < kTargetWaves) nw = std::min(2 * nw, max_nw);
  const int per_wave = (nsteps + nw - 1) / nw;
  const int groups = padded_rows(rows) / kRowGroup;
  const dim3 block(kWave * nw), grid(groups * kRowGroup);
  if (per_wave == 1)
    launch_kernel<kVector, B, 1>(grid, block, stream, x, rows, K, nchunks, groups, packed, rowsum, scale);
  else if (per_wave == 2)
    launch_kernel<kVector, B, 2>(grid, block, stream, x, rows, K, nchunks, groups, packed, rowsum, scale);
  else if (per_wave <= kMaxCachedSteps)
    launch_kernel<kVector, B, 4>(grid, block, stream, x, rows, K, nchunks, groups, packed, rowsum, scale);
  else
    launch_kernel<kVector, B, 0>(grid, block, stream, x, rows, K, nchunks, groups, packed, rowsum, scale);
  return hipGetLastError();
}

template <int B>
hipError_t launch_bits(const uint16_t* x, int rows, int K, uint32_t* packed, int32_t* rowsum,
                       uint16_t* scale, hipStream_t stream) {
  if (K % 16 == 0 && (reinterpret_cast<uintptr_t>(x) & 15u) == 0)
    return launch_vec_bits<true, B>(x, rows, K, packed, rowsum, scale, stream);
  return launch_vec_bits<false, B>(x, rows, K, packed, rowsum, scale, stream);
}

}  // namespace

hipError_t launch_quantize_pack(const uint16_t* x, int rows, int K, int bits, uint32_t* packed,
                                int32_t* rowsum, uint16_t* scale, hipStream_t stream) {
  switch (bits) {
    case 1: return launch_bits<1>(x, rows, K, packed, rowsum, scale, stream);
    case 2: return launch_bits<2>(x, rows, K, packed, rowsum, scale, stream);
    case 3: return launch_bits<3>(x, rows, K, packed, rowsum, scale, stream);
    case 4: return launch_bits<4>(x, rows, K, packed, rowsum, scale, stream);
    case 5: return launch_bits<5>(x, rows, K, packed, rowsum, scale, stream);
    case 6: return launch_bits<6>(x, rows, K, packed, rowsum, scale, stream);
    case 7: return launch_bits<7>(x, rows, K, packed, rowsum, scale, stream);
    case 8: return launch_bits<8>(x, rows, K, packed, rowsum, scale, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace apt
