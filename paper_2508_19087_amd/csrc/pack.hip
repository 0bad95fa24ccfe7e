// pack.hip - signed-INT -> bipolar-INT conversion and bit-plane packing for
// gfx950 (APT-LLM, arXiv 2508.19087: Sec. III-A conversion, Sec. IV-A
// decomposition and reassembly steps 1-3), from int8 codes or, quantizing
// per row (token) on the way, from fp16 activations.
//
// Quantizer of an fp16 row (the bipolar form of a linear quantizer, Sec.
// III-A; the scale rule and the rounding are this library's choice, the paper
// fixes neither): s = fp16(absmax_k |x[k]| / (2^b - 1)) with an IEEE fp32
// divide, so the largest magnitude lands on the outermost odd level; element
// x goes to the odd level 2 floor(t / 2) + 1 of t = x / s clamped to
// +-(2^b - 1), i.e. to the signed code floor(t / 2) clamped to
// [-2^(b-1), 2^(b-1) - 1].  A row with s = 0 gets t = 0.
//
// One workgroup per row; the last row's workgroup also writes the zero words
// of the padding rows of its 8-row group.  The row is split over the
// workgroup's nw waves in steps of 1024 elements: wave w takes steps w, w + nw,
// ...; lane l of a step takes elements [16 l, 16 l + 16) (buffer loads whose
// range is the row, so reads past K return 0).  When every wave
// has at most 4 steps (K <= 32768) the loaded values stay in registers: the
// fp16 source folds the row's largest magnitude first (pass 1, reduced over
// the workgroup through LDS) and quantizes from registers, so HBM sees every
// input byte once.  Longer rows are walked in rounds of 4 steps per wave (and
// loaded twice by the fp16 source).
//
// Conversion: u = (x mod 2^b) XOR 2^(b-1), four codes per dword.  Packing: the
// 16 bipolar words of a lane (one byte each) go through an 8x8 bit-matrix
// transpose per 8 elements, which leaves plane i of those elements in byte i;
// for b <= 4 the high nibbles are zero and the transpose reduces to two delta
// swaps on one dword.  Lanes 2m and 2m+1 hold the two 16-bit halves of one
// plane word; per pair of planes they swap halves with one DPP move, and the
// even lane stores plane i, the odd lane plane i+1.  The row sum of bipolar
// values 2u - (2^b - 1) is reduced over the workgroup.
//
// Workgroups are dispatched to the 8 XCDs round robin; when the row count is a
// multiple of 8, rows are assigned so that consecutive workgroups on one XCD
// take consecutive rows, and the 8 rows of a packed row group, which share
// every 128-byte plane segment (16 bytes each), meet in that XCD's L2.
//
// Division in the quantizer: instead of a correctly rounded fp32 divide per
// element, each row computes r = RN(1 / s) once and each element
//     h0 = fma(x, r / 2, +0),  e = fma(-h0, 2 s, x),  h = fma(e, r / 2, h0),
// the quotient correction of Markstein's division with a correctly rounded
// reciprocal, applied to the half quotient.  h equals RN(x / s) / 2 (up to the
// sign of a zero) for every finite fp16 x and positive finite fp16 s; the test
// suite checks all of those pairs on the CPU.
#include <algorithm>

#include "apt_internal.h"
#include "rowcode.h"

namespace apt {
namespace {

using namespace rowcode;

constexpr int kWave = 64;
constexpr int kMaxWaves = 8;
constexpr int kStep = kWave * kLaneElems;  // 1024 elements = 8 chunks
constexpr int kMaxCachedSteps = 4;
constexpr int kTargetWaves = 4096;  // 16 per CU
constexpr int kXcds = 8;

// kSteps: steps each wave keeps in registers (1, 2 or 4), or 0 for rows too
// long for that.  groups = rows / 8 selects the XCD-aware row order (rows a
// multiple of 8), 0 the plain one.  scale is written by the fp16 source only.
template <class Src, int B, int kSteps>
__global__ __launch_bounds__(kWave* kMaxWaves) void pack_rows_kernel(
    const uint8_t* __restrict__ src, int rows, int K, int nchunks, int groups,
    uint32_t* __restrict__ packed, int32_t* __restrict__ rowsum, uint16_t* __restrict__ scale) {
  constexpr int kHeld = kSteps > 0 ? kSteps : kMaxCachedSteps;
  __shared__ uint32_t lds_red[kMaxWaves];
  const int nw = blockDim.x / kWave;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x % kWave;
  const int row = groups > 0 ? (blockIdx.x % kXcds) * groups + blockIdx.x / kXcds : blockIdx.x;
  // the last row also writes the padding rows of its row group (uniform)
  const int pad_rows = row == rows - 1 ? (rows + kRowGroup - 1) / kRowGroup * kRowGroup - rows : 0;
  const int kpad = nchunks * kChunk;
  const int nsteps = (kpad + kStep - 1) / kStep;
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(src + (int64_t)row * K * Src::kElemBytes), 0,
      (uint32_t)K * Src::kElemBytes, kRawBufferFlags);
  auto k_of = [&](int j) { return j * kStep + lane * kLaneElems; };

  uint32_t d[kHeld][Src::kDwords];
  float rh = 0.0f, s2 = 0.0f;
  if constexpr (Src::kScaled) {
    // Pass 1: the row's largest magnitude, then its scale.
    ushort2_t mm = {0, 0};
    for (int j0 = wave; j0 < nsteps; j0 += kHeld * nw) {
#pragma unroll
      for (int t = 0; t < kHeld; ++t) Src::load(rsrc, k_of(j0 + t * nw), d[t]);
#pragma unroll
      for (int t = 0; t < kHeld; ++t) mm = Src::fold_max(mm, d[t]);
      if (kSteps > 0) break;  // one round covers all steps; d stays for pass 2
    }
    uint32_t m = max((uint32_t)mm.x, (uint32_t)mm.y);
    for (int off = kWave / 2; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
    if (lane == 0) lds_red[wave] = m;
    __syncthreads();
    m = 0u;
    for (int w = 0; w < nw; ++w) m = max(m, lds_red[w]);
    __syncthreads();  // lds_red is reused for the row sum
    const uint16_t s16 = row_scale<B>(m, rh, s2);
    if (threadIdx.x == 0) scale[row] = s16;
  } else if (kSteps > 0) {
#pragma unroll
    for (int t = 0; t < kHeld; ++t) Src::load(rsrc, k_of(wave + t * nw), d[t]);
  }

  // Pass 2: convert (or quantize) and pack.
  uint32_t usum = 0u;
  const bool odd = (lane & 1) != 0;
  auto process = [&](int j, const uint32_t* dd) __attribute__((always_inline)) {
    const int k0 = k_of(j);
    uint32_t u[4];
    Src::words(dd, rh, s2, u);
    // padding elements: all-zero words
    if (Src::kVector) {
      const uint32_t valid = k0 < K ? 0xFFFFFFFFu : 0u;  // K % 16 == 0
#pragma unroll
      for (int t = 0; t < 4; ++t) u[t] &= valid;
    } else {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int n_valid = K - (k0 + 4 * t);
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
      const uint32_t wv = plane_word(sa, sb, i % 4, odd);  // even: plane i, odd: plane i+1
      if (!odd || i + 1 < B) {
        uint32_t* w = dst + (i + (odd ? 1 : 0)) * kPlaneStride;
        *w = wv;
        for (int r = 1; r <= pad_rows; ++r) w[r * kWordsPerPlane] = 0u;
      }
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
      for (int t = 0; t < kHeld; ++t) Src::load(rsrc, k_of(j0 + t * nw), d[t]);
#pragma unroll
      for (int t = 0; t < kHeld; ++t)
        if (j0 + t * nw < nsteps) process(j0 + t * nw, d[t]);
    }
  }

  if (rowsum != nullptr) {
    for (int off = kWave / 2; off > 0; off >>= 1) usum += __shfl_xor(usum, off);
    if (nw > 1) {
      if (lane == 0) lds_red[wave] = usum;
      __syncthreads();
      usum = 0u;
      for (int w = 0; w < nw; ++w) usum += lds_red[w];
    }
    if (threadIdx.x == 0)
      // sum_k (2 u - (2^b - 1)) over the K real elements
      rowsum[row] = (int32_t)(2u * usum - ((1u << B) - 1u) * (uint32_t)K);
  }
}

template <class Src, int B>
hipError_t launch_rows(const void* src, int rows, int K, uint32_t* packed, int32_t* rowsum,
                       uint16_t* scale, hipStream_t stream) {
  const int nchunks = num_chunks(K);
  const int nsteps = (nchunks * kChunk + kStep - 1) / kStep;
  // Fewest waves per row that hold the row in registers (the per-row
  // reductions and the scale cost the same in every wave), but more while the
  // whole grid has fewer than kTargetWaves waves.
  const int max_nw = std::min(nsteps, kMaxWaves);
  int nw = std::min((nsteps + kMaxCachedSteps - 1) / kMaxCachedSteps, max_nw);
  while (nw < max_nw && (int64_t)rows * nw < kTargetWaves) nw = std::min(2 * nw, max_nw);
  const int per_wave = (nsteps + nw - 1) / nw;
  const int groups = rows % kRowGroup == 0 ? rows / kRowGroup : 0;
  const dim3 block(kWave * nw), grid(rows);
  const uint8_t* s = static_cast<const uint8_t*>(src);
  auto kern = per_wave == 1                   ? pack_rows_kernel<Src, B, 1>
              : per_wave == 2                 ? pack_rows_kernel<Src, B, 2>
              : per_wave <= kMaxCachedSteps   ? pack_rows_kernel<Src, B, 4>
                                              : pack_rows_kernel<Src, B, 0>;
  return launch_kernel(kern, grid, block, 0, stream, s, rows, K, nchunks, groups, packed, rowsum,
                       scale);
}

// The 16-byte load path needs whole 16-element groups and a 16-byte aligned base.
bool vector_ok(const void* p, int K) {
  return K % 16 == 0 && (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
}

template <int B>
hipError_t launch_pack_bits(const int8_t* codes, int rows, int K, uint32_t* packed,
                            int32_t* rowsum, hipStream_t stream) {
  if (vector_ok(codes, K))
    return launch_rows<CodeRow<true, B>, B>(codes, rows, K, packed, rowsum, nullptr, stream);
  return launch_rows<CodeRow<false, B>, B>(codes, rows, K, packed, rowsum, nullptr, stream);
}

template <int B>
hipError_t launch_quantize_bits(const uint16_t* x, int rows, int K, uint32_t* packed,
                                int32_t* rowsum, uint16_t* scale, hipStream_t stream) {
  if (vector_ok(x, K))
    return launch_rows<HalfRow<true, B>, B>(x, rows, K, packed, rowsum, scale, stream);
  return launch_rows<HalfRow<false, B>, B>(x, rows, K, packed, rowsum, scale, stream);
}

}  // namespace

hipError_t launch_pack(const int8_t* codes, int rows, int K, int bits, uint32_t* packed,
                       int32_t* rowsum, hipStream_t stream) {
  switch (bits) {
    case 1: return launch_pack_bits<1>(codes, rows, K, packed, rowsum, stream);
    case 2: return launch_pack_bits<2>(codes, rows, K, packed, rowsum, stream);
    case 3: return launch_pack_bits<3>(codes, rows, K, packed, rowsum, stream);
    case 4: return launch_pack_bits<4>(codes, rows, K, packed, rowsum, stream);
    case 5: return launch_pack_bits<5>(codes, rows, K, packed, rowsum, stream);
    case 6: return launch_pack_bits<6>(codes, rows, K, packed, rowsum, stream);
    case 7: return launch_pack_bits<7>(codes, rows, K, packed, rowsum, stream);
    case 8: return launch_pack_bits<8>(codes, rows, K, packed, rowsum, stream);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_quantize_pack(const uint16_t* x, int rows, int K, int bits, uint32_t* packed,
                                int32_t* rowsum, uint16_t* scale, hipStream_t stream) {
  switch (bits) {
    case 1: return launch_quantize_bits<1>(x, rows, K, packed, rowsum, scale, stream);
    case 2: return launch_quantize_bits<2>(x, rows, K, packed, rowsum, scale, stream);
    case 3: return launch_quantize_bits<3>(x, rows, K, packed, rowsum, scale, stream);
    case 4: return launch_quantize_bits<4>(x, rows, K, packed, rowsum, scale, stream);
    case 5: return launch_quantize_bits<5>(x, rows, K, packed, rowsum, scale, stream);
    case 6: return launch_quantize_bits<6>(x, rows, K, packed, rowsum, scale, stream);
    case 7: return launch_quantize_bits<7>(x, rows, K, packed, rowsum, scale, stream);
    case 8: return launch_quantize_bits<8>(x, rows, K, packed, rowsum, scale, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace apt
