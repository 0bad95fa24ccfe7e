// pack.hip - signed-INT -> bipolar-INT conversion and bit-plane packing for
// gfx950 (APT-LLM, arXiv 2508.19087: Sec. III-A conversion, Sec. IV-A
// decomposition and reassembly steps 1-3).
//
// A workgroup of 8 wavefronts owns one 8-row group of the packed layout; each
// wavefront owns one row and walks it in steps of 1024 codes: lane l converts
// codes [16 l, 16 l + 16) of the step (one 16-byte load), extracts each
// plane's 16 bits, and pairs with its neighbour lane to form one 32-bit word
// per plane.  Conversion flips the sign bit of the b-bit field; the row sum of
// bipolar values 2u - (2^b - 1) is reduced across the wave.  Wavefronts of the
// padding rows past the last row write zero words.
#include "apt_internal.h"

namespace apt {
namespace {

constexpr int kWave = 64;
constexpr int kWavesPerBlock = kRowGroup;
constexpr int kCodesPerLane = 16;
constexpr int kCodesPerStep = kWave * kCodesPerLane;  // 1024 = 8 chunks

template <bool kVector, int B>
__global__ __launch_bounds__(kWave* kWavesPerBlock) void pack_kernel(
    const int8_t* __restrict__ codes, int rows, int K, int nchunks,
    uint32_t* __restrict__ packed, int32_t* __restrict__ rowsum) {
  constexpr int bits = B;
  const int lane = threadIdx.x % kWave;
  const int row = blockIdx.x * kWavesPerBlock + threadIdx.x / kWave;  // < padded row count
  const bool real = row < rows;

  const uint32_t field_mask = ((1u << bits) - 1u) * 0x01010101u;
  const uint32_t sign_flip = (1u << (bits - 1)) * 0x01010101u;
  const int kpad = nchunks * kChunk;
  const int8_t* src = codes + (int64_t)min(row, rows - 1) * K;
  uint32_t usum = 0;

  auto load = [&](int base, uint32_t d[4]) {
    const int k0 = base + lane * kCodesPerLane;
    d[0] = d[1] = d[2] = d[3] = 0u;
    if (kVector) {
      // K % 16 == 0: the lane's 16 codes are all valid or all padding.
      if (real && k0 < K) {
        uint4 v = *reinterpret_cast<const uint4*>(src + k0);
        d[0] = v.x; d[1] = v.y; d[2] = v.z; d[3] = v.w;
      }
    } else if (real) {
#pragma unroll
      for (int t = 0; t < kCodesPerLane; ++t) {
        int k = k0 + t;
        uint32_t b = (k < K) ? (uint32_t)(uint8_t)src[k] : 0u;
        d[t / 4] |= b << (8 * (t % 4));
      }
    }
  };
  auto process = [&](int base, const uint32_t d[4]) {
    const int k0 = base + lane * kCodesPerLane;
    // Bipolar words, one per byte; padding codes and padding rows stay all-zero.
    uint32_t u[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      uint32_t valid_bytes = 0xFFFFFFFFu;
      int kt = k0 + 4 * t;
      if (!real) {
        valid_bytes = 0u;
      } else if (!kVector) {
        int n_valid = K - kt;
        valid_bytes = n_valid >= 4 ? 0xFFFFFFFFu : (n_valid <= 0 ? 0u : ((1u << (8 * n_valid)) - 1u));
      } else if (k0 >= K) {
        valid_bytes = 0u;
      }
      u[t] = ((d[t] & field_mask) ^ sign_flip) & valid_bytes;
      usum = __builtin_amdgcn_sad_u8(u[t], 0u, usum);
    }
    const int chunk = k0 / kChunk;
    const int word = (k0 % kChunk) / 32;
    const bool upper_half = (lane & 1) != 0;  // codes 16..31 of the word
    const bool in_range = k0 < kpad;
#pragma unroll
    for (int i = 0; i < bits; ++i) {
      uint32_t half = gather_plane_nibble(u[0], i) | (gather_plane_nibble(u[1], i) << 4) |
                      (gather_plane_nibble(u[2], i) << 8) | (gather_plane_nibble(u[3], i) << 12);
      uint32_t other = __shfl_xor(half, 1);
      if (!upper_half && in_range) {
        packed[plane_words(row, chunk, i, nchunks, bits) + word] = half | (other << 16);
      }
    }
  };

  // Four steps per trip: their loads are all in flight before the first is
  // used.
  constexpr int kGroup = 4;
  int base = 0;
  for (; base + kGroup * kCodesPerStep <= kpad; base += kGroup * kCodesPerStep) {
    uint32_t d[kGroup][4];
#pragma unroll
    for (int s = 0; s < kGroup; ++s) load(base + s * kCodesPerStep, d[s]);
#pragma unroll
    for (int s = 0; s < kGroup; ++s) process(base + s * kCodesPerStep, d[s]);
  }
  for (; base < kpad; base += kCodesPerStep) {
    uint32_t d[4];
    load(base, d);
    process(base, d);
  }

  if (rowsum != nullptr && real) {
    for (int off = kWave / 2; off > 0; off >>= 1) usum += __shfl_xor(usum, off);
    if (lane == 0) {
      // sum_k (2 u - (2^b - 1)) over the K real codes
      uint32_t top = (1u << bits) - 1u;
      rowsum[row] = (int32_t)(2u * usum - top * (uint32_t)K);
    }
  }
}

template <int B>
hipError_t launch_pack_bits(const int8_t* codes, int rows, int K, uint32_t* packed, int32_t* rowsum,
                            hipStream_t stream) {
  const int nchunks = num_chunks(K);
  dim3 block(kWave * kWavesPerBlock);
  dim3 grid(padded_rows(rows) / kWavesPerBlock);
  const bool vec = (K % 16 == 0) && ((reinterpret_cast<uintptr_t>(codes) & 15u) == 0);
  if (vec)
    hipLaunchKernelGGL((pack_kernel<true, B>), grid, block, 0, stream, codes, rows, K, nchunks,
                       packed, rowsum);
  else
    hipLaunchKernelGGL((pack_kernel<false, B>), grid, block, 0, stream, codes, rows, K, nchunks,
                       packed, rowsum);
  return hipGetLastError();
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

}  // namespace apt
