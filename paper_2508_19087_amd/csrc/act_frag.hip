// act_frag.hip - activations straight from int8 codes or fp16 values into the
// int8 MFMA route's operand fragments, for gfx950 (APT-LLM, arXiv 2508.19087:
// Sec. III-A conversion and, for fp16, the bipolar form of the per-row
// linear quantizer).
//
// The reassembled int8 route (gemm_int8.h) multiplies the bipolar words u of
// the activations as whole bytes: its expansion kernel rebuilds them from the
// packed bit-planes.  When the caller holds the codes (or fp16 values) this
// kernel writes the same fragment bytes from them directly, so the packer's
// planes are never written and read back: one launch instead of two, and the
// activation bytes cross HBM once.  The bytes, the row sums and the scales
// equal those of the packer followed by the expansion, bit for bit.
//
// Fragment layout (that of expand_a_kernel, int8 format): for 32-row block
// mb and k-step s (32 elements: chunk s / 4, word s mod 4), 64 vectors of 16
// bytes; row l of the block takes vector l (dwords 0..3) and vector 32 + l
// (dwords 4..7), and byte j of dword t is the operand byte y of element
// 8 j + t of the word: y = u for b <= 7, u XOR 0x80 for b = 8.  Elements past
// K are padding (u = 0), the k-steps of the chunk that makes the chunk count
// even are all-zero bytes, and rows past M up to the block are padding rows.
//
// A workgroup takes 8 consecutive rows and walks their K: lane l of a wave
// takes row l mod 8 and word l / 8 of each group of 8 words, so that one
// store instruction writes the 16-byte pieces of 8 rows that make one whole
// 128-byte line of a fragment, and one load instruction reads 8 rows' 256
// contiguous bytes.  The fp16 row maximum and the row sum are reductions over
// the lanes of a row (three lane swaps, then LDS across waves).  The loads of
// up to kHeldIters word groups per lane are issued before any is used.
#include <algorithm>
#include <type_traits>

#include "apt_internal.h"
#include "rowcode.h"

namespace apt {
namespace {

using namespace rowcode;

constexpr int kWave = 64;
constexpr int kMaxWaves = 16;
constexpr int kRows = 8;                      // rows per workgroup
constexpr int kWordLanes = kWave / kRows;     // words per wave and iteration
constexpr int kWordElems = 32;
constexpr int kBlockRows = 32;
// word groups per lane whose source stays in registers (issued up front)
constexpr int kHeldIters = 4;

typedef int v4i __attribute__((ext_vector_type(4)));

template <bool kHalf, bool kVec, int B>
__global__ __launch_bounds__(kWave* kMaxWaves) void act_frag_kernel(
    const uint8_t* __restrict__ src, int M, int K, int nchunks, int nsteps, int mblocks,
    v4i* __restrict__ frag, int32_t* __restrict__ rowsum, uint16_t* __restrict__ scale,
    uint16_t* __restrict__ scale_out, int* __restrict__ counters, int ncounters) {
  using Src = typename std::conditional<kHalf, HalfRow<kVec, B>, CodeRow<kVec, B>>::type;
  constexpr int kD = Src::kDwords;
  __shared__ uint32_t lds_red[kMaxWaves][kRows];
  // The stream-K arrival counters of this call start cleared (the GEMM
  // launch follows in stream order).
  for (int i = blockIdx.x * (int)blockDim.x + threadIdx.x; i < ncounters; i += gridDim.x * blockDim.x)
    counters[i] = 0;
  const int nw = blockDim.x / kWave;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int r = lane % kRows, wl = lane / kRows;
  const int row = blockIdx.x * kRows + r;  // < mblocks * 32 (the grid covers the blocks exactly)
  const bool real = row < M;
  const int words = nchunks * kWordsPerPlane;  // words holding elements (up to K_pad)
  const int step = kWordLanes * nw;            // words per iteration of the workgroup
  const int iters = (words + step - 1) / step;
  // one resource over the whole [M][K] source: offsets past its end (rows
  // past M) read zeros; elements past K of a row are masked below
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(src), 0, (uint32_t)((int64_t)M * K * Src::kElemBytes), kRawBufferFlags);
  const int64_t row_off = (int64_t)row * K;  // elements
  auto word_of = [&](int it) { return it * step + wave * kWordLanes + wl; };
  // the 32 elements of word w of this lane's row, elements past K as zero bits
  auto load = [&](int w, uint32_t (&d)[2][kD]) __attribute__((always_inline)) {
    const int k0 = w * kWordElems;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int kh = k0 + h * kLaneElems;
      // (whole-source byte offsets stay below 2^31: the host checks)
      Src::load(rsrc, (int)(row_off + (kh < K ? kh : 0)), d[h]);
      const int n_valid = real ? K - kh : 0;
#pragma unroll
      for (int t = 0; t < kD; ++t) {
        constexpr int per = kLaneElems / kD;  // elements per dword: 4 codes or 2 halves
        const int nv = n_valid - per * t;
        const uint32_t keep = nv >= per ? 0xFFFFFFFFu : (nv <= 0 ? 0u : ((1u << (8 * Src::kElemBytes * nv)) - 1u));
        d[h][t] &= keep;
      }
    }
  };

  uint32_t held[kHeldIters][2][kD];
#pragma unroll
  for (int i = 0; i < kHeldIters; ++i)
    if (i < iters && word_of(i) < words) load(word_of(i), held[i]);
  float rh = 0.0f, s2 = 0.0f;
  if constexpr (kHalf) {
    // Pass 1: the row's largest magnitude, then its scale.
    ushort2_t mm = {0, 0};
#pragma unroll
    for (int i = 0; i < kHeldIters; ++i)
      if (i < iters && word_of(i) < words) {
        mm = Src::fold_max(mm, held[i][0]);
        mm = Src::fold_max(mm, held[i][1]);
      }
    for (int it = kHeldIters; it < iters; ++it) {
      const int w = word_of(it);
      if (w >= words) continue;
      uint32_t d[2][kD];
      load(w, d);
      mm = Src::fold_max(mm, d[0]);
      mm = Src::fold_max(mm, d[1]);
    }
    uint32_t m = max((uint32_t)mm.x, (uint32_t)mm.y);
    for (int off = kRows; off < kWave; off <<= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
    if (wl == 0) lds_red[wave][r] = m;
    __syncthreads();
    m = 0u;
    for (int v = 0; v < nw; ++v) m = max(m, lds_red[v][r]);
    __syncthreads();  // lds_red is reused for the row sum
    const uint16_t s16 = row_scale<B>(m, rh, s2);
    if (wave == 0 && wl == 0 && real) {
      scale[row] = s16;
      if (scale_out != nullptr) scale_out[row] = s16;
    }
  }

  // Pass 2: operand bytes of each word, in the fragment order.
  const int mb = row / kBlockRows, l = row % kBlockRows;
  uint32_t usum = 0u;
  auto emit = [&](int w, const uint32_t (&d)[2][kD]) __attribute__((always_inline)) {
    uint32_t c[8];  // byte b of c[i]: u of element 4 i + b of the word
    Src::words(d[0], rh, s2, c);
    Src::words(d[1], rh, s2, c + 4);
    const int k0 = w * kWordElems;
#pragma unroll
    for (int t = 0; t < 8; ++t) {  // padding elements and padding rows: u = 0
      const int n_valid = real ? K - (k0 + 4 * t) : 0;
      c[t] &= n_valid >= 4 ? 0xFFFFFFFFu : (n_valid <= 0 ? 0u : ((1u << (8 * n_valid)) - 1u));
      usum = __builtin_amdgcn_sad_u8(c[t], 0u, usum);
      if (B == 8) c[t] ^= 0x80808080u;
    }
    // o[t], byte j = element 8 j + t = byte t mod 4 of c[2 j + t / 4]
    uint32_t o[8];
#pragma unroll
    for (int h = 0; h < 2; ++h) {          // h = t / 4: the odd or even c
#pragma unroll
      for (int tp = 0; tp < 4; tp += 2) {  // t mod 4 in pairs
        // [c0.b, c2.b, c0.b', c2.b'] and [c4.b, c6.b, c4.b', c6.b'] with b = tp, b' = tp + 1
        const uint32_t sel = (uint32_t)(tp | (4 + tp) << 8 | (tp + 1) << 16 | (5 + tp) << 24);
        const uint32_t lo = __builtin_amdgcn_perm(c[2 + h], c[h], sel);
        const uint32_t hi = __builtin_amdgcn_perm(c[6 + h], c[4 + h], sel);
        o[4 * h + tp] = __builtin_amdgcn_perm(hi, lo, 0x05040100u);
        o[4 * h + tp + 1] = __builtin_amdgcn_perm(hi, lo, 0x07060302u);
      }
    }
    v4i* f = frag + ((int64_t)mb * nsteps + w) * kWave;
    f[l] = v4i{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
    f[l + 32] = v4i{(int)o[4], (int)o[5], (int)o[6], (int)o[7]};
  };
#pragma unroll
  for (int i = 0; i < kHeldIters; ++i)
    if (i < iters && word_of(i) < words) emit(word_of(i), held[i]);
  for (int it = kHeldIters; it < iters; ++it) {
    const int w = word_of(it);
    if (w >= words) continue;
    uint32_t d[2][kD];
    load(w, d);
    emit(w, d);
  }
  // the chunk that makes the count even: all-zero bytes
  for (int w = words + wave * kWordLanes + wl; w < nsteps; w += step) {
    v4i* f = frag + ((int64_t)mb * nsteps + w) * kWave;
    f[l] = v4i{0, 0, 0, 0};
    f[l + 32] = v4i{0, 0, 0, 0};
  }

  for (int off = kRows; off < kWave; off <<= 1) usum += __shfl_xor(usum, off);
  if (nw > 1) {
    if (wl == 0) lds_red[wave][r] = usum;
    __syncthreads();
    usum = 0u;
    for (int v = 0; v < nw; ++v) usum += lds_red[v][r];
  }
  if (wave == 0 && wl == 0 && real)
    // sum_k (2 u - (2^b - 1)) over the K real elements
    rowsum[row] = (int32_t)(2u * usum - ((1u << B) - 1u) * (uint32_t)K);
}

template <bool kHalf, bool kVec, int B>
hipError_t launch_one(const void* src, int M, int K, int nchunks, int nsteps, void* frag,
                      int32_t* rowsum, uint16_t* scale, uint16_t* scale_out, int* counters,
                      int ncounters, hipStream_t s) {
  const int mblocks = (M + kBlockRows - 1) / kBlockRows;
  const dim3 grid((unsigned)(mblocks * (kBlockRows / kRows)));
  // waves: enough for the words of a row at 8 per wave, at most kMaxWaves
  // for the fp16 source (its conversion needs them) and 8 for codes (smaller
  // workgroups find room sooner beside another call's GEMM)
  const int words = nchunks * kWordsPerPlane;
  const int cap = kHalf ? kMaxWaves : 8;
  const int waves = std::min(cap, (words + kWordLanes - 1) / kWordLanes);
  return launch_kernel(act_frag_kernel<kHalf, kVec, B>, grid, dim3(waves * kWave), 0, s,
                       static_cast<const uint8_t*>(src), M, K, nchunks, nsteps, mblocks,
                       static_cast<v4i*>(frag), rowsum, scale, scale_out, counters, ncounters);
}

template <int B>
hipError_t launch_b(const void* src, bool fp16, bool vec, int M, int K, int nchunks, int nsteps,
                    void* frag, int32_t* rowsum, uint16_t* scale, uint16_t* scale_out,
                    int* counters, int ncounters, hipStream_t s) {
  if (fp16)
    return vec ? launch_one<true, true, B>(src, M, K, nchunks, nsteps, frag, rowsum, scale,
                                           scale_out, counters, ncounters, s)
               : launch_one<true, false, B>(src, M, K, nchunks, nsteps, frag, rowsum, scale,
                                            scale_out, counters, ncounters, s);
  return vec ? launch_one<false, true, B>(src, M, K, nchunks, nsteps, frag, rowsum, scale,
                                          scale_out, counters, ncounters, s)
             : launch_one<false, false, B>(src, M, K, nchunks, nsteps, frag, rowsum, scale,
                                           scale_out, counters, ncounters, s);
}

}  // namespace

hipError_t launch_act_frag(const void* src, bool fp16, int M, int K, int q, int nsteps, void* frag,
                           int32_t* rowsum, uint16_t* scale, uint16_t* scale_out, int* counters,
                           int ncounters, hipStream_t s) {
  const int nchunks = num_chunks(K);
  // 16-byte loads: every row starts 16-byte aligned and holds whole vectors
  const bool vec = (reinterpret_cast<uintptr_t>(src) & 15u) == 0 && K % 16 == 0;
  switch (q) {
    case 1: return launch_b<1>(src, fp16, vec, M, K, nchunks, nsteps, frag, rowsum, scale, scale_out, counters, ncounters, s);
    case 2: return launch_b<2>(src, fp16, vec, M, K, nchunks, nsteps, frag, rowsum, scale, scale_out, counters, ncounters, s);
    case 3: return launch_b<3>(src, fp16, vec, M, K, nchunks, nsteps, frag, rowsum, scale, scale_out, counters, ncounters, s);
    case 4: return launch_b<4>(src, fp16, vec, M, K, nchunks, nsteps, frag, rowsum, scale, scale_out, counters, ncounters, s);
    case 5: return launch_b<5>(src, fp16, vec, M, K, nchunks, nsteps, frag, rowsum, scale, scale_out, counters, ncounters, s);
    case 6: return launch_b<6>(src, fp16, vec, M, K, nchunks, nsteps, frag, rowsum, scale, scale_out, counters, ncounters, s);
    case 7: return launch_b<7>(src, fp16, vec, M, K, nchunks, nsteps, frag, rowsum, scale, scale_out, counters, ncounters, s);
    case 8: return launch_b<8>(src, fp16, vec, M, K, nchunks, nsteps, frag, rowsum, scale, scale_out, counters, ncounters, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace apt
