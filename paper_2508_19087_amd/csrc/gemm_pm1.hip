// gemm_pm1.hip - the plane-pair +-1 MFMA route of the WpAq bipolar-INT GEMM
// for gfx950 (APT-LLM, arXiv 2508.19087, Sec. III-B).
//
// Every weight plane i and activation plane j stays a separate 1-bit matrix,
// as in the paper's decomposition, and every (i, j) pair is one int8 matrix
// multiply on the matrix cores.  A bit b of plane j becomes the int8 operand
// (2b - 1) 2^j, so the product of planes i and j is 2^(i+j) Y(i,j) and the
// paper's shift-and-sum recovery (Sec. III-B) happens inside the accumulator:
// all p*q plane products of an output accumulate in the same registers.
// Operands up to 2^6 fit int8, so this route takes p, q <= 7.
//
// Padding bits are zero, i.e. operand -2^j on both sides, so each padding
// element adds sum_{i,j} 2^(i+j) = (2^p-1)(2^q-1) to every output; the
// epilogue subtracts (K_pad - K)(2^p-1)(2^q-1).
//
// The route exists as the p*q-MFMA comparison point for the reassembled int8
// route, which does one MFMA per element pair.
#include "apt_internal.h"

namespace apt {
namespace {

constexpr int kWave = 64;
constexpr int kRowBytes = kChunk + 16;
constexpr int kBM = 64, kBN = 64, kWM = 2, kWN = 2;
constexpr int kThreads = kWM * kWN * kWave;

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

struct Pm1Params {
  GemmArgs g;
  int nchunks;
  int tiles_n;
};

// Operand bytes of plane word pw for scale 2^j, element order as in the
// reassembled route (dword t, byte e <- bit 8e + t).  Per byte,
// ((bit << (j+1)) + 0x80 - 2^j) XOR 0x80 is 2^j for bit 1 and -2^j for bit 0
// with no carry between bytes (all sums stay below 0x100 for j <= 6).
__device__ __forceinline__ void plane_bytes(uint32_t pw, int j, uint32_t out[8]) {
  const uint32_t bias = (0x80u - (1u << j)) * 0x01010101u;
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    uint32_t bits = (pw >> t) & 0x01010101u;
    out[t] = ((bits << (j + 1)) + bias) ^ 0x80808080u;
  }
}

// One 128-element chunk of ROWS rows (B planes each) -> B*ROWS LDS rows.
// A work item is one 32-element word of one row (all B planes of it).
template <int B, int ROWS>
struct PlaneStage {
  static constexpr int kItems = ROWS * kWordsPerPlane / kThreads;
  static_assert(ROWS * kWordsPerPlane % kThreads == 0, "items must divide evenly");
  uint32_t raw[kItems][B];

  __device__ __forceinline__ void load(const uint32_t* __restrict__ packed, int row0, int rows,
                                       int nchunks, int chunk, int tid) {
#pragma unroll
    for (int it = 0; it < kItems; ++it) {
      const int item = tid + kThreads * it;
      const int r = row0 + item / kWordsPerPlane;
      const int w = item % kWordsPerPlane;
      if (r < rows) {
        const uint32_t* src = packed + plane_words(r, chunk, 0, nchunks, B) + w;
#pragma unroll
        for (int i = 0; i < B; ++i) raw[it][i] = src[i * kPlaneStride];
      } else {
#pragma unroll
        for (int i = 0; i < B; ++i) raw[it][i] = 0u;
      }
    }
  }

  __device__ __forceinline__ void store(uint8_t* lds_tile, int tid) const {
#pragma unroll
    for (int it = 0; it < kItems; ++it) {
      const int item = tid + kThreads * it;
      const int r = item / kWordsPerPlane;
      const int w = item % kWordsPerPlane;
#pragma unroll
      for (int i = 0; i < B; ++i) {
        uint32_t o[8];
        plane_bytes(raw[it][i], i, o);
        uint4* d4 = reinterpret_cast<uint4*>(lds_tile + (i * ROWS + r) * kRowBytes + w * 32);
        d4[0] = make_uint4(o[0], o[1], o[2], o[3]);
        d4[1] = make_uint4(o[4], o[5], o[6], o[7]);
      }
    }
  }
};

template <int P, int Q>
__global__ __launch_bounds__(kThreads) void gemm_pm1_kernel(Pm1Params prm) {
  constexpr int WTM = kBM / kWM, WTN = kBN / kWN;
  static_assert(WTM == 32 && WTN == 32, "one 32x32 MFMA tile per wave");
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const GemmArgs& g = prm.g;
  const int NC = prm.nchunks;
  const int tid = threadIdx.x;
  const int lane = tid % kWave;
  const int wave = tid / kWave;
  const int wm = wave / kWN, wn = wave % kWN;
  const int tm = blockIdx.x / prm.tiles_n, tn = blockIdx.x % prm.tiles_n;
  const int m0 = tm * kBM, n0 = tn * kBN;

  PlaneStage<Q, kBM> sa;
  PlaneStage<P, kBN> sw;
  v16i acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0;

  const int lrow = lane % 32;
  const int lk = (lane / 32) * 16;
  uint8_t* lds_w = lds + Q * kBM * kRowBytes;

  sa.load(g.a_packed, m0, g.M, NC, 0, tid);
  sw.load(g.w_packed, n0, g.N, NC, 0, tid);
  for (int c = 0; c < NC; ++c) {
    __syncthreads();  // previous chunk's MFMA reads are done
    sa.store(lds, tid);
    sw.store(lds_w, tid);
    __syncthreads();
    if (c + 1 < NC) {
      sa.load(g.a_packed, m0, g.M, NC, c + 1, tid);
      sw.load(g.w_packed, n0, g.N, NC, c + 1, tid);
    }
#pragma unroll
    for (int ks = 0; ks < kChunk / 32; ++ks) {
      v4i bf[P];
#pragma unroll
      for (int i = 0; i < P; ++i)
        bf[i] = *reinterpret_cast<const v4i*>(lds_w + (i * kBN + wn * WTN + lrow) * kRowBytes + lk + ks * 32);
#pragma unroll
      for (int j = 0; j < Q; ++j) {
        v4i af = *reinterpret_cast<const v4i*>(lds + (j * kBM + wm * WTM + lrow) * kRowBytes + lk + ks * 32);
#pragma unroll
        for (int i = 0; i < P; ++i) acc = __builtin_amdgcn_mfma_i32_32x32x32_i8(af, bf[i], acc, 0, 0, 0);
      }
    }
  }

  const uint32_t ab = ((1u << P) - 1u) * ((1u << Q) - 1u);
  const uint32_t pad_term = (uint32_t)(NC * kChunk - g.K) * ab;
  const int n = n0 + wn * WTN + lrow;
  if (n >= g.N) return;
  const float sw_f = g.c_fp16 ? __half2float(g.w_scale[n]) : 0.f;
  // zero-point terms of column n (the zeros need the row sums)
  const bool affine = g.a_zero != nullptr;
  const float zw_f = affine ? __half2float(g.w_zero[n]) : 0.f;
  const float col_f = affine ? sw_f * (float)g.w_rowsum[n] + (float)g.K * zw_f : 0.f;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int m = m0 + wm * WTM + (v / 4) * 8 + (lane / 32) * 4 + (v % 4);
    if (m < g.M) {
      const int32_t cval = (int32_t)((uint32_t)acc[v] - pad_term);
      const int64_t o = (int64_t)m * g.N + n;
      if (g.c_int32) g.c_int32[o] = cval;
      if (g.c_fp16) {
        float f;
        if (affine) {
          f = affine_value(cval, __half2float(g.a_scale[m]), sw_f, zw_f, (float)g.a_rowsum[m],
                           __half2float(g.a_zero[m]), col_f);
        } else {
          f = (float)cval * __half2float(g.a_scale[m]);
          f = f * sw_f;
        }
        g.c_fp16[o] = __float2half_rn(f);
      }
    }
  }
}

template <int P, int Q>
hipError_t launch_pq(const Pm1Params& prm0, hipStream_t stream) {
  Pm1Params prm = prm0;
  prm.tiles_n = (prm.g.N + kBN - 1) / kBN;
  const int tiles_m = (prm.g.M + kBM - 1) / kBM;
  const size_t lds = (size_t)(Q * kBM + P * kBN) * kRowBytes;
  auto kern = gemm_pm1_kernel<P, Q>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  return launch_kernel(kern, dim3(tiles_m * prm.tiles_n), dim3(kThreads), lds, stream, prm);
}

template <int P>
hipError_t launch_p(int q, const Pm1Params& prm, hipStream_t stream) {
  switch (q) {
    case 1: return launch_pq<P, 1>(prm, stream);
    case 2: return launch_pq<P, 2>(prm, stream);
    case 3: return launch_pq<P, 3>(prm, stream);
    case 4: return launch_pq<P, 4>(prm, stream);
    case 5: return launch_pq<P, 5>(prm, stream);
    case 6: return launch_pq<P, 6>(prm, stream);
    case 7: return launch_pq<P, 7>(prm, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace

bool pm1_config_ok(const apt_config_t& cfg, int p, int q) {
  return p <= 7 && q <= 7 && (cfg.bm == 0 || cfg.bm == kBM) && (cfg.bn == 0 || cfg.bn == kBN);
}

// The launch's one-dimensional grid holds one workgroup per tile.
bool pm1_sizes_ok(int M, int N) {
  return (int64_t)((M + kBM - 1) / kBM) * ((N + kBN - 1) / kBN) < ((int64_t)1 << 31);
}

hipError_t launch_gemm_pm1(const GemmArgs& g, const apt_config_t&, hipStream_t stream) {
  Pm1Params prm;
  prm.g = g;
  prm.nchunks = num_chunks(g.K);
  prm.tiles_n = 0;
  switch (g.p) {
    case 1: return launch_p<1>(g.q, prm, stream);
    case 2: return launch_p<2>(g.q, prm, stream);
    case 3: return launch_p<3>(g.q, prm, stream);
    case 4: return launch_p<4>(g.q, prm, stream);
    case 5: return launch_p<5>(g.q, prm, stream);
    case 6: return launch_p<6>(g.q, prm, stream);
    case 7: return launch_p<7>(g.q, prm, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace apt
