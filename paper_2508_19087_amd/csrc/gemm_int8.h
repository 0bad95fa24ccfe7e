// gemm_int8.h - the reassembled-int8 MFMA route of the WpAq bipolar-INT
// GEMM for gfx950 (APT-LLM, arXiv 2508.19087, Sec. III-B and IV-B).
//
// Each workgroup owns one BM x BN output tile and every bit-plane pair of it,
// as the paper's recovery-oriented scheduling does (Sec. IV-B).  K advances
// one 128-element chunk per pipeline step:
//   1. global -> registers: the packed planes of the tile's A rows (q planes)
//      and W rows (p planes), prefetched one step ahead;
//   2. registers -> LDS: each row's planes are merged back into one byte per
//      element (reassemble.h) and written to a double-buffered LDS tile;
//   3. LDS -> MFMA: v_mfma_i32_32x32x32_i8 over the reassembled bytes.
// Recombination therefore happens before the multiply; the paper's Sec. III-B
// sum over plane products is the same number by distributivity.
//
// Operand bytes are y = u (b <= 7) or u - 128 (b == 8) with bipolar value
// v = 2y + c.  Expanding sum_k v_a v_w over the real K gives the epilogue
//   C = 4 D - 4 (K_pad - K) y_pad,a y_pad,w + c_w R_a[m] + c_a R_w[n] - c_a c_w K,
// where D is the MFMA sum over K_pad, y_pad the operand byte of a padding
// element, and R the row sums of bipolar values from the packers.  The
// arithmetic is done modulo 2^32; the true C fits in int32 (checked by the
// host), so the wrapped result is exact.
#pragma once

#include "apt_internal.h"
#include "reassemble.h"

namespace apt {
namespace int8 {

constexpr int kWave = 64;
constexpr int kRowBytes = kChunk + 16;  // padded LDS row: 128 operand bytes + 16

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

struct Int8Params {
  GemmArgs g;
  int nchunks;
  int tiles_n;
};

// Staging of one operand: ROWS rows of a tile, each split into SPLIT items of
// 128/SPLIT elements (4/SPLIT words per plane).
template <int B, int ROWS, int SPLIT, int T>
struct Stage {
  static constexpr int kWpi = kWordsPerPlane / SPLIT;
  static constexpr int kItems = ROWS * SPLIT / T;
  static_assert(ROWS * SPLIT % T == 0, "items must divide evenly");
  uint32_t raw[kItems][B][kWpi];

  __device__ __forceinline__ void load(const uint32_t* __restrict__ packed, int row0, int rows,
                                       int nchunks, int chunk, int tid) {
#pragma unroll
    for (int it = 0; it < kItems; ++it) {
      const int item = tid + T * it;
      const int r = row0 + item / SPLIT;
      const int sub = item % SPLIT;
      if (r < rows) {
        const uint32_t* src = packed + (((int64_t)r * nchunks + chunk) * B) * kWordsPerPlane + sub * kWpi;
#pragma unroll
        for (int i = 0; i < B; ++i) {
          if (kWpi == 4) {
            uint4 v = *reinterpret_cast<const uint4*>(src + i * kWordsPerPlane);
            raw[it][i][0] = v.x; raw[it][i][1] = v.y; raw[it][i][2] = v.z; raw[it][i][3] = v.w;
          } else if (kWpi == 2) {
            uint2 v = *reinterpret_cast<const uint2*>(src + i * kWordsPerPlane);
            raw[it][i][0] = v.x; raw[it][i][1] = v.y;
          } else {
            raw[it][i][0] = src[i * kWordsPerPlane];
          }
        }
      } else {
#pragma unroll
        for (int i = 0; i < B; ++i)
#pragma unroll
          for (int w = 0; w < kWpi; ++w) raw[it][i][w] = 0u;
      }
    }
  }

  __device__ __forceinline__ void store(uint8_t* lds_tile, int tid) const {
#pragma unroll
    for (int it = 0; it < kItems; ++it) {
      const int item = tid + T * it;
      const int r = item / SPLIT;
      const int sub = item % SPLIT;
      uint8_t* dst = lds_tile + r * kRowBytes + sub * kWpi * 32;
#pragma unroll
      for (int w = 0; w < kWpi; ++w) {
        uint32_t pw[B];
#pragma unroll
        for (int i = 0; i < B; ++i) pw[i] = raw[it][i][w];
        uint32_t o[8];
        reassemble_word<B>(pw, o);
        uint4* d4 = reinterpret_cast<uint4*>(dst + w * 32);
        d4[0] = make_uint4(o[0], o[1], o[2], o[3]);
        d4[1] = make_uint4(o[4], o[5], o[6], o[7]);
      }
    }
  }
};

template <int P, int Q, int BM, int BN, int WM, int WN, int SPLIT>
__global__ __launch_bounds__(WM* WN* kWave) void gemm_int8_kernel(Int8Params prm) {
  constexpr int T = WM * WN * kWave;
  constexpr int WTM = BM / WM, WTN = BN / WN;  // wave tile
  constexpr int FM = WTM / 32, FN = WTN / 32;  // 32x32 MFMA tiles per wave
  constexpr int kStageBytes = (BM + BN) * kRowBytes;
  static_assert(FM >= 1 && FN >= 1, "wave tile too small");
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];

  const GemmArgs& g = prm.g;
  const int NC = prm.nchunks;
  const int tid = threadIdx.x;
  const int lane = tid % kWave;
  const int wave = tid / kWave;
  const int wm = wave / WN, wn = wave % WN;

  const int tile = blockIdx.x;
  const int tm = tile / prm.tiles_n, tn = tile % prm.tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;

  Stage<Q, BM, SPLIT, T> sa;
  Stage<P, BN, SPLIT, T> sw;

  v16i acc[FM][FN];
#pragma unroll
  for (int a = 0; a < FM; ++a)
#pragma unroll
    for (int b = 0; b < FN; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][b][v] = 0;

  sa.load(g.a_packed, m0, g.M, NC, 0, tid);
  sw.load(g.w_packed, n0, g.N, NC, 0, tid);
  sa.store(lds, tid);
  sw.store(lds + BM * kRowBytes, tid);
  __syncthreads();

  const int lrow = lane % 32;
  const int lk = (lane / 32) * 16;
  for (int c = 0; c < NC; ++c) {
    const bool more = c + 1 < NC;
    if (more) {
      sa.load(g.a_packed, m0, g.M, NC, c + 1, tid);
      sw.load(g.w_packed, n0, g.N, NC, c + 1, tid);
    }
    const uint8_t* st = lds + (c & 1) * kStageBytes;
    const uint8_t* a_t = st + (wm * WTM + lrow) * kRowBytes + lk;
    const uint8_t* w_t = st + (BM + wn * WTN + lrow) * kRowBytes + lk;
#pragma unroll
    for (int ks = 0; ks < kChunk / 32; ++ks) {
      v4i af[FM], bf[FN];
#pragma unroll
      for (int a = 0; a < FM; ++a)
        af[a] = *reinterpret_cast<const v4i*>(a_t + a * 32 * kRowBytes + ks * 32);
#pragma unroll
      for (int b = 0; b < FN; ++b)
        bf[b] = *reinterpret_cast<const v4i*>(w_t + b * 32 * kRowBytes + ks * 32);
#pragma unroll
      for (int a = 0; a < FM; ++a)
#pragma unroll
        for (int b = 0; b < FN; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[a], bf[b], acc[a][b], 0, 0, 0);
    }
    if (more) {
      uint8_t* nx = lds + ((c + 1) & 1) * kStageBytes;
      sa.store(nx, tid);
      sw.store(nx + BM * kRowBytes, tid);
    }
    __syncthreads();
  }

  // Epilogue: affine correction, optional fp16 scaling, stores.
  constexpr int ca = operand_offset<Q>(), cw = operand_offset<P>();
  const uint32_t pad_term =
      4u * (uint32_t)(NC * kChunk - g.K) * (uint32_t)(operand_pad<Q>() * operand_pad<P>());
  const uint32_t const_term = (uint32_t)(ca * cw) * (uint32_t)g.K + pad_term;
#pragma unroll
  for (int b = 0; b < FN; ++b) {
    const int n = n0 + wn * WTN + b * 32 + lrow;
    if (n >= g.N) continue;
    const uint32_t wterm = (uint32_t)ca * (uint32_t)g.w_rowsum[n];
    const float sw_f = g.c_fp16 ? __half2float(g.w_scale[n]) : 0.f;
#pragma unroll
    for (int a = 0; a < FM; ++a) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int m = m0 + wm * WTM + a * 32 + (v / 4) * 8 + (lane / 32) * 4 + (v % 4);
        if (m < g.M) {
          const uint32_t d = (uint32_t)acc[a][b][v];
          const uint32_t cval = 4u * d + (uint32_t)cw * (uint32_t)g.a_rowsum[m] + wterm - const_term;
          const int64_t o = (int64_t)m * g.N + n;
          if (g.c_int32) g.c_int32[o] = (int32_t)cval;
          if (g.c_fp16) {
            float f = (float)(int32_t)cval * __half2float(g.a_scale[m]);
            g.c_fp16[o] = __float2half_rn(f * sw_f);
          }
        }
      }
    }
  }
}

struct TileShape {
  int bm, bn, wm, wn, split;
};
constexpr TileShape kShapes[] = {
    {128, 128, 2, 2, 2},
    {256, 128, 2, 2, 2},
    {256, 256, 2, 2, 1},
};
constexpr int kNumShapes = sizeof(kShapes) / sizeof(kShapes[0]);

template <int P, int Q, int S>
hipError_t launch_shape(const Int8Params& prm0, hipStream_t stream) {
  constexpr TileShape sh = kShapes[S];
  Int8Params prm = prm0;
  prm.tiles_n = (prm.g.N + sh.bn - 1) / sh.bn;
  const int tiles_m = (prm.g.M + sh.bm - 1) / sh.bm;
  const size_t lds = 2 * (size_t)(sh.bm + sh.bn) * kRowBytes;
  auto kern = gemm_int8_kernel<P, Q, sh.bm, sh.bn, sh.wm, sh.wn, sh.split>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(tiles_m * prm.tiles_n), dim3(sh.wm * sh.wn * kWave), lds, stream, prm);
  return hipGetLastError();
}

template <int P, int Q>
inline hipError_t launch_pq(int shape, const Int8Params& prm, hipStream_t stream) {
  switch (shape) {
    case 0: return launch_shape<P, Q, 0>(prm, stream);
    case 1: return launch_shape<P, Q, 1>(prm, stream);
    case 2: return launch_shape<P, Q, 2>(prm, stream);
  }
  return hipErrorInvalidValue;
}

// Launch for weight bits P and any activation bits; one explicit
// instantiation per P lives in gemm_int8_inst.hip (built once per P).
template <int P>
hipError_t launch_for_p(int q, int shape, const Int8Params& prm, hipStream_t stream);

}  // namespace int8
}  // namespace apt
