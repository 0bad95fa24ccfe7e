// gemm_xor.h - the XOR + popcount route of the WpAq bipolar-INT GEMM for
// gfx950 (APT-LLM, arXiv 2508.19087, Sec. III-B).
//
// For bipolar bits a, w in {0,1} standing for 2a-1 and 2w-1,
// (2a-1)(2w-1) = 1 - 2 (a XOR w), so the plane product over K elements is
// Y(i,j) = K - 2 popc(W_i XOR A_j).  Recovery (Sec. III-B) then gives
//     C = sum_{i,j} 2^(i+j) Y(i,j) = K (2^p-1)(2^q-1) - 2 sum_{i,j} 2^(i+j) popc(W_i XOR A_j).
// Padding bits are zero in both operands, so they XOR to zero and the true K
// enters the constant term.
//
// Work split: a workgroup owns one 8-row group of weight rows and up to 8
// activation rows (staged in LDS when they fit).  Lane l of wave v takes weight
// row slot l mod 8 and the chunks c = (l / 8) + 8 v + 32 t, so the 8 lanes that
// share a chunk read one 128-byte line per plane.  All 1-bit products of an
// output stay in registers (the register analogue of the paper's fragment-level
// recovery, Sec. IV-B); partial sums meet through lane shuffles and one LDS
// exchange, and nothing intermediate goes to global memory.
#include "apt_internal.h"

namespace apt {
namespace xorpop {

constexpr int kWave = 64;
constexpr int kWaves = 4;
constexpr int kMT = 8;                       // activation rows per workgroup
constexpr int kSlots = kWaves * kWave / kRowGroup;  // chunk slots per workgroup (32)

struct XorParams {
  GemmArgs g;
  int nchunks;
};

template <int P, int Q, bool kALds>
__global__ __launch_bounds__(kWave* kWaves) void gemm_xor_kernel(XorParams prm) {
  extern __shared__ uint4 a_lds[];
  __shared__ uint32_t red[kWaves][kMT][kRowGroup];
  const GemmArgs& g = prm.g;
  const int NC = prm.nchunks;
  const int m0 = blockIdx.y * kMT;
  const int mrows = min(kMT, g.M - m0);
  const int n0 = blockIdx.x * kRowGroup;

  // The activation rows m0 .. m0+7 are one row group: NC * Q * 8 uint4,
  // ordered (chunk, plane, row).  In LDS each chunk's Q * 8 vectors are
  // followed by one pad vector: the 8 chunks a wave reads at once then start
  // 32 Q + 4 dwords apart and fall in different banks (without the pad, every
  // even Q puts them in the same ones).
  constexpr int kChunkVecs = Q * kRowGroup;
  const uint4* a_src = reinterpret_cast<const uint4*>(g.a_packed) + (int64_t)(m0 / kRowGroup) * NC * kChunkVecs;
  if (kALds) {
    const int n_vec = NC * kChunkVecs;
    for (int t = threadIdx.x; t < n_vec; t += blockDim.x) a_lds[t + t / kChunkVecs] = a_src[t];
    __syncthreads();
  }
  const uint4* a_base = kALds ? a_lds : a_src;
  const int a_chunk_stride = kALds ? kChunkVecs + 1 : kChunkVecs;

  const int lane = threadIdx.x % kWave;
  const int wave = threadIdx.x / kWave;
  const int slot = lane % kRowGroup;
  const int cs = lane / kRowGroup + (kWave / kRowGroup) * wave;
  const uint4* w_grp = reinterpret_cast<const uint4*>(g.w_packed) + (int64_t)blockIdx.x * NC * P * kRowGroup;

  uint32_t S[kMT];
#pragma unroll
  for (int m = 0; m < kMT; ++m) S[m] = 0u;
  for (int c = cs; c < NC; c += kSlots) {
    uint4 wv[P];
#pragma unroll
    for (int i = 0; i < P; ++i) wv[i] = w_grp[(c * P + i) * kRowGroup + slot];
#pragma unroll
    for (int m = 0; m < kMT; ++m) {
      if (m < mrows) {
        uint32_t s = 0u;
#pragma unroll
        for (int j = 0; j < Q; ++j) {
          const uint4 av = a_base[c * a_chunk_stride + j * kRowGroup + m];
#pragma unroll
          for (int i = 0; i < P; ++i) {
            uint32_t cnt = __builtin_popcount(wv[i].x ^ av.x);
            cnt += __builtin_popcount(wv[i].y ^ av.y);
            cnt += __builtin_popcount(wv[i].z ^ av.z);
            cnt += __builtin_popcount(wv[i].w ^ av.w);
            s += cnt << (i + j);
          }
        }
        S[m] += s;
      }
    }
  }
  // Sum over the 8 chunk slots of the wave (lanes with equal slot), then over
  // the 4 waves through LDS.
#pragma unroll
  for (int m = 0; m < kMT; ++m) {
    S[m] += __shfl_xor(S[m], 8);
    S[m] += __shfl_xor(S[m], 16);
    S[m] += __shfl_xor(S[m], 32);
  }
  if (lane < kRowGroup) {
#pragma unroll
    for (int m = 0; m < kMT; ++m) red[wave][m][slot] = S[m];
  }
  __syncthreads();
  if (threadIdx.x < kMT * kRowGroup) {
    const int m = threadIdx.x / kRowGroup, sl = threadIdx.x % kRowGroup;
    const int mg = m0 + m, n = n0 + sl;
    if (m < mrows && n < g.N) {
      uint32_t tot = 0u;
#pragma unroll
      for (int v = 0; v < kWaves; ++v) tot += red[v][m][sl];
      const uint32_t kabq = (uint32_t)g.K * ((1u << P) - 1u) * ((1u << Q) - 1u);
      const int32_t c = (int32_t)(kabq - 2u * tot);
      const int64_t o = (int64_t)mg * g.N + n;
      if (g.c_int32) g.c_int32[o] = c;
      if (g.c_fp16) {
        float f;
        if (g.a_zero) {
          const float sw = __half2float(g.w_scale[n]), zw = __half2float(g.w_zero[n]);
          f = affine_value(c, __half2float(g.a_scale[mg]), sw, zw, (float)g.a_rowsum[mg],
                           __half2float(g.a_zero[mg]),
                           sw * (float)g.w_rowsum[n] + (float)g.K * zw);
        } else {
          f = (float)c * __half2float(g.a_scale[mg]);
          f = f * __half2float(g.w_scale[n]);
        }
        g.c_fp16[o] = __float2half_rn(f);
      }
    }
  }
}

template <int P, int Q>
inline hipError_t launch_pq(const XorParams& prm, int grid_x, int grid_y, size_t lds, hipStream_t s) {
  dim3 grid(grid_x, grid_y), block(kWave * kWaves);
  if (lds > 0) return launch_kernel(gemm_xor_kernel<P, Q, true>, grid, block, lds, s, prm);
  return launch_kernel(gemm_xor_kernel<P, Q, false>, grid, block, 0, s, prm);
}

// Launch for weight bits P and any activation bits; one explicit
// instantiation per P lives in gemm_xor_inst.hip (built once per P).
template <int P>
hipError_t launch_for_p(int q, const XorParams& prm, int gx, int gy, size_t lds, hipStream_t s);

}  // namespace xorpop
}  // namespace apt
