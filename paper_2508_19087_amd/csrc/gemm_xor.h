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
// Work split: a workgroup owns up to 8 activation rows (staged in LDS when they
// fit) and walks weight rows in a grid-stride loop; a group of LPR lanes shares
// one weight row, each lane taking every LPR-th 128-element chunk, and the
// per-lane sums meet in a butterfly over the group.  All 1-bit products of one
// output stay in registers (the register analogue of the paper's fragment-level
// recovery, Sec. IV-B); nothing intermediate goes to global memory.
#pragma once

#include "apt_internal.h"

namespace apt {
namespace xorpop {

constexpr int kWave = 64;
constexpr int kWaves = 4;
constexpr int kMT = 8;  // activation rows per workgroup

struct XorParams {
  GemmArgs g;
  int nchunks;
  int lpr_log2;
};

template <int P, int Q, bool kALds>
__global__ __launch_bounds__(kWave* kWaves) void gemm_xor_kernel(XorParams prm) {
  extern __shared__ uint4 a_lds[];
  const GemmArgs& g = prm.g;
  const int NC = prm.nchunks;
  const int m0 = blockIdx.y * kMT;
  const int mrows = min(kMT, g.M - m0);

  const uint4* a_src = reinterpret_cast<const uint4*>(g.a_packed) + (int64_t)m0 * NC * Q;
  if (kALds) {
    // The activation rows m0 .. m0+mrows-1 are contiguous in the packed layout.
    const int n_vec = mrows * NC * Q;
    for (int t = threadIdx.x; t < n_vec; t += blockDim.x) a_lds[t] = a_src[t];
    __syncthreads();
  }
  const uint4* a_base = kALds ? a_lds : a_src;

  const int lane = threadIdx.x % kWave;
  const int wave = blockIdx.x * kWaves + threadIdx.x / kWave;
  const int total_waves = gridDim.x * kWaves;
  const int lpr = 1 << prm.lpr_log2;
  const int rpw = kWave / lpr;
  const int group = lane >> prm.lpr_log2;
  const int sub = lane & (lpr - 1);

  const uint32_t kabq = (uint32_t)g.K * ((1u << P) - 1u) * ((1u << Q) - 1u);
  const uint4* w_all = reinterpret_cast<const uint4*>(g.w_packed);

  for (int n_base = wave * rpw; n_base < g.N; n_base += total_waves * rpw) {
    const int n = n_base + group;
    uint32_t S[kMT];
#pragma unroll
    for (int m = 0; m < kMT; ++m) S[m] = 0u;
    if (n < g.N) {
      const uint4* w_row = w_all + (int64_t)n * NC * P;
      for (int c = sub; c < NC; c += lpr) {
        uint4 wv[P];
#pragma unroll
        for (int i = 0; i < P; ++i) wv[i] = w_row[c * P + i];
#pragma unroll
        for (int m = 0; m < kMT; ++m) {
          if (m < mrows) {
            const uint4* a_chunk = a_base + ((int64_t)m * NC + c) * Q;
            uint32_t s = 0u;
#pragma unroll
            for (int j = 0; j < Q; ++j) {
              const uint4 av = a_chunk[j];
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
    }
    // Sum the group's partial counts (all lanes take part in the shuffles).
#pragma unroll
    for (int m = 0; m < kMT; ++m) {
      for (int off = lpr >> 1; off > 0; off >>= 1) S[m] += __shfl_xor(S[m], off);
    }
    if (n < g.N) {
#pragma unroll
      for (int m = 0; m < kMT; ++m) {
        if (m < mrows && (m % lpr) == sub) {
          const int mg = m0 + m;
          const int32_t c = (int32_t)(kabq - 2u * S[m]);
          const int64_t o = (int64_t)mg * g.N + n;
          if (g.c_int32) g.c_int32[o] = c;
          if (g.c_fp16) {
            float f = (float)c * __half2float(g.a_scale[mg]);
            f = f * __half2float(g.w_scale[n]);
            g.c_fp16[o] = __float2half_rn(f);
          }
        }
      }
    }
  }
}

template <int P, int Q>
inline hipError_t launch_pq(const XorParams& prm, int grid_x, int grid_y, size_t lds, hipStream_t s) {
  dim3 grid(grid_x, grid_y), block(kWave * kWaves);
  if (lds > 0)
    hipLaunchKernelGGL((gemm_xor_kernel<P, Q, true>), grid, block, lds, s, prm);
  else
    hipLaunchKernelGGL((gemm_xor_kernel<P, Q, false>), grid, block, 0, s, prm);
  return hipGetLastError();
}

// Launch for weight bits P and any activation bits; one explicit
// instantiation per P lives in gemm_xor_inst.hip (built once per P).
template <int P>
hipError_t launch_for_p(int q, const XorParams& prm, int gx, int gy, size_t lds, hipStream_t s);

}  // namespace xorpop
}  // namespace apt
