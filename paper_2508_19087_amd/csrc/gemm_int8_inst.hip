// gemm_int8_inst.hip - instantiates the reassembled MFMA kernels for one bit
// width, APT_INST_P: the main kernel for weight width APT_INST_P and the
// activation expansion for activation width APT_INST_P, with int8 operands
// and, for widths of at most 2 bits, FP4 operands (the build compiles this
// file once per width).
#include "gemm_int8.h"

namespace apt {
namespace int8 {

template <int P>
hipError_t launch_for_p(bool fp4, int shape, const Int8Params& prm, int grid, hipStream_t stream) {
  if constexpr (P <= 2) {
    if (fp4) return launch_p_shape<P, 1>(shape, prm, grid, stream);
  } else {
    if (fp4) return hipErrorInvalidValue;
  }
  return launch_p_shape<P, 0>(shape, prm, grid, stream);
}

template <int P>
hipError_t launch_pair_for_p(bool fp4, int sa, const Int8Params& pa, int ga, int sb,
                             const Int8Params& pb, int gb, hipStream_t stream) {
  if constexpr (P <= 2) {
    if (fp4) return launch_p_pair<P, 1>(sa, pa, ga, sb, pb, gb, stream);
  } else {
    if (fp4) return hipErrorInvalidValue;
  }
  return launch_p_pair<P, 0>(sa, pa, ga, sb, pb, gb, stream);
}

template <int Q, int F>
hipError_t launch_expand(const uint32_t* a_packed, int M, int nchunks, int nsteps, int mblocks,
                         v4i* out, int* counters, int ncounters, hipStream_t stream) {
  int64_t threads = (int64_t)mblocks * 32 * (nsteps / Fmt<F>::kSteps) * kWordsPerPlane;
  if (threads < ncounters) threads = ncounters;
  const int blocks = (int)((threads + 255) / 256);
  hipLaunchKernelGGL((expand_a_kernel<Q, F>), dim3(blocks), dim3(256), 0, stream, a_packed, M,
                     nchunks, nsteps, mblocks, out, counters, ncounters);
  return hipGetLastError();
}

template <int Q>
hipError_t launch_expand_for_q(bool fp4, const uint32_t* a_packed, int M, int nchunks, int nsteps,
                               int mblocks, v4i* out, int* counters, int ncounters,
                               hipStream_t stream) {
  if constexpr (Q <= 2) {
    if (fp4)
      return launch_expand<Q, 1>(a_packed, M, nchunks, nsteps, mblocks, out, counters, ncounters,
                                 stream);
  } else {
    if (fp4) return hipErrorInvalidValue;
  }
  return launch_expand<Q, 0>(a_packed, M, nchunks, nsteps, mblocks, out, counters, ncounters,
                             stream);
}

template hipError_t launch_for_p<APT_INST_P>(bool, int, const Int8Params&, int, hipStream_t);
template hipError_t launch_pair_for_p<APT_INST_P>(bool, int, const Int8Params&, int, int,
                                                   const Int8Params&, int, hipStream_t);
template hipError_t launch_expand_for_q<APT_INST_P>(bool, const uint32_t*, int, int, int, int,
                                                     v4i*, int*, int, hipStream_t);

}  // namespace int8
}  // namespace apt
