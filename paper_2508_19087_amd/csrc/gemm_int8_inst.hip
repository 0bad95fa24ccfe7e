// gemm_int8_inst.hip - instantiates the reassembled-int8 MFMA kernels for one
// bit width, APT_INST_P: the main kernel for weight width APT_INST_P and the
// activation expansion for activation width APT_INST_P (the build compiles
// this file once per width).
#include "gemm_int8.h"

namespace apt {
namespace int8 {

template <int P>
hipError_t launch_for_p(int shape, const Int8Params& prm, int grid, hipStream_t stream) {
  return launch_p_shape<P>(shape, prm, grid, stream);
}

template <int P>
hipError_t launch_pair_for_p(int sa, const Int8Params& pa, int ga, int sb, const Int8Params& pb,
                             int gb, hipStream_t stream) {
  return launch_p_pair<P>(sa, pa, ga, sb, pb, gb, stream);
}

template <int Q>
hipError_t launch_expand_for_q(const uint32_t* a_packed, int M, int nchunks, int nsteps,
                               int mblocks, v4i* out, int* counters, int ncounters,
                               hipStream_t stream) {
  int64_t threads = (int64_t)mblocks * 32 * (nsteps / kSteps) * kWordsPerPlane;
  if (threads < ncounters) threads = ncounters;
  const int blocks = (int)((threads + 255) / 256);
  hipLaunchKernelGGL(expand_a_kernel<Q>, dim3(blocks), dim3(256), 0, stream, a_packed, M, nchunks,
                     nsteps, mblocks, out, counters, ncounters);
  return hipGetLastError();
}

template hipError_t launch_for_p<APT_INST_P>(int, const Int8Params&, int, hipStream_t);
template hipError_t launch_pair_for_p<APT_INST_P>(int, const Int8Params&, int, int,
                                                   const Int8Params&, int, hipStream_t);
template hipError_t launch_expand_for_q<APT_INST_P>(const uint32_t*, int, int, int, int, v4i*,
                                                     int*, int, hipStream_t);

}  // namespace int8
}  // namespace apt
