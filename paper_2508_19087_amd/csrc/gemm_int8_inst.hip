// gemm_int8_inst.hip - instantiates the reassembled MFMA kernels for one bit
// width, APT_INST_P: the main kernel for weight width APT_INST_P and the
// activation expansion for activation width APT_INST_P, with int8 operands
// and, where the widths allow, FP4 weights with FP4 or FP8 activations, FP6
// operands and FP8 operands (the build compiles this file once per width).
#include "gemm_int8.h"

namespace apt {
namespace int8 {

template <int P>
hipError_t launch_for_p(int fmt, int shape, const Int8Params& prm, int grid, hipStream_t stream) {
  if (fmt == 0) return launch_p_shape<P, 0>(shape, prm, grid, stream);
  if constexpr (P <= 2) {
    if (fmt == 1) return launch_p_shape<P, 1>(shape, prm, grid, stream);
    if (fmt == 2) return launch_p_shape<P, 2>(shape, prm, grid, stream);
  }
  if constexpr (P <= 3) {
    if (fmt == 3) return launch_p_shape<P, 3>(shape, prm, grid, stream);
  }
  if constexpr (P <= 4) {
    if (fmt == 4) return launch_p_shape<P, 4>(shape, prm, grid, stream);
  }
  return hipErrorInvalidValue;
}

template <int P>
hipError_t launch_pair_for_p(int fmt, int sa, const Int8Params& pa, int ga, int sb,
                             const Int8Params& pb, int gb, hipStream_t stream) {
  if (fmt == 0) return launch_p_pair<P, 0>(sa, pa, ga, sb, pb, gb, stream);
  if constexpr (P <= 2) {
    if (fmt == 1) return launch_p_pair<P, 1>(sa, pa, ga, sb, pb, gb, stream);
    if (fmt == 2) return launch_p_pair<P, 2>(sa, pa, ga, sb, pb, gb, stream);
  }
  if constexpr (P <= 3) {
    if (fmt == 3) return launch_p_pair<P, 3>(sa, pa, ga, sb, pb, gb, stream);
  }
  if constexpr (P <= 4) {
    if (fmt == 4) return launch_p_pair<P, 4>(sa, pa, ga, sb, pb, gb, stream);
  }
  return hipErrorInvalidValue;
}

template <int Q, int F>
hipError_t launch_expand(const uint32_t* a_packed, int M, int nchunks, int nsteps, int mblocks,
                         v4i* out, int* counters, int ncounters, hipStream_t stream) {
  // x: (row, word) pairs of one chunk; y: the chunks (an even count)
  const int blocks = (mblocks * 32 * kWordsPerPlane + 255) / 256;
  return launch_kernel(expand_a_kernel<Q, F>, dim3(blocks, nsteps / Fmt<F>::kSteps), dim3(256), 0,
                       stream, a_packed, M, nchunks, nsteps, mblocks, out, counters, ncounters);
}

template <int Q>
hipError_t launch_expand_for_q(int fmt, const uint32_t* a_packed, int M, int nchunks, int nsteps,
                               int mblocks, v4i* out, int* counters, int ncounters,
                               hipStream_t stream) {
  if (fmt == 0)
    return launch_expand<Q, 0>(a_packed, M, nchunks, nsteps, mblocks, out, counters, ncounters,
                               stream);
  if constexpr (Q <= 2) {
    if (fmt == 1)
      return launch_expand<Q, 1>(a_packed, M, nchunks, nsteps, mblocks, out, counters, ncounters,
                                 stream);
  }
  if constexpr (Q >= 3 && Q <= 4) {
    if (fmt == 2)
      return launch_expand<Q, 2>(a_packed, M, nchunks, nsteps, mblocks, out, counters, ncounters,
                                 stream);
  }
  if constexpr (Q <= 3) {
    if (fmt == 3)
      return launch_expand<Q, 3>(a_packed, M, nchunks, nsteps, mblocks, out, counters, ncounters,
                                 stream);
  }
  if constexpr (Q <= 4) {
    if (fmt == 4)
      return launch_expand<Q, 4>(a_packed, M, nchunks, nsteps, mblocks, out, counters, ncounters,
                                 stream);
  }
  return hipErrorInvalidValue;
}

template hipError_t launch_for_p<APT_INST_P>(int, int, const Int8Params&, int, hipStream_t);
template hipError_t launch_pair_for_p<APT_INST_P>(int, int, const Int8Params&, int, int,
                                                   const Int8Params&, int, hipStream_t);
template hipError_t launch_expand_for_q<APT_INST_P>(int, const uint32_t*, int, int, int, int,
                                                     v4i*, int*, int, hipStream_t);

}  // namespace int8
}  // namespace apt
