// gemm_int8_inst.hip - instantiates the reassembled-int8 MFMA kernels for one
// weight bit width, APT_INST_P (the build compiles this file once per width).
#include "gemm_int8.h"

namespace apt {
namespace int8 {

template <int P>
hipError_t launch_for_p(int q, int shape, const Int8Params& prm, hipStream_t stream) {
  switch (q) {
    case 1: return launch_pq<P, 1>(shape, prm, stream);
    case 2: return launch_pq<P, 2>(shape, prm, stream);
    case 3: return launch_pq<P, 3>(shape, prm, stream);
    case 4: return launch_pq<P, 4>(shape, prm, stream);
    case 5: return launch_pq<P, 5>(shape, prm, stream);
    case 6: return launch_pq<P, 6>(shape, prm, stream);
    case 7: return launch_pq<P, 7>(shape, prm, stream);
    case 8: return launch_pq<P, 8>(shape, prm, stream);
  }
  return hipErrorInvalidValue;
}

template hipError_t launch_for_p<APT_INST_P>(int, int, const Int8Params&, hipStream_t);

}  // namespace int8
}  // namespace apt
