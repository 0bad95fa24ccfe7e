// gemm_xor_inst.hip - instantiates the XOR + popcount kernels for one weight
// bit width, APT_INST_P (the build compiles this file once per width).
#include "gemm_xor.h"

namespace apt {
namespace xorpop {

template <int P>
hipError_t launch_for_p(int q, const XorParams& prm, const XorLaunch& L, hipStream_t s) {
  switch (q) {
    case 1: return launch_pq<P, 1>(prm, L, s);
    case 2: return launch_pq<P, 2>(prm, L, s);
    case 3: return launch_pq<P, 3>(prm, L, s);
    case 4: return launch_pq<P, 4>(prm, L, s);
    case 5: return launch_pq<P, 5>(prm, L, s);
    case 6: return launch_pq<P, 6>(prm, L, s);
    case 7: return launch_pq<P, 7>(prm, L, s);
    case 8: return launch_pq<P, 8>(prm, L, s);
  }
  return hipErrorInvalidValue;
}

template hipError_t launch_for_p<APT_INST_P>(int, const XorParams&, const XorLaunch&, hipStream_t);

}  // namespace xorpop
}  // namespace apt
