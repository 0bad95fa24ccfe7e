// gemm_xor.hip - launch geometry and dispatch of the XOR + popcount route;
// the kernel is in gemm_xor.h.
#include "gemm_xor.h"

namespace apt {

using xorpop::kMT;
using xorpop::XorParams;

bool xor_config_ok(const apt_config_t& cfg) { return cfg.mt == 0 || cfg.mt == kMT; }

hipError_t launch_gemm_xor(const GemmArgs& g, const apt_config_t&, hipStream_t stream) {
  XorParams prm;
  prm.g = g;
  prm.nchunks = num_chunks(g.K);
  const int grid_x = padded_rows(g.N) / kRowGroup;
  const int grid_y = (g.M + kMT - 1) / kMT;
  // staged activations: Q * 8 vectors of 16 bytes per chunk plus one pad vector
  size_t lds = (size_t)prm.nchunks * (g.q * kRowGroup + 1) * 16;
  // Read the activation chunks from global memory instead of staging them
  // when they do not fit, or when only one activation row is real: staging
  // would copy 8 rows and put a barrier between the two memory latencies.
  if (lds > 64 * 1024 || g.M == 1) lds = 0;
  switch (g.p) {
    case 1: return xorpop::launch_for_p<1>(g.q, prm, grid_x, grid_y, lds, stream);
    case 2: return xorpop::launch_for_p<2>(g.q, prm, grid_x, grid_y, lds, stream);
    case 3: return xorpop::launch_for_p<3>(g.q, prm, grid_x, grid_y, lds, stream);
    case 4: return xorpop::launch_for_p<4>(g.q, prm, grid_x, grid_y, lds, stream);
    case 5: return xorpop::launch_for_p<5>(g.q, prm, grid_x, grid_y, lds, stream);
    case 6: return xorpop::launch_for_p<6>(g.q, prm, grid_x, grid_y, lds, stream);
    case 7: return xorpop::launch_for_p<7>(g.q, prm, grid_x, grid_y, lds, stream);
    case 8: return xorpop::launch_for_p<8>(g.q, prm, grid_x, grid_y, lds, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace apt
