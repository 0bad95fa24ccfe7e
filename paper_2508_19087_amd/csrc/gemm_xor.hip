// gemm_xor.hip - launch geometry and dispatch of the XOR + popcount route;
// the kernel is in gemm_xor.h.
#include "gemm_xor.h"

namespace apt {

using xorpop::kMT;
using xorpop::kWave;
using xorpop::kWaves;
using xorpop::XorParams;

bool xor_config_ok(const apt_config_t& cfg) { return cfg.mt == 0 || cfg.mt == kMT; }

hipError_t launch_gemm_xor(const GemmArgs& g, const apt_config_t&, hipStream_t stream) {
  XorParams prm;
  prm.g = g;
  prm.nchunks = num_chunks(g.K);
  int lpr_log2 = 0;
  while ((2 << lpr_log2) <= kWave && (2 << lpr_log2) <= prm.nchunks) ++lpr_log2;
  prm.lpr_log2 = lpr_log2;
  const int rows_per_block = kWaves * (kWave >> lpr_log2);
  int grid_x = (g.N + rows_per_block - 1) / rows_per_block;
  if (grid_x > 65535) grid_x = 65535;
  const int grid_y = (g.M + kMT - 1) / kMT;
  size_t lds = (size_t)kMT * prm.nchunks * g.q * 16;
  if (lds > 64 * 1024) lds = 0;  // read the activation chunks from global memory instead
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
