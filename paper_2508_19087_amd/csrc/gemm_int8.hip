// gemm_int8.hip - config checks and dispatch of the reassembled-int8 MFMA
// route; the kernel is in gemm_int8.h.
#include "gemm_int8.h"

namespace apt {
namespace int8 {
namespace {

int shape_index(const apt_config_t& cfg) {
  for (int s = 0; s < kNumShapes; ++s)
    if (kShapes[s].bm == cfg.bm && kShapes[s].bn == cfg.bn && kShapes[s].wm == cfg.waves_m &&
        kShapes[s].wn == cfg.waves_n)
      return s;
  return -1;
}

}  // namespace
}  // namespace int8

using int8::shape_index;
using int8::Int8Params;

bool int8_config_ok(const apt_config_t& cfg) {
  return shape_index(cfg) >= 0 && (cfg.bk == 0 || cfg.bk == kChunk) &&
         (cfg.lds_stages == 0 || cfg.lds_stages == 2) && cfg.k_split <= 1;
}

hipError_t launch_gemm_int8(const GemmArgs& g, const apt_config_t& cfg, hipStream_t stream) {
  const int shape = shape_index(cfg);
  if (shape < 0) return hipErrorInvalidValue;
  Int8Params prm;
  prm.g = g;
  prm.nchunks = num_chunks(g.K);
  prm.tiles_n = 0;
  switch (g.p) {
    case 1: return int8::launch_for_p<1>(g.q, shape, prm, stream);
    case 2: return int8::launch_for_p<2>(g.q, shape, prm, stream);
    case 3: return int8::launch_for_p<3>(g.q, shape, prm, stream);
    case 4: return int8::launch_for_p<4>(g.q, shape, prm, stream);
    case 5: return int8::launch_for_p<5>(g.q, shape, prm, stream);
    case 6: return int8::launch_for_p<6>(g.q, shape, prm, stream);
    case 7: return int8::launch_for_p<7>(g.q, shape, prm, stream);
    case 8: return int8::launch_for_p<8>(g.q, shape, prm, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace apt
