// gemm_xor.hip - launch geometry and dispatch of the XOR + popcount route;
// the kernel is in gemm_xor.h.
#include <algorithm>

#include "gemm_xor.h"

namespace apt {

using xorpop::XorLaunch;
using xorpop::XorParams;

// Config fields of the XOR route: mt = activation rows per block row (0:
// 1 when M = 1, else 8); waves_m = waves per workgroup, each owning one 8-row
// group of weight rows (0: chosen below, or 1, 2 or 4); waves_n = K split, the
// waves of a workgroup sharing one row group (0: chosen below, 1 = none, or 2
// or 4; with 2 or 4, waves_m is ignored).
bool xor_config_ok(const apt_config_t& cfg) {
  auto w_ok = [](int w) { return w == 0 || w == 1 || w == 2 || w == 4; };
  return (cfg.mt == 0 || cfg.mt == 1 || cfg.mt == 8) && w_ok(cfg.waves_m) && w_ok(cfg.waves_n);
}

namespace {

size_t act_lds_bytes_q(int q, int mt, int nchunks) {
  const int per = mt == 8 ? q * kRowGroup + 1 : q;
  return (size_t)xorpop::staged_chunks(nchunks) * per * 16;
}

}  // namespace

XorLaunch xor_launch_shape(int M, int N, int K, int p, int q, const apt_config_t& cfg) {
  XorLaunch L;
  L.mt = cfg.mt != 0 ? cfg.mt : (M == 1 ? 1 : 8);
  const int groups = padded_rows(N) / kRowGroup;
  const int rounds = xorpop::staged_chunks(num_chunks(K)) / xorpop::kChunkLanes;
  // K split over four waves when one wave per row group would leave most
  // SIMDs without a wave (fewer than 1024 row groups) and a wave would walk
  // 8 or more chunk rounds (K > 7168); measured on MI355X with cold weights:
  // 4096 x 11008 at W2A4 5.0 against 7.1 us (one token) and 14.5 against
  // 22.3 us (8 tokens), while at K = 4096 the split is 3-8% slower
  L.ksplit = cfg.waves_n != 0 ? cfg.waves_n : (groups < 1024 && rounds >= 8 ? 4 : 1);
  // one activation row: deep batches once a wave has more than one batch of
  // the plain form (8 / p chunks per lane)
  const int wave_rounds = (rounds + L.ksplit - 1) / L.ksplit;
  L.deep = L.mt == 1 && wave_rounds > std::max(1, 8 / p);
  // waves per workgroup: one while the row groups alone would not give every
  // compute unit a workgroup of four (so that they spread over all compute
  // units), two in the deep form, else four (cold weights on MI355X: equal
  // within noise at 4 MB, four 4-10% faster from 22 MB up and with eight
  // activation rows, two 4% faster at K = 11008)
  if (L.ksplit > 1)
    L.waves = L.ksplit;
  else
    L.waves = cfg.waves_m != 0 ? cfg.waves_m : groups < 1024 ? 1 : (L.deep ? 2 : 4);
  L.grid = dim3(L.ksplit > 1 ? groups : (groups + L.waves - 1) / L.waves, (M + L.mt - 1) / L.mt);
  L.lds_bytes = act_lds_bytes_q(q, L.mt, num_chunks(K));
  L.lds = L.lds_bytes <= xorpop::kMaxActLds;
  if (!L.lds) L.lds_bytes = 0;
  L.src = xorpop::kSrcPacked;
  return L;
}

bool xor_sizes_ok(int M, int N, int K, int p, int q, const apt_config_t& cfg) {
  const XorLaunch L = xor_launch_shape(M, N, K, p, q, cfg);
  return L.grid.x <= 0x7fffffffu && L.grid.y <= 65535u;
}

// The fused form runs one activation row per block row and builds its LDS
// copy from the source: mt must resolve to 1 and the copy must fit in LDS.
bool xor_act_config_ok(const apt_config_t& cfg) { return xor_config_ok(cfg) && cfg.mt != 8; }

bool xor_act_sizes_ok(int M, int N, int K, int p, int q, const apt_config_t& cfg) {
  apt_config_t c = cfg;
  c.mt = 1;
  const XorLaunch L = xor_launch_shape(M, N, K, p, q, c);
  return L.lds && L.grid.x <= 0x7fffffffu && L.grid.y <= 65535u;
}

namespace {

hipError_t launch_xor(const XorParams& prm, const XorLaunch& L, hipStream_t stream);

}  // namespace

hipError_t launch_gemm_xor(const GemmArgs& g, const apt_config_t& cfg, hipStream_t stream) {
  XorParams prm;
  prm.g = g;
  prm.nchunks = num_chunks(g.K);
  prm.groups = padded_rows(g.N) / kRowGroup;
  prm.a_src = nullptr;
  prm.a_vec = 0;
  prm.a_scale_out = nullptr;
  const XorLaunch L = xor_launch_shape(g.M, g.N, g.K, g.p, g.q, cfg);
  prm.ksplit = L.ksplit;
  return launch_xor(prm, L, stream);
}

hipError_t launch_gemm_xor_act(const GemmArgs& g, const void* a_src, bool fp16_src,
                               uint16_t* a_scale_out, const apt_config_t& cfg, hipStream_t stream) {
  apt_config_t c = cfg;
  c.mt = 1;
  XorParams prm;
  prm.g = g;
  prm.nchunks = num_chunks(g.K);
  prm.groups = padded_rows(g.N) / kRowGroup;
  prm.a_src = a_src;
  // 16-byte loads: every row starts 16-byte aligned and holds whole vectors
  prm.a_vec = (reinterpret_cast<uintptr_t>(a_src) & 15u) == 0 && g.K % 16 == 0;
  prm.a_scale_out = fp16_src ? a_scale_out : nullptr;
  XorLaunch L = xor_launch_shape(g.M, g.N, g.K, g.p, g.q, c);
  if (!L.lds) return hipErrorInvalidValue;
  L.src = fp16_src ? xorpop::kSrcHalf : xorpop::kSrcCodes;
  prm.ksplit = L.ksplit;
  return launch_xor(prm, L, stream);
}

namespace {

hipError_t launch_xor(const XorParams& prm, const XorLaunch& L, hipStream_t stream) {
  const GemmArgs& g = prm.g;
  switch (g.p) {
    case 1: return xorpop::launch_for_p<1>(g.q, prm, L, stream);
    case 2: return xorpop::launch_for_p<2>(g.q, prm, L, stream);
    case 3: return xorpop::launch_for_p<3>(g.q, prm, L, stream);
    case 4: return xorpop::launch_for_p<4>(g.q, prm, L, stream);
    case 5: return xorpop::launch_for_p<5>(g.q, prm, L, stream);
    case 6: return xorpop::launch_for_p<6>(g.q, prm, L, stream);
    case 7: return xorpop::launch_for_p<7>(g.q, prm, L, stream);
    case 8: return xorpop::launch_for_p<8>(g.q, prm, L, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace

}  // namespace apt
