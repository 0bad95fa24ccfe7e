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

namespace {

// Activation rows per block row when the config leaves it open (cold weights
// on MI355X, W2A2 and W2A4, M = 2..8, N = 4096..22016, K = 4096 and 11008).
// Eight rows per wave multiply the popcount work of a wave by eight; with few
// row groups that leaves too few waves to spread it, and one row per block
// row, which reads each weight line from L2 once per row, is faster (M = 8
// at 4096 x 4096, W2A4: 6.3 against 10.5 us).  With many row groups eight
// rows are faster from M = 4 (11008 x 4096, M = 8: 14.3 against 14.5-19 us;
// 22016 x 4096: 19.9 against 27.3 us), and from M = 2 past 2047 row groups.
// The fused form, which converts its rows in every workgroup, keeps one row
// also where the weights would take the K split (K = 11008, N = 4096: 8 rows
// of fp16 in 21.5 against 35.1 us), and from fp16, whose conversion costs
// more per row, below 2048 row groups (11008 x 4096, 8 rows: 17.8 against
// 21.8 us).
int auto_mt(int M, int groups, int rounds, int src) {
  if (M == 1) return 1;
  if (groups < 1024) return (src != xorpop::kSrcPacked || rounds < 8 || M <= 2) ? 1 : 8;
  if (groups < 2048 && (M <= 2 || src == xorpop::kSrcHalf)) return 1;
  return 8;
}

}  // namespace

XorLaunch xor_launch_shape(int M, int N, int K, int p, int q, const apt_config_t& cfg, int src) {
  XorLaunch L;
  const bool fused = src != xorpop::kSrcPacked;
  const int groups = padded_rows(N) / kRowGroup;
  const int rounds = xorpop::staged_chunks(num_chunks(K)) / xorpop::kChunkLanes;
  L.mt = cfg.mt != 0 ? cfg.mt : auto_mt(M, groups, rounds, src);
  // the fused form needs its rows' copy in LDS: one row at a time if 8 do not fit
  if (fused && cfg.mt == 0 && L.mt == 8 && act_lds_bytes_q(q, 8, num_chunks(K)) > xorpop::kMaxActLds)
    L.mt = 1;
  // waves that one wave per row group gives (row groups x block rows)
  const int spread = groups * ((M + L.mt - 1) / L.mt);
  // K split over four waves when one wave per row group would leave most
  // SIMDs without a wave (fewer than 1024 waves) and a wave would walk
  // 8 or more chunk rounds (K > 7168); measured on MI355X with cold weights:
  // 4096 x 11008 at W2A4 5.0 against 7.1 us (one token) and 14.5 against
  // 22.3 us (8 tokens), while at K = 4096 the split is 3-8% slower
  L.ksplit = cfg.waves_n != 0 ? cfg.waves_n : (spread < 1024 && rounds >= 8 ? 4 : 1);
  // one activation row: deep batches once a wave has more than one batch of
  // the plain form (8 / p chunks per lane)
  const int wave_rounds = (rounds + L.ksplit - 1) / L.ksplit;
  L.deep = L.mt == 1 && wave_rounds > std::max(1, 8 / p);
  // waves per workgroup: one while the waves alone would not give every
  // compute unit a workgroup of four (so that they spread over all compute
  // units), two in the deep form of one token, else four (cold weights on
  // MI355X: equal within noise at 4 MB, four 4-10% faster from 22 MB up and
  // with eight activation rows, two 4% faster at K = 11008 for one token).
  // The fused form converts its activation rows in every workgroup: four
  // waves share that work and there are four times fewer copies of it (one
  // token from fp16 at 4096 x 4096: 4.3 against 5.4 us).
  if (L.ksplit > 1)
    L.waves = L.ksplit;
  else
    L.waves = cfg.waves_m != 0 ? cfg.waves_m
              : fused          ? 4
              : spread < 1024  ? 1
              : (L.deep && M == 1) ? 2 : 4;
  L.grid = dim3(L.ksplit > 1 ? groups : (groups + L.waves - 1) / L.waves, (M + L.mt - 1) / L.mt);
  L.lds_bytes = act_lds_bytes_q(q, L.mt, num_chunks(K));
  L.lds = L.lds_bytes <= xorpop::kMaxActLds;
  if (!L.lds) L.lds_bytes = 0;
  L.src = src;
  return L;
}

bool xor_sizes_ok(int M, int N, int K, int p, int q, const apt_config_t& cfg) {
  const XorLaunch L = xor_launch_shape(M, N, K, p, q, cfg, xorpop::kSrcPacked);
  return L.grid.x <= 0x7fffffffu && L.grid.y <= 65535u;
}

// The fused form builds its LDS copy from the source, so the copy must fit.
bool xor_act_sizes_ok(int M, int N, int K, int p, int q, const apt_config_t& cfg, bool fp16_src) {
  const XorLaunch L =
      xor_launch_shape(M, N, K, p, q, cfg, fp16_src ? xorpop::kSrcHalf : xorpop::kSrcCodes);
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
  const XorLaunch L = xor_launch_shape(g.M, g.N, g.K, g.p, g.q, cfg, xorpop::kSrcPacked);
  prm.ksplit = L.ksplit;
  return launch_xor(prm, L, stream);
}

hipError_t launch_gemm_xor_act(const GemmArgs& g, const void* a_src, bool fp16_src,
                               uint16_t* a_scale_out, const apt_config_t& cfg, hipStream_t stream) {
  XorParams prm;
  prm.g = g;
  prm.nchunks = num_chunks(g.K);
  prm.groups = padded_rows(g.N) / kRowGroup;
  prm.a_src = a_src;
  // 16-byte loads: every row starts 16-byte aligned and holds whole vectors
  prm.a_vec = (reinterpret_cast<uintptr_t>(a_src) & 15u) == 0 && g.K % 16 == 0;
  prm.a_scale_out = fp16_src ? a_scale_out : nullptr;
  const XorLaunch L =
      xor_launch_shape(g.M, g.N, g.K, g.p, g.q, cfg, fp16_src ? xorpop::kSrcHalf : xorpop::kSrcCodes);
  if (!L.lds) return hipErrorInvalidValue;
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
