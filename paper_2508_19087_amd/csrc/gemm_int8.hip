// gemm_int8.hip - config checks, workspace size and dispatch of the
// reassembled-int8 MFMA route; the kernels are in gemm_int8.h.
#include "gemm_int8.h"

namespace apt {
namespace int8 {
namespace {

// A config names a shape by its tile and wave grid; lds_stages == 3 asks for
// the variant with explicit instruction-interleaving hints (experimental).
int shape_index(const apt_config_t& cfg) {
  for (int s = 0; s < kNumShapes; ++s)
    if (kShapes[s].bm == cfg.bm && kShapes[s].bn == cfg.bn && kShapes[s].wm == cfg.waves_m &&
        kShapes[s].wn == cfg.waves_n && kShapes[s].hints == (cfg.lds_stages == 3))
      return s;
  return -1;
}

// The tail tile is named by its size; the first shape of that size is used.
int tail_index(const apt_config_t& cfg) {
  for (int s = 0; s < kNumShapes; ++s)
    if (kShapes[s].bm == cfg.tail_bm && kShapes[s].bn == cfg.tail_bn && !kShapes[s].hints) return s;
  return -1;
}

hipError_t launch_p(int p, int shape, const Int8Params& prm, int n_count, hipStream_t stream) {
  switch (p) {
    case 1: return launch_for_p<1>(shape, prm, n_count, stream);
    case 2: return launch_for_p<2>(shape, prm, n_count, stream);
    case 3: return launch_for_p<3>(shape, prm, n_count, stream);
    case 4: return launch_for_p<4>(shape, prm, n_count, stream);
    case 5: return launch_for_p<5>(shape, prm, n_count, stream);
    case 6: return launch_for_p<6>(shape, prm, n_count, stream);
    case 7: return launch_for_p<7>(shape, prm, n_count, stream);
    case 8: return launch_for_p<8>(shape, prm, n_count, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace
}  // namespace int8

bool int8_config_ok(const apt_config_t& cfg, int N, int K) {
  if (int8::shape_index(cfg) < 0 || !(cfg.bk == 0 || cfg.bk == kChunk) || cfg.k_split < 0 ||
      cfg.k_split > 2)
    return false;
  if (cfg.split_n == 0) return cfg.k_split <= 1;
  if (cfg.k_split == 2 && num_chunks(K) < 3) return false;  // each K half needs a chunk pair
  return cfg.split_n > 0 && cfg.split_n < N && cfg.split_n % cfg.bn == 0 &&
         cfg.split_n % kRowGroup == 0 && int8::tail_index(cfg) >= 0;
}

namespace {

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// Tiles of the tail launch (0 when the config has none).
size_t tail_tiles(int M, int N, const apt_config_t& cfg) {
  if (cfg.split_n == 0) return 0;
  return (size_t)((M + cfg.tail_bm - 1) / cfg.tail_bm) *
         ((N - cfg.split_n + cfg.tail_bn - 1) / cfg.tail_bn);
}

}  // namespace

// Workspace: activation fragments, then (K-split tail) one int32 partial tile
// and one flag per tail tile.
size_t int8_workspace_bytes(int M, int N, int K, const apt_config_t& cfg) {
  size_t bytes = align256(int8::a_frag_bytes(M, K));
  if (cfg.k_split == 2) {
    const size_t tt = tail_tiles(M, N, cfg);
    bytes += align256(tt * (size_t)cfg.tail_bm * cfg.tail_bn * 4) + align256(tt * 4);
  }
  return bytes;
}

hipError_t launch_gemm_int8(const GemmArgs& g, const apt_config_t& cfg, void* workspace,
                            hipStream_t stream) {
  using namespace int8;
  const int shape = shape_index(cfg);
  if (shape < 0) return hipErrorInvalidValue;
  Int8Params prm;
  prm.g = g;
  prm.nchunks = num_chunks(g.K);
  prm.nsteps = ((prm.nchunks + 1) & ~1) * kSteps;
  prm.tiles_n = 0;
  prm.n_begin = 0;
  prm.mblocks = (g.M + 31) / 32;
  prm.a_frag = static_cast<const v4i*>(workspace);
  prm.ksplit = 1;
  prm.partial = nullptr;
  prm.flags = nullptr;
  v4i* frag = static_cast<v4i*>(workspace);
  int nflags = 0;
  if (cfg.k_split == 2) {
    uint8_t* base = static_cast<uint8_t*>(workspace) + align256(a_frag_bytes(g.M, g.K));
    const size_t tt = tail_tiles(g.M, g.N, cfg);
    prm.partial = reinterpret_cast<v4i*>(base);
    prm.flags = reinterpret_cast<int*>(base + align256(tt * (size_t)cfg.tail_bm * cfg.tail_bn * 4));
    nflags = (int)tt;
  }
  hipError_t e = hipErrorInvalidValue;
  switch (g.q) {
    case 1: e = launch_expand_for_q<1>(g.a_packed, g.M, prm.nchunks, prm.nsteps, prm.mblocks, frag, prm.flags, nflags, stream); break;
    case 2: e = launch_expand_for_q<2>(g.a_packed, g.M, prm.nchunks, prm.nsteps, prm.mblocks, frag, prm.flags, nflags, stream); break;
    case 3: e = launch_expand_for_q<3>(g.a_packed, g.M, prm.nchunks, prm.nsteps, prm.mblocks, frag, prm.flags, nflags, stream); break;
    case 4: e = launch_expand_for_q<4>(g.a_packed, g.M, prm.nchunks, prm.nsteps, prm.mblocks, frag, prm.flags, nflags, stream); break;
    case 5: e = launch_expand_for_q<5>(g.a_packed, g.M, prm.nchunks, prm.nsteps, prm.mblocks, frag, prm.flags, nflags, stream); break;
    case 6: e = launch_expand_for_q<6>(g.a_packed, g.M, prm.nchunks, prm.nsteps, prm.mblocks, frag, prm.flags, nflags, stream); break;
    case 7: e = launch_expand_for_q<7>(g.a_packed, g.M, prm.nchunks, prm.nsteps, prm.mblocks, frag, prm.flags, nflags, stream); break;
    case 8: e = launch_expand_for_q<8>(g.a_packed, g.M, prm.nchunks, prm.nsteps, prm.mblocks, frag, prm.flags, nflags, stream); break;
  }
  if (e != hipSuccess) return e;
  prm.n_begin = 0;
  if (cfg.split_n == 0) return launch_p(g.p, shape, prm, g.N, stream);
  e = launch_p(g.p, shape, prm, cfg.split_n, stream);
  if (e != hipSuccess) return e;
  prm.n_begin = cfg.split_n;
  prm.ksplit = cfg.k_split == 2 ? 2 : 1;
  return launch_p(g.p, tail_index(cfg), prm, g.N - cfg.split_n, stream);
}

}  // namespace apt
