// gemm_int8.hip - config checks, workspace size and dispatch of the
// reassembled-int8 MFMA route; the kernels are in gemm_int8.h.
#include <algorithm>

#include "gemm_int8.h"

namespace apt {
namespace int8 {
namespace {

// A config names a shape by its tile and wave grid; the weight ring is always
// kStages deep (lds_stages 0 or kStages).
int shape_index(const apt_config_t& cfg) {
  if (cfg.lds_stages != 0 && cfg.lds_stages != kStages) return -1;
  for (int s = 0; s < kNumShapes; ++s)
    if (kShapes[s].bm == cfg.bm && kShapes[s].bn == cfg.bn && kShapes[s].wm == cfg.waves_m &&
        kShapes[s].wn == cfg.waves_n)
      return s;
  return -1;
}

hipError_t launch_p(int p, int fmt, int shape, const Int8Params& prm, int grid,
                    hipStream_t stream) {
  switch (p) {
    case 1: return launch_for_p<1>(fmt, shape, prm, grid, stream);
    case 2: return launch_for_p<2>(fmt, shape, prm, grid, stream);
    case 3: return launch_for_p<3>(fmt, shape, prm, grid, stream);
    case 4: return launch_for_p<4>(fmt, shape, prm, grid, stream);
    case 5: return launch_for_p<5>(fmt, shape, prm, grid, stream);
    case 6: return launch_for_p<6>(fmt, shape, prm, grid, stream);
    case 7: return launch_for_p<7>(fmt, shape, prm, grid, stream);
    case 8: return launch_for_p<8>(fmt, shape, prm, grid, stream);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_pair(int p, int fmt, int sa, const Int8Params& pa, int ga, int sb,
                       const Int8Params& pb, int gb, hipStream_t stream) {
  switch (p) {
    case 1: return launch_pair_for_p<1>(fmt, sa, pa, ga, sb, pb, gb, stream);
    case 2: return launch_pair_for_p<2>(fmt, sa, pa, ga, sb, pb, gb, stream);
    case 3: return launch_pair_for_p<3>(fmt, sa, pa, ga, sb, pb, gb, stream);
    case 4: return launch_pair_for_p<4>(fmt, sa, pa, ga, sb, pb, gb, stream);
    case 5: return launch_pair_for_p<5>(fmt, sa, pa, ga, sb, pb, gb, stream);
    case 6: return launch_pair_for_p<6>(fmt, sa, pa, ga, sb, pb, gb, stream);
    case 7: return launch_pair_for_p<7>(fmt, sa, pa, ga, sb, pb, gb, stream);
    case 8: return launch_pair_for_p<8>(fmt, sa, pa, ga, sb, pb, gb, stream);
  }
  return hipErrorInvalidValue;
}

// Operand format of a config (the F of the kernels): int8 for the int8 route;
// for the FP4 route FP4 activations when q <= 2, FP8 activations otherwise;
// FP6 and FP8 operands for the FP6 and FP8 routes.
int operand_format(const apt_config_t& cfg, int q) {
  if (cfg.route == APT_ROUTE_FP8_MFMA) return 4;
  if (cfg.route == APT_ROUTE_FP6_MFMA) return 3;
  if (cfg.route != APT_ROUTE_FP4_MFMA) return 0;
  return q <= 2 ? 1 : 2;
}

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// The work decomposition of one launch: shape `shape` over output columns
// [n_begin, n_begin + n_cols) with `grid` persistent workgroups (see
// gemm_int8_kernel).
struct Plan {
  int shape, n_begin, tiles_n, tiles, grid, dp_tiles, sk_tiles, sk_pairs, sk_grid;
  size_t partial_bytes, counter_bytes;
};

// Parts per stream-K tile.  When the leftover tiles are more than half of
// the compute units the grid covers but no more than all of them, each stays
// whole and simply extends one workgroup's chunk stream, one per compute unit:
// that saves the launch and pipeline start of a second round without any
// partial traffic (MI355X, interleaved runs: W4A4 2048x11008x4096, 176
// leftover 256x128 tiles on 512 workgroups, 85.4 us whole against 88.0 us
// for one workgroup per tile and 98.0 us in two parts; W2A4 1024x11008x4096,
// 176 leftover 128x128 tiles, 51.5 against 54.0 us).  Otherwise about two
// parts per tile: more parts only add partial traffic.
int64_t sk_parts(const TileShape& sh, int grid, int sk_tiles) {
  const int per_cu = sh.wm * sh.wn <= 4 ? 2 : 1;  // resident workgroups per compute unit
  const int64_t units = std::max(1, grid / per_cu);
  return 2 * (int64_t)sk_tiles > units && sk_tiles <= units ? 1 : 2;
}

Plan make_plan(int M, int K, int shape, int n_begin, int n_cols, int grid) {
  Plan pl;
  pl.shape = shape;
  const TileShape& sh = kShapes[shape];
  pl.n_begin = n_begin;
  pl.tiles_n = (n_cols + sh.bn - 1) / sh.bn;
  pl.tiles = ((M + sh.bm - 1) / sh.bm) * pl.tiles_n;
  const int pairs = ((num_chunks(K) + 1) & ~1) / 2;
  const int64_t units = (int64_t)pl.tiles * pairs;
  pl.grid = grid == 0 ? pl.tiles : (int)std::min<int64_t>(grid, units);
  pl.dp_tiles = pl.tiles / pl.grid;
  pl.sk_tiles = pl.tiles - pl.dp_tiles * pl.grid;
  pl.sk_pairs = pl.sk_tiles * pairs;
  pl.sk_grid = (int)std::min<int64_t>(pl.grid, std::max<int64_t>(1, sk_parts(sh, pl.grid, pl.sk_tiles) *
                                                                    (int64_t)pl.sk_tiles));
  // one workgroup per leftover tile (sk_grid == sk_tiles): every part is a
  // whole tile, so no partial tile or counter is ever used
  const bool shared = pl.sk_tiles > 0 && pl.sk_grid != pl.sk_tiles;
  pl.partial_bytes = shared ? 2 * (size_t)pl.grid * sh.bm * sh.bn * 4 : 0;
  pl.counter_bytes = shared ? (size_t)pl.sk_tiles * 4 : 0;
  return pl;
}

// The tail tile is named by its size: of the shapes of that size, the one
// with the main shape's wave count (so that the two can share a launch), else
// the first.
int tail_index(const apt_config_t& cfg) {
  int first = -1;
  const int waves = cfg.waves_m * cfg.waves_n;
  for (int s = 0; s < kNumShapes; ++s)
    if (kShapes[s].bm == cfg.tail_bm && kShapes[s].bn == cfg.tail_bn) {
      if (kShapes[s].wm * kShapes[s].wn == waves) return s;
      if (first < 0) first = s;
    }
  return first;
}

// One or two launches: (main over [0, split_n), tail over [split_n, N)).
int make_plans(int M, int N, int K, const apt_config_t& cfg, Plan* pl) {
  if (cfg.split_n == 0) {
    pl[0] = make_plan(M, K, shape_index(cfg), 0, N, cfg.grid);
    return 1;
  }
  pl[0] = make_plan(M, K, shape_index(cfg), 0, cfg.split_n, cfg.grid);
  pl[1] = make_plan(M, K, tail_index(cfg), cfg.split_n, N - cfg.split_n, cfg.tail_grid);
  return 2;
}

}  // namespace
}  // namespace int8

bool int8_config_ok(const apt_config_t& cfg, int N) {
  if (int8::shape_index(cfg) < 0 || !(cfg.bk == 0 || cfg.bk == kChunk) || cfg.grid < 0 ||
      cfg.grid > kMaxGrid)
    return false;
  if (cfg.split_n == 0) return true;
  return cfg.split_n > 0 && cfg.split_n < N && cfg.split_n % cfg.bn == 0 &&
         cfg.split_n % kRowGroup == 0 && int8::tail_index(cfg) >= 0 && cfg.tail_grid >= 0 &&
         cfg.tail_grid <= kMaxGrid;
}

// The kernels address the packed weights, the activation fragments and the
// stream-K partial tiles with 32-bit buffer offsets.
bool int8_sizes_ok(int M, int N, int K, int p, int q, const apt_config_t& cfg) {
  const uint64_t limit = (uint64_t)1 << 32;
  // tile and chunk-pair counts are 32-bit in the plans and kernels (smallest tile 128x128)
  const int64_t tiles = (int64_t)((M + 127) / 128) * ((N + 127) / 128);
  if (tiles * (((int64_t)num_chunks(K) + 1) / 2) >= ((int64_t)1 << 31)) return false;
  // the activation expansion runs one grid row per chunk (an even count)
  if (((num_chunks(K) + 1) & ~1) > 65535) return false;
  int8::Plan pl[2];
  const int n = int8::make_plans(M, N, K, cfg, pl);
  for (int i = 0; i < n; ++i)
    if (pl[i].partial_bytes >= limit) return false;
  return apt_packed_bytes(N, K, p) < limit &&
         int8::a_frag_bytes(M, K, int8::operand_format(cfg, q)) < limit;
}

// Workspace: activation fragments, then per launch (stream-K) one arrival
// counter per stream-K tile, then per launch two int32 partial tiles per
// workgroup.
size_t int8_workspace_bytes(int M, int N, int K, int q, const apt_config_t& cfg) {
  int8::Plan pl[2];
  const int n = int8::make_plans(M, N, K, cfg, pl);
  size_t bytes = int8::align256(int8::a_frag_bytes(M, K, int8::operand_format(cfg, q)));
  for (int i = 0; i < n; ++i)
    bytes += int8::align256(pl[i].partial_bytes) + int8::align256(pl[i].counter_bytes);
  return bytes;
}

int int8_operand_format(const apt_config_t& cfg, int q) { return int8::operand_format(cfg, q); }

hipError_t launch_gemm_int8(const GemmArgs& g, const apt_config_t& cfg, void* workspace,
                            hipStream_t stream, const ActSource* src) {
  using namespace int8;
  Plan pl[2];
  const int nl = make_plans(g.M, g.N, g.K, cfg, pl);
  Int8Params prm[2];
  const int fmt = operand_format(cfg, g.q);
  uint8_t* base = static_cast<uint8_t*>(workspace) + align256(a_frag_bytes(g.M, g.K, fmt));
  int* counters = nullptr;
  int ncounters = 0;
  for (int i = 0; i < nl; ++i) {
    Int8Params& p = prm[i];
    p.g = g;
    p.nchunks = num_chunks(g.K);
    p.nsteps = ((p.nchunks + 1) & ~1) * (fmt ? Fmt<1>::kSteps : Fmt<0>::kSteps);
    p.mblocks = (g.M + 31) / 32;
    p.a_frag = static_cast<const v4i*>(workspace);
    p.a_bytes = (uint32_t)a_frag_bytes(g.M, g.K, fmt);
    p.w_bytes = (uint32_t)apt_packed_bytes(g.N, g.K, g.p);
    p.n_begin = pl[i].n_begin;
    p.tiles_n = pl[i].tiles_n;
    p.tiles = pl[i].tiles;
    p.dp_tiles = pl[i].dp_tiles;
    p.sk_pairs = pl[i].sk_pairs;
    p.sk_grid = pl[i].sk_grid;
    p.vec_out = g.N % 4 == 0 && (reinterpret_cast<uintptr_t>(g.c_int32) & 15) == 0 &&
                (reinterpret_cast<uintptr_t>(g.c_fp16) & 7) == 0;
    p.partial_bytes = (uint32_t)pl[i].partial_bytes;
  }
  // Counters of all launches first (one clearing pass), then partial tiles.
  counters = reinterpret_cast<int*>(base);
  for (int i = 0; i < nl; ++i) {
    prm[i].counters = reinterpret_cast<int*>(base);
    base += align256(pl[i].counter_bytes);
  }
  ncounters = (int)(reinterpret_cast<int*>(base) - counters);
  for (int i = 0; i < nl; ++i) {
    prm[i].partial = reinterpret_cast<v4i*>(base);
    base += align256(pl[i].partial_bytes);
  }
  v4i* frag = static_cast<v4i*>(workspace);
  const Int8Params& p0 = prm[0];
  hipError_t e = hipErrorInvalidValue;
  if (src != nullptr) {
    if (fmt != 0) return hipErrorInvalidValue;
    e = launch_act_frag(src->data, src->fp16, g.M, g.K, g.q, p0.nsteps, frag, src->rowsum,
                        src->scale, src->scale_out, counters, ncounters, stream);
  } else switch (g.q) {
    case 1: e = launch_expand_for_q<1>(fmt, g.a_packed, g.M, p0.nchunks, p0.nsteps, p0.mblocks, frag, counters, ncounters, stream); break;
    case 2: e = launch_expand_for_q<2>(fmt, g.a_packed, g.M, p0.nchunks, p0.nsteps, p0.mblocks, frag, counters, ncounters, stream); break;
    case 3: e = launch_expand_for_q<3>(fmt, g.a_packed, g.M, p0.nchunks, p0.nsteps, p0.mblocks, frag, counters, ncounters, stream); break;
    case 4: e = launch_expand_for_q<4>(fmt, g.a_packed, g.M, p0.nchunks, p0.nsteps, p0.mblocks, frag, counters, ncounters, stream); break;
    case 5: e = launch_expand_for_q<5>(fmt, g.a_packed, g.M, p0.nchunks, p0.nsteps, p0.mblocks, frag, counters, ncounters, stream); break;
    case 6: e = launch_expand_for_q<6>(fmt, g.a_packed, g.M, p0.nchunks, p0.nsteps, p0.mblocks, frag, counters, ncounters, stream); break;
    case 7: e = launch_expand_for_q<7>(fmt, g.a_packed, g.M, p0.nchunks, p0.nsteps, p0.mblocks, frag, counters, ncounters, stream); break;
    case 8: e = launch_expand_for_q<8>(fmt, g.a_packed, g.M, p0.nchunks, p0.nsteps, p0.mblocks, frag, counters, ncounters, stream); break;
  }
  if (e != hipSuccess) return e;
  if (nl == 2 && pair_supported(pl[0].shape, pl[1].shape))
    return launch_pair(g.p, fmt, pl[0].shape, prm[0], pl[0].grid, pl[1].shape, prm[1], pl[1].grid,
                       stream);
  for (int i = 0; i < nl && e == hipSuccess; ++i)
    e = launch_p(g.p, fmt, pl[i].shape, prm[i], pl[i].grid, stream);
  return e;
}

}  // namespace apt
