// select.hip - host-side kernel-config selector (APT-LLM, arXiv 2508.19087,
// Sec. V: tunable hyperparameters, lookup table, approximate matching).
//
// Lookup tables: configs found by the search module (apt_search_config, Sec.
// V-B "best kernel search") are kept per (M, N, K, p, q) and win over
// everything else for exactly that problem; next comes the shipped table of
// searched configs for the workload shapes, matched approximately (same p, q
// and M bucket, nearest N and K within a radius); every other problem takes
// the model.
//
// The paper searches, per (M, N, K, bits), the block/warp shapes that satisfy
// its tile constraint and stores the fastest in a table.  Here the
// configuration space is the route plus the workgroup tile and wave grid the
// library is built with.  Decode-sized M takes the XOR + popcount route, which
// streams the weight planes once; larger M takes the reassembled int8 MFMA
// route, with the tile shape chosen by a model of how many rounds of tiles the
// compute units run, how fast each tile shape runs and what the stream-K
// partial tiles cost.  A choice never changes results.
#include <algorithm>
#include <array>
#include <map>
#include <cmath>
#include <mutex>

#include "apt_internal.h"

namespace apt {
namespace {

struct ShapeTimes {
  double pair_us;        // microseconds per chunk pair of one workgroup, per_cu of them on its CU
  double pair_alone_us;  // the same with the workgroup alone on its compute unit
  double fixed_us;       // launch, first loads and the last epilogue of one full round
};

struct Int8Shape {
  int bm, bn, wm, wn;
  int per_cu;            // workgroups resident per compute unit (registers and LDS)
  ShapeTimes t[4];       // operand classes: int8 with weights of <= 2, <= 4 and <= 8 bits; FP4
};

// Operand class of the model's figures: the loop's cost grows with the weight
// planes reassembled per chunk (p), while the activations reach it as int8
// (or FP4) fragments whatever q is.
inline int time_class(bool fp4, int p) { return fp4 ? 3 : p <= 2 ? 0 : p <= 4 ? 1 : 2; }

// Measured on MI355X by bench.py --calibrate: apt_gemm call times with
// M = 2048 at K = 2048 and 6144 (the K slope gives the pair time, its
// intercept the fixed time), with one full round of tiles and, for the 4-wave
// shapes, half a round (one workgroup per compute unit); int8 operands at
// W2A4, W4A4 and W8A4, FP4 operands at W2A2 (the model's only FP4 use: FP4
// weights with FP8 activations measured no faster than int8 operands, so that
// form is left to the search module).
constexpr Int8Shape kInt8Shapes[] = {
    {256, 256, 4, 2, 1, {{2.91, 2.91, 20.4}, {3.15, 3.15, 19.8}, {4.42, 4.42, 22.8}, {1.83, 1.83, 20.6}}},
    {512, 128, 8, 1, 1, {{3.17, 3.17, 19.4}, {3.87, 3.87, 15.3}, {4.96, 4.96, 16.4}, {2.25, 2.25, 16.1}}},
    {256, 128, 4, 1, 2, {{3.09, 1.70, 16.1}, {3.56, 1.72, 14.2}, {4.08, 2.29, 28.3}, {2.29, 1.18, 14.3}}},
    {256, 128, 4, 2, 1, {{1.94, 1.94, 10.9}, {2.65, 2.65, 9.3}, {3.94, 3.94, 7.7}, {1.36, 1.36, 10.8}}},
    {128, 128, 2, 2, 2, {{2.11, 1.25, 8.2}, {2.46, 1.27, 7.4}, {3.23, 1.68, 9.4}, {1.60, 0.98, 7.5}}},
};
constexpr int kNumInt8Shapes = (int)(sizeof(kInt8Shapes) / sizeof(kInt8Shapes[0]));
// Main shapes of a split launch (the first three above) and their tails (the
// last three); a main and a tail with the same wave count share one launch.
constexpr int kNumMainShapes = 3;
constexpr int kFirstTail = 2;
// Device-wide rate at which stream-K partial tiles are written and read back
// (bytes per microsecond), as the stream-K launches measured on MI355X show.
constexpr double kPartialBytesPerUs = 2.5e6;

int compute_units() {
  static int cus = 0;
  if (cus == 0) {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
      cus = n;
    else
      cus = 256;
  }
  return cus;
}

apt_config_t base_config(int route) {
  apt_config_t c;
  c.route = route;
  c.bm = c.bn = c.bk = 0;
  c.waves_m = c.waves_n = 0;
  c.grid = 0;
  c.lds_stages = 0;
  c.mt = 0;
  c.split_n = c.tail_bm = c.tail_bn = c.tail_grid = 0;
  c.reserved[0] = c.reserved[1] = c.reserved[2] = 0;
  return c;
}

// Modelled microseconds of shape s with operand class f (time_class) and
// `grid` workgroups (0 = one per tile), without the fixed time.  Workgroups
// run in rounds of cus * per_cu; a last partial round of at most one
// workgroup per compute unit runs at the alone rate.
double model_loop_us(const Int8Shape& s, int f, int M, int N, int K, int grid, int cus) {
  const int64_t tiles = (int64_t)((M + s.bm - 1) / s.bm) * ((N + s.bn - 1) / s.bn);
  const int64_t pairs = (((K + kChunk - 1) / kChunk) + 1) / 2;
  const int64_t slots = (int64_t)cus * s.per_cu;
  auto round_us = [&](int64_t wgs, int64_t wg_pairs) {
    return (double)wg_pairs * (wgs <= cus ? s.t[f].pair_alone_us : s.t[f].pair_us);
  };
  if (grid == 0) {
    // a second round of workgroups starts its pipeline again (the loads of
    // its first chunks and the ring fill, about two pairs alone: W4A4
    // 2048x11008x4096 88.6 us against 85.0 us with the leftover tiles
    // chained onto the first round's workgroups)
    const int64_t full = tiles / slots, rem = tiles % slots;
    return (double)full * round_us(slots, pairs) +
           (rem ? round_us(rem, pairs) + (full ? 2.0 * s.t[f].pair_alone_us : 0.0) : 0.0);
  }
  const int64_t g = std::min<int64_t>(grid, tiles * pairs);
  const int64_t dp = tiles / g, sk_tiles = tiles - dp * g;
  const int64_t sk_pairs = sk_tiles * pairs;
  // stream-K tiles whole when they are more than half of the compute units
  // the grid covers and no more than all of them, else in about two parts
  // (the launch's rule)
  const int64_t units = std::max<int64_t>(1, g / s.per_cu);
  const int64_t k = 2 * sk_tiles > units && sk_tiles <= units ? 1 : 2;
  const int64_t sk_g = sk_tiles ? std::min<int64_t>(g, k * sk_tiles) : 0;
  if (k == 1 && dp >= 1 && s.per_cu == 2 && g == slots) {
    // whole leftover tiles extend the chunk streams of sk_g <= cus
    // workgroups, at most one per compute unit (which holds workgroups w and
    // w + cus), which runs its extra pairs alone after the shared rounds
    return (double)dp * pairs * s.t[f].pair_us + (double)pairs * s.t[f].pair_alone_us;
  }
  const int64_t per_wg = dp * pairs + (sk_g ? (sk_pairs + sk_g - 1) / sk_g : 0);
  const int64_t active = dp ? g : sk_g;
  const int64_t rounds = (active + slots - 1) / slots;
  double us = (double)rounds * round_us(std::min(active, slots), per_wg);
  if (sk_tiles > 0 && k > 1) {
    // every shared tile: (parts - 1) partials written and read back; a tile
    // has sk_g / sk_tiles parts, one more where part bounds fall inside it
    const double parts = (double)sk_g / (double)sk_tiles + 0.5;
    const double bytes = 2.0 * sk_tiles * std::max(0.0, parts - 1.0) * s.bm * s.bn * 4.0;
    us += bytes / kPartialBytesPerUs;
  }
  return us;
}

double model_us(const Int8Shape& s, int f, int M, int N, int K, int grid, int cus) {
  return model_loop_us(s, f, M, N, K, grid, cus) + s.t[f].fixed_us;
}

// The tail shape a split config with main shape i and tail size of shape t
// runs: of the shapes of that size, the one with the main shape's wave count
// (the library's rule), else t itself.
// Modelled microseconds of the XOR route (8 activation rows per block row):
// a fixed part and a cost per 32-bit word pair of an 8-row activation block
// and one weight row, rising with the activation planes read from LDS (q) and
// with the p*q plane products.  Fitted (least squares on the relative error)
// to MI355X timings for M = 16 to 256, N and K from 1024 to 14336 and p*q
// from 2 to 16: median error 8%.
double model_xor_us(int M, int N, int K, int p, int q) {
  const double words = 8.0 * ((M + 7) / 8) * (double)N * K / 32.0;
  return 3.564 + words * (-0.2140 + 0.1792 * q + 0.0439 * p * q) * 1e-6;
}

bool tail_runs_as(int i, int t) {
  const Int8Shape &m = kInt8Shapes[i], &ts = kInt8Shapes[t];
  for (int u = 0; u < kNumInt8Shapes; ++u) {
    const Int8Shape& o = kInt8Shapes[u];
    if (u != t && o.bm == ts.bm && o.bn == ts.bn && o.wm * o.wn == m.wm * m.wn) return false;
  }
  return true;
}

// Columns [0, split) that fill whole rounds of shape s's tiles, or 0 when
// there is no such split short of N.
int split_columns(const Int8Shape& s, int M, int N, int cus) {
  const int tiles_m = (M + s.bm - 1) / s.bm;
  const int cols_per_round = cus * s.per_cu / tiles_m;
  const int tiles_n = (N + s.bn - 1) / s.bn;
  if (cols_per_round < 1 || tiles_n <= cols_per_round) return 0;
  const int split = tiles_n / cols_per_round * cols_per_round * s.bn;
  return split < N ? split : 0;
}

// The shipped lookup table (Sec. V-B keeps the search results for common LLM
// shapes): the configs the best-kernel search module picked on MI355X for the
// workload shapes with M > 8 (bench.py --search), keyed by the M bucket
// ceil(log2 M), N, K, p and q.  Smaller M always takes the XOR route.  The
// two 11008 x 4096 entries run one persistent round with the leftover tiles
// chained whole onto its workgroups (measured 3-5% faster than one workgroup
// per tile; see sk_parts in gemm_int8.hip).
struct ShippedEntry {
  int mlog, N, K, p, q;
  apt_config_t cfg;
};
constexpr ShippedEntry kShipped[] = {
    { 4,   512,   512, 1, 2, {1, 0, 0, 0, 0, 0, 0, 0, 8, 0, 0, 0, 0, {0, 0, 0}}},  // w1a2_16x512x512
    {11, 11008,  4096, 4, 4, {3, 256, 128, 128, 4, 1, 512, 3, 0, 0, 0, 0, 0, {0, 0, 0}}},  // w4a4_prefill_2048x11008x4096
    { 9,  4096, 11008, 1, 1, {4, 128, 128, 128, 2, 2, 512, 3, 0, 0, 0, 0, 0, {0, 0, 0}}},  // sweep_w1a1_512x4096x11008
    { 9,  4096, 11008, 1, 4, {3, 128, 128, 128, 2, 2, 512, 3, 0, 0, 0, 0, 0, {0, 0, 0}}},  // sweep_w1a4_512x4096x11008
    { 9,  4096, 11008, 2, 8, {3, 128, 128, 128, 2, 2, 512, 3, 0, 0, 0, 0, 0, {0, 0, 0}}},  // sweep_w2a8_512x4096x11008
    { 9,  4096, 11008, 3, 3, {3, 128, 128, 128, 2, 2, 512, 3, 0, 0, 0, 0, 0, {0, 0, 0}}},  // sweep_w3a3_512x4096x11008
    { 9,  4096, 11008, 3, 8, {3, 128, 128, 128, 2, 2, 512, 3, 0, 0, 0, 0, 0, {0, 0, 0}}},  // sweep_w3a8_512x4096x11008
    { 9,  4096, 11008, 4, 8, {3, 128, 128, 128, 2, 2, 512, 3, 0, 0, 0, 0, 0, {0, 0, 0}}},  // sweep_w4a8_512x4096x11008
    {10,  4096,  4096, 2, 4, {3, 128, 128, 128, 2, 2, 0, 3, 0, 0, 0, 0, 0, {0, 0, 0}}},  // w2a4_q_m1024
    {10, 11008,  4096, 2, 4, {3, 128, 128, 128, 2, 2, 512, 3, 0, 0, 0, 0, 0, {0, 0, 0}}},  // w2a4_gate_m1024
    {10,  4096, 11008, 2, 4, {3, 128, 128, 128, 2, 2, 0, 3, 0, 0, 0, 0, 0, {0, 0, 0}}},  // w2a4_down_m1024
};

// Approximate matching (Sec. V-B; the paper gives no distance): an entry
// matches a problem with the same p, q and M bucket when
// |log2(N / N_e)| + |log2(K / K_e)| <= kMatchRadius; the nearest such entry
// whose config is valid for the problem wins, and a problem no entry matches
// takes the model.  The radius admits shapes within about 1.4x of a tabled one
// in one dimension (a TP shard of a tabled layer, a neighbouring hidden size).
constexpr double kMatchRadius = 0.5;

int mlog_of(int M) {
  int l = 0;
  while ((1 << l) < M) ++l;
  return l;
}

}  // namespace

bool shipped_lookup(int M, int N, int K, int p, int q, apt_config_t* out) {
  const int ml = mlog_of(M);
  double best = kMatchRadius + 1e-9;
  const ShippedEntry* hit = nullptr;
  for (const ShippedEntry& e : kShipped) {
    if (e.mlog != ml || e.p != p || e.q != q) continue;
    const double d = std::fabs(std::log2((double)N / e.N)) + std::fabs(std::log2((double)K / e.K));
    if (d > best) continue;
    const apt_config_t& c = e.cfg;
    if (mfma_route(c.route) && (!int8_config_ok(c, N) || !int8_sizes_ok(M, N, K, p, q, c))) continue;
    if (c.route == APT_ROUTE_FP4_MFMA && !fp4_route_ok(K, p, q)) continue;
    if (c.route == APT_ROUTE_FP6_MFMA && !fp6_route_ok(K, p, q)) continue;
    if (c.route == APT_ROUTE_FP8_MFMA && !fp8_route_ok(K, p, q)) continue;
    best = d;
    hit = &e;
  }
  if (hit == nullptr) return false;
  *out = hit->cfg;
  return true;
}

int shipped_table_size() { return (int)(sizeof(kShipped) / sizeof(kShipped[0])); }

namespace {

// The table; its lock makes the library's only mutable state safe to share
// between threads.
std::mutex g_table_mu;
std::map<std::array<int, 5>, apt_config_t> g_table;

}  // namespace

bool table_lookup(int M, int N, int K, int p, int q, apt_config_t* out) {
  std::lock_guard<std::mutex> lock(g_table_mu);
  auto it = g_table.find({M, N, K, p, q});
  if (it == g_table.end()) return false;
  *out = it->second;
  return true;
}

void table_store(int M, int N, int K, int p, int q, const apt_config_t& c) {
  std::lock_guard<std::mutex> lock(g_table_mu);
  g_table[{M, N, K, p, q}] = c;
}

void table_clear() {
  std::lock_guard<std::mutex> lock(g_table_mu);
  g_table.clear();
}

int table_size() {
  std::lock_guard<std::mutex> lock(g_table_mu);
  return (int)g_table.size();
}

// Every config the search module times for (M, N, K, p, q): the XOR route,
// the +-1 plane route where its operands fit (p, q <= 7), each int8 tile shape
// with one workgroup per tile and with a persistent grid of one round of
// workgroups, and the split launches the model considers (a main shape over
// whole rounds of columns, a smaller shape on the rest); each of these again
// on the FP4 route where it applies (FP4 or FP8 activations).
// The most configs candidate_configs can list: XOR (three launch shapes),
// +-1 planes, then for each
// operand format every shape twice and every main shape with every tail.
static_assert(4 + 2 * (2 * kNumInt8Shapes + kNumMainShapes * (kNumInt8Shapes - kFirstTail)) <=
                  kMaxCandidates,
              "the search module's candidate list must hold every config");

int candidate_configs(int M, int N, int K, int p, int q, apt_config_t* out, int max_out) {
  int n = 0;
  auto add = [&](const apt_config_t& c) {
    if (n < max_out) out[n++] = c;
  };
  // the XOR route with the library's launch shape, and with the K split
  // forced off and on
  for (int ks = 0; ks <= 4; ks += 4) {
    apt_config_t x = base_config(APT_ROUTE_XOR);
    x.waves_n = ks;
    add(x);
    if (ks == 0) {
      x.waves_n = 1;
      add(x);
    }
  }
  if (p <= 7 && q <= 7) add(base_config(APT_ROUTE_PM1_MFMA));
  const int cus = compute_units();
  auto int8_cfg = [&](const Int8Shape& s, int grid) {
    apt_config_t c = base_config(APT_ROUTE_INT8_MFMA);
    c.bm = s.bm;
    c.bn = s.bn;
    c.bk = kChunk;
    c.waves_m = s.wm;
    c.waves_n = s.wn;
    c.lds_stages = 3;
    c.grid = grid;
    return c;
  };
  for (int i = 0; i < kNumInt8Shapes; ++i) {
    const Int8Shape& s = kInt8Shapes[i];
    add(int8_cfg(s, 0));
    add(int8_cfg(s, std::min(cus * s.per_cu, kMaxGrid)));
  }
  const int n_int8_single = n;
  for (int i = 0; i < kNumMainShapes; ++i) {
    const Int8Shape& s = kInt8Shapes[i];
    const int split = split_columns(s, M, N, cus);
    if (split == 0) continue;
    for (int t = kFirstTail; t < kNumInt8Shapes; ++t) {
      if (!tail_runs_as(i, t)) continue;
      apt_config_t c = int8_cfg(s, 0);
      c.split_n = split;
      c.tail_bm = kInt8Shapes[t].bm;
      c.tail_bn = kInt8Shapes[t].bn;
      add(c);
    }
  }
  // the same tile configs with FP4 operands where they apply, with FP6
  // operands where those apply and FP4 does not (p or q = 3), and with FP8
  // operands where neither applies (p or q = 4)
  const int end = n;
  const int route = fp4_route_ok(K, p, q)   ? APT_ROUTE_FP4_MFMA
                    : fp6_route_ok(K, p, q) ? APT_ROUTE_FP6_MFMA
                    : fp8_route_ok(K, p, q) ? APT_ROUTE_FP8_MFMA : 0;
  if (route != 0) {
    for (int j = n_int8_single - 2 * kNumInt8Shapes; j < end; ++j) {
      apt_config_t c = out[j];
      c.route = route;
      add(c);
    }
  }
  return n;
}

apt_config_t select_config(int M, int N, int K, int p, int q) {
  apt_config_t hit;
  if (table_lookup(M, N, K, p, q, &hit)) return hit;
  if (M > 8 && shipped_lookup(M, N, K, p, q, &hit)) return hit;
  if (M <= 8) return base_config(APT_ROUTE_XOR);  // launch shape chosen by the route
  const int cus = compute_units();
  // Candidates: each shape alone, with one workgroup per tile or a
  // persistent grid of one round; and each main shape over the columns that
  // fill whole rounds of its tiles, with each tail shape (one workgroup per
  // tile) on the remaining columns.
  double best = 0.0;
  int best_i = -1, best_grid = 0, best_split = 0, best_tail = -1;
  bool best_fp4 = false;
  bool fp4 = false;
  auto consider = [&](double t, int i, int grid, int split, int tail) {
    if (best_i < 0 || t < best) {
      best = t;
      best_i = i;
      best_grid = grid;
      best_split = split;
      best_tail = tail;
      best_fp4 = fp4;
    }
  };
  // int8 operands, then (where they apply) FP4 operands for both sides
  for (int fi = 0; fi < (fp4_route_ok(K, p, q) && q <= 2 ? 2 : 1); ++fi) {
    fp4 = fi == 1;
    const int f = time_class(fp4, p);
    for (int i = 0; i < kNumInt8Shapes; ++i) {
      const Int8Shape& s = kInt8Shapes[i];
      const int round = std::min(cus * s.per_cu, kMaxGrid);
      consider(model_us(s, f, M, N, K, 0, cus), i, 0, 0, -1);
      consider(model_us(s, f, M, N, K, round, cus), i, round, 0, -1);
    }
    for (int i = 0; i < kNumMainShapes; ++i) {
      const Int8Shape& s = kInt8Shapes[i];
      const int split = split_columns(s, M, N, cus);
      if (split == 0) continue;
      for (int t = kFirstTail; t < kNumInt8Shapes; ++t) {
        if (!tail_runs_as(i, t)) continue;
        const Int8Shape& ts = kInt8Shapes[t];
        // one launch when the wave counts match: one fixed time, else two
        const bool paired = ts.wm * ts.wn == s.wm * s.wn;
        const double fs = s.t[f].fixed_us, ft = ts.t[f].fixed_us;
        consider(model_loop_us(s, f, M, split, K, 0, cus) +
                     model_loop_us(ts, f, M, N - split, K, 0, cus) +
                     (paired ? std::max(fs, ft) : fs + ft),
                 i, 0, split, t);
      }
    }
  }
  // small problems: the XOR route's single launch against the MFMA routes'
  // fixed costs.  The MFMA figures were measured with every compute unit
  // busy and overstate grids of a few tiles by 10-40%, so they count at 90%
  // here (measured over M = 16..256, N, K = 1024..14336, p*q = 2..16).
  if (model_xor_us(M, N, K, p, q) < 0.9 * best) return base_config(APT_ROUTE_XOR);
  const Int8Shape& s = kInt8Shapes[best_i];
  apt_config_t c = base_config(best_fp4 ? APT_ROUTE_FP4_MFMA : APT_ROUTE_INT8_MFMA);
  c.bm = s.bm;
  c.bn = s.bn;
  c.bk = kChunk;
  c.waves_m = s.wm;
  c.waves_n = s.wn;
  c.lds_stages = 3;
  c.grid = best_grid;
  if (best_split > 0) {
    c.split_n = best_split;
    c.tail_bm = kInt8Shapes[best_tail].bm;
    c.tail_bn = kInt8Shapes[best_tail].bn;
    c.tail_grid = 0;
  }
  return c;
}

}  // namespace apt
