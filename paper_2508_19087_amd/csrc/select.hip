// select.hip - host-side kernel-config selector (APT-LLM, arXiv 2508.19087,
// Sec. V: tunable hyperparameters, lookup table, approximate matching).
//
// Lookup table: configs found by the search module (apt_search_config, Sec.
// V-B "best kernel search") are kept per (M, N, K, p, q) and win over the
// model below for exactly that problem; every other problem takes the model,
// which plays the part of the paper's approximate matching.
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
#include <mutex>

#include "apt_internal.h"

namespace apt {
namespace {

struct Int8Shape {
  int bm, bn, wm, wn;
  int per_cu;           // workgroups resident per compute unit (LDS-limited)
  double pair_cycles;   // cycles per chunk pair of one workgroup, compute unit full
};

// Measured on MI355X for K = 4096 tiles (kernel clock about 1.9 GHz).
constexpr Int8Shape kInt8Shapes[] = {
    {256, 256, 4, 2, 1, 5200.0},
    {512, 128, 8, 1, 1, 4800.0},
    {256, 128, 4, 2, 1, 3000.0},
    {128, 128, 2, 2, 2, 3000.0},
};
// Main shapes that pair with a tail shape in one launch (same wave count):
// the first two above with the third.
constexpr int kNumMainShapes = 2;
constexpr int kPairTail = 2;
constexpr int kNumInt8Shapes = (int)(sizeof(kInt8Shapes) / sizeof(kInt8Shapes[0]));
constexpr double kPartialBytesPerCycle = 2500.0;  // device-wide partial-tile traffic rate
constexpr double kTileFixedCycles = 4000.0;      // start-up and final epilogue of a workgroup

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

// Modelled cycles of shape s with `grid` workgroups (0 = one per tile).
double model_cycles(const Int8Shape& s, int M, int N, int K, int grid, int cus) {
  const int64_t tiles = (int64_t)((M + s.bm - 1) / s.bm) * ((N + s.bn - 1) / s.bn);
  const int64_t pairs = (((K + kChunk - 1) / kChunk) + 1) / 2;
  const int64_t slots = (int64_t)cus * s.per_cu;
  if (grid == 0) {  // one workgroup per tile, in rounds of `slots`
    const int64_t rounds = (tiles + slots - 1) / slots;
    return (double)rounds * (pairs * s.pair_cycles + kTileFixedCycles);
  }
  const int64_t g = std::min<int64_t>(grid, tiles * pairs);
  const int64_t dp = tiles / g, sk_tiles = tiles - dp * g;
  const int64_t sk_pairs = sk_tiles * pairs;
  const int64_t per_wg = dp * pairs + (sk_pairs + g - 1) / g;
  const int64_t rounds = (g + slots - 1) / slots;
  double cycles = (double)rounds * (per_wg * s.pair_cycles + kTileFixedCycles);
  if (sk_tiles > 0) {
    // every shared tile: about (parts - 1) partials written and read back
    const double parts = std::min<double>((double)g, (double)pairs * g / (double)sk_pairs + 1.0);
    const double bytes = 2.0 * sk_tiles * (parts - 1.0) * s.bm * s.bn * 4.0;
    cycles += bytes / kPartialBytesPerCycle;
  }
  return cycles;
}

}  // namespace

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
// whole rounds of columns, a smaller shape on the rest).
int candidate_configs(int M, int N, int K, int p, int q, apt_config_t* out, int max_out) {
  (void)K;
  int n = 0;
  auto add = [&](const apt_config_t& c) {
    if (n < max_out) out[n++] = c;
  };
  apt_config_t x = base_config(APT_ROUTE_XOR);
  x.mt = 8;
  add(x);
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
  for (int i = 0; i < kNumMainShapes; ++i) {
    const Int8Shape& s = kInt8Shapes[i];
    const int tiles_m = (M + s.bm - 1) / s.bm;
    const int cols_per_round = cus * s.per_cu / tiles_m;
    const int tiles_n = (N + s.bn - 1) / s.bn;
    if (cols_per_round < 1 || tiles_n <= cols_per_round) continue;
    const int split = tiles_n / cols_per_round * cols_per_round * s.bn;
    if (split >= N) continue;
    for (int t = kNumMainShapes; t < kNumInt8Shapes; ++t) {
      apt_config_t c = int8_cfg(s, 0);
      c.split_n = split;
      c.tail_bm = kInt8Shapes[t].bm;
      c.tail_bn = kInt8Shapes[t].bn;
      add(c);
    }
  }
  return n;
}

apt_config_t select_config(int M, int N, int K, int p, int q) {
  apt_config_t hit;
  if (table_lookup(M, N, K, p, q, &hit)) return hit;
  if (M <= 8) {
    apt_config_t c = base_config(APT_ROUTE_XOR);
    c.mt = 8;
    return c;
  }
  const int cus = compute_units();
  // Candidates: each shape alone, with one workgroup per tile or a full
  // persistent grid; and the first shape over the columns that fill whole
  // rounds of its tiles with each smaller shape (one workgroup per tile) on
  // the remaining columns.
  double best = 0.0;
  int best_i = -1, best_grid = 0, best_split = 0, best_tail = -1;
  auto consider = [&](double t, int i, int grid, int split, int tail) {
    if (best_i < 0 || t < best) {
      best = t;
      best_i = i;
      best_grid = grid;
      best_split = split;
      best_tail = tail;
    }
  };
  for (int i = 0; i < kNumInt8Shapes; ++i) {
    const Int8Shape& s = kInt8Shapes[i];
    consider(model_cycles(s, M, N, K, 0, cus), i, 0, 0, -1);
    consider(model_cycles(s, M, N, K, std::min(cus * s.per_cu, kMaxGrid), cus), i,
             std::min(cus * s.per_cu, kMaxGrid), 0, -1);
  }
  for (int i = 0; i < kNumMainShapes; ++i) {
    const Int8Shape& s = kInt8Shapes[i];
    const int tiles_m = (M + s.bm - 1) / s.bm;
    const int cols_per_round = cus * s.per_cu / tiles_m;
    const int tiles_n = (N + s.bn - 1) / s.bn;
    if (cols_per_round >= 1 && tiles_n > cols_per_round) {
      const int split = tiles_n / cols_per_round * cols_per_round * s.bn;
      if (split < N)
        for (int t = kNumMainShapes; t < kNumInt8Shapes; ++t)
          // a paired launch saves the second launch's start-up and drain
          consider(model_cycles(s, M, split, K, 0, cus) +
                       model_cycles(kInt8Shapes[t], M, N - split, K, 0, cus) -
                       (t == kPairTail ? kTileFixedCycles : 0.0),
                   i, 0, split, t);
    }
  }
  const Int8Shape& s = kInt8Shapes[best_i];
  apt_config_t c = base_config(APT_ROUTE_INT8_MFMA);
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
