// select.hip - host-side kernel-config selector (APT-LLM, arXiv 2508.19087,
// Sec. V: tunable hyperparameters, lookup table, approximate matching).
//
// The paper searches, per (M, N, K, bits), the block/warp shapes that satisfy
// its tile constraint and stores the fastest in a table.  Here the
// configuration space is the route plus the workgroup tile and wave grid the
// library is built with.  Decode-sized M takes the XOR + popcount route, which
// streams the weight planes once; larger M takes the reassembled int8 MFMA
// route, with the tile shape chosen by a model of how many rounds of tiles the
// 256 compute units run and how fast each tile shape runs.  A choice never
// changes results.
#include "apt_internal.h"

namespace apt {
namespace {

constexpr int kComputeUnits = 256;

struct Int8Shape {
  int bm, bn, wm, wn;
  int per_cu;        // workgroups resident per compute unit (LDS-limited)
  double rel_speed;  // throughput of one resident tile set relative to 256x256
};

constexpr Int8Shape kInt8Shapes[] = {
    {256, 256, 4, 2, 1, 1.00},
    {256, 128, 4, 2, 1, 0.80},
    {128, 128, 2, 2, 3, 0.40},
};

apt_config_t base_config(int route) {
  apt_config_t c;
  c.route = route;
  c.bm = c.bn = c.bk = 0;
  c.waves_m = c.waves_n = 0;
  c.k_split = 0;
  c.lds_stages = 0;
  c.mt = 0;
  c.split_n = c.tail_bm = c.tail_bn = 0;
  return c;
}

// Model time of covering n_cols output columns with shape s: rounds of
// resident tiles x work per tile / tile speed (arbitrary units).
double model_time(const Int8Shape& s, int M, int n_cols) {
  const long tiles = (long)((M + s.bm - 1) / s.bm) * ((n_cols + s.bn - 1) / s.bn);
  const long slots = (long)kComputeUnits * s.per_cu;
  const long rounds = (tiles + slots - 1) / slots;
  return (double)rounds * s.bm * s.bn * s.per_cu / s.rel_speed;
}

constexpr int kNumInt8Shapes = (int)(sizeof(kInt8Shapes) / sizeof(kInt8Shapes[0]));
constexpr int kTailShape = kNumInt8Shapes - 1;  // the smallest tile
constexpr double kLaunchCost = 2.0e4;           // a second launch, in model units

}  // namespace

apt_config_t select_config(int M, int N, int K, int p, int q) {
  (void)K;
  (void)p;
  (void)q;
  if (M <= 8) {
    apt_config_t c = base_config(APT_ROUTE_XOR);
    c.mt = 8;
    return c;
  }
  // Candidates: every shape alone, and every shape on the columns that fill
  // whole rounds with the smallest shape on the rest.
  double best = 0.0;
  int best_i = -1, best_split = 0;
  for (int i = 0; i < kNumInt8Shapes; ++i) {
    const Int8Shape& s = kInt8Shapes[i];
    const double t = model_time(s, M, N);
    if (best_i < 0 || t < best) {
      best = t;
      best_i = i;
      best_split = 0;
    }
    const int tiles_m = (M + s.bm - 1) / s.bm;
    const int cols_per_round = kComputeUnits * s.per_cu / tiles_m;
    const int tiles_n = (N + s.bn - 1) / s.bn;
    if (i == kTailShape || cols_per_round < 1) continue;
    const int full = tiles_n / cols_per_round * cols_per_round;
    if (full < 1 || full * s.bn >= N) continue;
    const int split = full * s.bn;
    const double ts = model_time(s, M, split) + model_time(kInt8Shapes[kTailShape], M, N - split) +
                      kLaunchCost;
    if (ts < best) {
      best = ts;
      best_i = i;
      best_split = split;
    }
  }
  const Int8Shape& s = kInt8Shapes[best_i];
  apt_config_t c = base_config(APT_ROUTE_INT8_MFMA);
  c.bm = s.bm;
  c.bn = s.bn;
  c.bk = kChunk;
  c.waves_m = s.wm;
  c.waves_n = s.wn;
  c.lds_stages = 2;
  if (best_split > 0) {
    c.split_n = best_split;
    c.tail_bm = kInt8Shapes[kTailShape].bm;
    c.tail_bn = kInt8Shapes[kTailShape].bn;
  }
  return c;
}

}  // namespace apt
