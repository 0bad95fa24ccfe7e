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
    {128, 128, 2, 2, 2, 0.60},
};

apt_config_t base_config(int route) {
  apt_config_t c;
  c.route = route;
  c.bm = c.bn = c.bk = 0;
  c.waves_m = c.waves_n = 0;
  c.k_split = 0;
  c.lds_stages = 0;
  c.mt = 0;
  c.reserved[0] = c.reserved[1] = c.reserved[2] = 0;
  return c;
}

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
  // Time model: rounds of resident tiles x work per tile / tile speed.
  double best = 0.0;
  int best_i = 0;
  for (int i = 0; i < (int)(sizeof(kInt8Shapes) / sizeof(kInt8Shapes[0])); ++i) {
    const Int8Shape& s = kInt8Shapes[i];
    const long tiles = (long)((M + s.bm - 1) / s.bm) * ((N + s.bn - 1) / s.bn);
    const long slots = (long)kComputeUnits * s.per_cu;
    const long rounds = (tiles + slots - 1) / slots;
    const double t = (double)rounds * s.bm * s.bn * s.per_cu / s.rel_speed;
    if (i == 0 || t < best) {
      best = t;
      best_i = i;
    }
  }
  apt_config_t c = base_config(APT_ROUTE_INT8_MFMA);
  c.bm = kInt8Shapes[best_i].bm;
  c.bn = kInt8Shapes[best_i].bn;
  c.bk = kChunk;
  c.waves_m = kInt8Shapes[best_i].wm;
  c.waves_n = kInt8Shapes[best_i].wn;
  c.lds_stages = 2;
  return c;
}

}  // namespace apt
