// api.hip - the extern "C" entry points declared in include/apt.h: argument
// validation, config resolution and kernel launch on the caller's stream.
// Validation always runs before any HIP call, so a rejected call touches
// neither the device nor the runtime.
#include <string.h>

#include <algorithm>

#include "apt_internal.h"

namespace apt {

// hipError_t of the last call of this thread that returned APT_ERR_HIP.
thread_local int t_last_hip_error = 0;

apt_status_t hip_status(hipError_t e) {
  if (e == hipSuccess) return APT_OK;
  t_last_hip_error = (int)e;
  return APT_ERR_HIP;
}

}  // namespace apt

namespace {

using apt::hip_status;

bool bits_ok(int b) { return b >= 1 && b <= 8; }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// K (2^p - 1)(2^q - 1) bounds |C|; it must stay below 2^31.
bool fits_int32(int K, int p, int q) {
  const int64_t bound = (int64_t)K * ((1 << p) - 1) * ((1 << q) - 1);
  return bound < ((int64_t)1 << 31);
}


// The packers index a row's elements with 32-bit ints.
constexpr int kMaxPackK = 1 << 30;

apt_status_t pack_common(const int8_t* codes, int rows, int K, int bits, void* packed,
                         int32_t* rowsum, void* stream) {
  if (rows < 1 || K < 1 || !bits_ok(bits) || codes == nullptr || packed == nullptr ||
      !aligned16(packed))
    return APT_ERR_INVALID_ARG;
  if (K > kMaxPackK) return APT_ERR_UNSUPPORTED;
  return hip_status(apt::launch_pack(codes, rows, K, bits, static_cast<uint32_t*>(packed), rowsum,
                                     static_cast<hipStream_t>(stream)));
}

// Checks a config against the problem; returns APT_OK or the status to report.
apt_status_t check_config(const apt_config_t& c, int M, int N, int K, int p, int q,
                          bool have_rowsums) {
  switch (c.route) {
    case APT_ROUTE_XOR:
      if (!apt::xor_config_ok(c)) return APT_ERR_INVALID_ARG;
      if (!apt::xor_sizes_ok(M, N, K, p, q, c)) return APT_ERR_UNSUPPORTED;
      return APT_OK;
    case APT_ROUTE_FP4_MFMA:
      if (!apt::fp4_route_ok(K, p, q)) return APT_ERR_UNSUPPORTED;
      [[fallthrough]];
    case APT_ROUTE_FP6_MFMA:
      if (c.route == APT_ROUTE_FP6_MFMA && !apt::fp6_route_ok(K, p, q)) return APT_ERR_UNSUPPORTED;
      [[fallthrough]];
    case APT_ROUTE_FP8_MFMA:
      if (c.route == APT_ROUTE_FP8_MFMA && !apt::fp8_route_ok(K, p, q)) return APT_ERR_UNSUPPORTED;
      [[fallthrough]];
    case APT_ROUTE_INT8_MFMA:
      if (!apt::int8_config_ok(c, N)) return APT_ERR_INVALID_ARG;
      if (!have_rowsums) return APT_ERR_INVALID_ARG;
      if (!apt::int8_sizes_ok(M, N, K, p, q, c)) return APT_ERR_UNSUPPORTED;
      return APT_OK;
    case APT_ROUTE_PM1_MFMA:
      if (p > 7 || q > 7) return APT_ERR_UNSUPPORTED;
      if (!apt::pm1_config_ok(c, p, q)) return APT_ERR_INVALID_ARG;
      if (!apt::pm1_sizes_ok(M, N)) return APT_ERR_UNSUPPORTED;
      return APT_OK;
    default:
      return APT_ERR_INVALID_ARG;
  }
}

}  // namespace

extern "C" {

size_t apt_packed_bytes(int rows, int K, int bits) {
  if (rows < 1 || K < 1 || !bits_ok(bits)) return 0;
  return (size_t)apt::padded_rows(rows) * (size_t)apt::num_chunks(K) * (size_t)bits *
         apt::kWordsPerPlane * 4;
}

apt_status_t apt_pack_weights(const int8_t* w_codes, int N, int K, int p, void* w_packed,
                              int32_t* w_rowsum, void* stream) {
  return pack_common(w_codes, N, K, p, w_packed, w_rowsum, stream);
}

apt_status_t apt_quantize_pack_activations(const int8_t* a_codes, int M, int K, int q,
                                           void* a_packed, int32_t* a_rowsum, void* stream) {
  return pack_common(a_codes, M, K, q, a_packed, a_rowsum, stream);
}

apt_status_t apt_quantize_pack_activations_fp16(const uint16_t* a_fp16, int M, int K, int q,
                                                void* a_packed, int32_t* a_rowsum,
                                                uint16_t* a_scale, void* stream) {
  if (M < 1 || K < 1 || !bits_ok(q) || a_fp16 == nullptr || a_packed == nullptr ||
      a_scale == nullptr || !aligned16(a_packed))
    return APT_ERR_INVALID_ARG;
  if (K > kMaxPackK) return APT_ERR_UNSUPPORTED;
  return hip_status(apt::launch_quantize_pack(a_fp16, M, K, q, static_cast<uint32_t*>(a_packed),
                                              a_rowsum, a_scale, static_cast<hipStream_t>(stream)));
}

apt_status_t apt_select_config(int M, int N, int K, int p, int q, apt_config_t* out) {
  if (M < 1 || N < 1 || K < 1 || !bits_ok(p) || !bits_ok(q) || out == nullptr)
    return APT_ERR_INVALID_ARG;
  *out = apt::select_config(M, N, K, p, q);
  return APT_OK;
}

size_t apt_gemm_workspace_bytes(int M, int N, int K, int p, int q, const apt_config_t* cfg) {
  if (M < 1 || N < 1 || K < 1 || !bits_ok(p) || !bits_ok(q)) return 0;
  const apt_config_t c = (cfg == nullptr || cfg->route == APT_ROUTE_AUTO)
                             ? apt::select_config(M, N, K, p, q)
                             : *cfg;
  if (!apt::mfma_route(c.route)) return 0;
  if (check_config(c, M, N, K, p, q, true) != APT_OK) return 0;
  return apt::int8_workspace_bytes(M, N, K, q, c);
}

}  // extern "C"

namespace apt {

apt_status_t gemm_check(int M, int N, int K, int p, int q, const void* a_packed,
                        const void* w_packed, const int32_t* a_rowsum, const int32_t* w_rowsum,
                        const int32_t* c_int32, const uint16_t* a_scale, const uint16_t* w_scale,
                        const uint16_t* c_fp16, const apt_config_t* cfg, apt_config_t* resolved) {
  if (M < 1 || N < 1 || K < 1 || !bits_ok(p) || !bits_ok(q)) return APT_ERR_INVALID_ARG;
  if (a_packed == nullptr || w_packed == nullptr || !aligned16(a_packed) || !aligned16(w_packed))
    return APT_ERR_INVALID_ARG;
  if (c_int32 == nullptr && c_fp16 == nullptr) return APT_ERR_INVALID_ARG;
  if (c_fp16 != nullptr && (a_scale == nullptr || w_scale == nullptr)) return APT_ERR_INVALID_ARG;
  if (!fits_int32(K, p, q)) return APT_ERR_UNSUPPORTED;
  apt_config_t c;
  if (cfg == nullptr || cfg->route == APT_ROUTE_AUTO)
    c = select_config(M, N, K, p, q);
  else
    c = *cfg;
  const bool have_rowsums = a_rowsum != nullptr && w_rowsum != nullptr;
  const apt_status_t st = check_config(c, M, N, K, p, q, have_rowsums);
  if (st != APT_OK) return st;
  *resolved = c;
  return APT_OK;
}

size_t gemm_workspace_need(int M, int N, int K, int q, const apt_config_t& c) {
  if (!mfma_route(c.route)) return 0;
  return int8_workspace_bytes(M, N, K, q, c);
}

apt_status_t gemm_launch(int M, int N, int K, int p, int q, const void* a_packed,
                         const void* w_packed, const int32_t* a_rowsum, const int32_t* w_rowsum,
                         int32_t* c_int32, const uint16_t* a_scale, const uint16_t* w_scale,
                         uint16_t* c_fp16, const uint16_t* a_zero, const uint16_t* w_zero,
                         const apt_config_t& c, void* workspace, size_t workspace_bytes,
                         void* stream) {
  const size_t need = gemm_workspace_need(M, N, K, q, c);
  if (need > 0) {
    if (workspace == nullptr || workspace_bytes < need) return APT_ERR_WORKSPACE;
    if (!aligned16(workspace)) return APT_ERR_INVALID_ARG;
  }
  GemmArgs g;
  g.M = M; g.N = N; g.K = K; g.p = p; g.q = q;
  g.a_packed = static_cast<const uint32_t*>(a_packed);
  g.w_packed = static_cast<const uint32_t*>(w_packed);
  g.a_rowsum = a_rowsum;
  g.w_rowsum = w_rowsum;
  g.c_int32 = c_int32;
  g.a_scale = reinterpret_cast<const __half*>(a_scale);
  g.w_scale = reinterpret_cast<const __half*>(w_scale);
  g.c_fp16 = reinterpret_cast<__half*>(c_fp16);
  g.a_zero = reinterpret_cast<const __half*>(a_zero);
  g.w_zero = reinterpret_cast<const __half*>(w_zero);
  hipStream_t s = static_cast<hipStream_t>(stream);
  switch (c.route) {
    case APT_ROUTE_XOR: return hip_status(launch_gemm_xor(g, c, s));
    case APT_ROUTE_INT8_MFMA:
    case APT_ROUTE_FP4_MFMA:
    case APT_ROUTE_FP6_MFMA:
    case APT_ROUTE_FP8_MFMA: return hip_status(launch_gemm_int8(g, c, workspace, s));
    case APT_ROUTE_PM1_MFMA: return hip_status(launch_gemm_pm1(g, c, s));
  }
  return APT_ERR_INVALID_ARG;
}

apt_status_t gemm_common(int M, int N, int K, int p, int q, const void* a_packed,
                         const void* w_packed, const int32_t* a_rowsum, const int32_t* w_rowsum,
                         int32_t* c_int32, const uint16_t* a_scale, const uint16_t* w_scale,
                         uint16_t* c_fp16, const uint16_t* a_zero, const uint16_t* w_zero,
                         const apt_config_t* cfg, void* workspace, size_t workspace_bytes,
                         void* stream) {
  apt_config_t c;
  const apt_status_t st = gemm_check(M, N, K, p, q, a_packed, w_packed, a_rowsum, w_rowsum,
                                     c_int32, a_scale, w_scale, c_fp16, cfg, &c);
  if (st != APT_OK) return st;
  return gemm_launch(M, N, K, p, q, a_packed, w_packed, a_rowsum, w_rowsum, c_int32, a_scale,
                     w_scale, c_fp16, a_zero, w_zero, c, workspace, workspace_bytes, stream);
}

// ---- GEMM from unpacked activations (apt_gemm_act) ----------------------
//
// How a resolved config consumes the activations: the XOR route's fused form
// (M <= 8, rows converted in the GEMV's LDS), the int8-format MFMA route's
// fragments written straight from the source, or else the packer into the
// workspace followed by the route as apt_gemm runs it.
enum class ActPlan { kFusedXor, kFragments, kPack };

struct ActLayout {
  ActPlan plan;
  size_t route_bytes;  // the route's own workspace, at offset 0
  size_t planes_off;   // packed activations (kPack)
  size_t rowsum_off;   // int32 [M] row sums (kFragments, kPack)
  size_t scale_off;    // fp16 [M] scales of an fp16 source (kFragments, kPack)
  size_t total;
};

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

ActLayout act_layout(int M, int N, int K, int p, int q, bool fp16, const apt_config_t& c) {
  ActLayout L{};
  if (c.route == APT_ROUTE_XOR && M <= APT_DECODE_MAX_M &&
      xor_act_sizes_ok(M, N, K, p, q, c, fp16)) {
    L.plan = ActPlan::kFusedXor;
    return L;
  }
  // (the fragment writer addresses the whole source with 31-bit byte offsets)
  const bool frags = c.route == APT_ROUTE_INT8_MFMA && int8_operand_format(c, q) == 0 &&
                     (int64_t)M * K * (fp16 ? 2 : 1) < ((int64_t)1 << 31);
  L.plan = frags ? ActPlan::kFragments : ActPlan::kPack;
  L.route_bytes = align256(gemm_workspace_need(M, N, K, q, c));
  size_t off = L.route_bytes;
  L.planes_off = off;
  if (!frags) off += align256(apt_packed_bytes(M, K, q));
  L.rowsum_off = off;
  off += align256((size_t)M * 4);
  L.scale_off = off;
  off += align256((size_t)M * 2);
  L.total = off;
  return L;
}

// Validates an apt_gemm_act call and resolves its config; returns APT_OK or
// the status to report.
apt_status_t act_check(int M, int N, int K, int p, int q, const void* a_src, int a_kind,
                       const void* w_packed, const int32_t* w_rowsum, const int32_t* c_int32,
                       const uint16_t* a_scale, const uint16_t* w_scale, const uint16_t* c_fp16,
                       const uint16_t* a_scale_out, const apt_config_t* cfg, apt_config_t* resolved,
                       ActLayout* layout) {
  if (M < 1 || N < 1 || K < 1 || !bits_ok(p) || !bits_ok(q)) return APT_ERR_INVALID_ARG;
  if (a_kind != APT_ACT_CODES && a_kind != APT_ACT_FP16) return APT_ERR_INVALID_ARG;
  const bool fp16 = a_kind == APT_ACT_FP16;
  if (a_src == nullptr || w_packed == nullptr || !aligned16(w_packed)) return APT_ERR_INVALID_ARG;
  if (fp16 && (reinterpret_cast<uintptr_t>(a_src) & 1u) != 0) return APT_ERR_INVALID_ARG;
  if (c_int32 == nullptr && c_fp16 == nullptr) return APT_ERR_INVALID_ARG;
  if (c_fp16 != nullptr && (w_scale == nullptr || (!fp16 && a_scale == nullptr)))
    return APT_ERR_INVALID_ARG;
  if (fp16 ? a_scale != nullptr : a_scale_out != nullptr) return APT_ERR_INVALID_ARG;
  if (!fits_int32(K, p, q)) return APT_ERR_UNSUPPORTED;
  if (K > kMaxPackK) return APT_ERR_UNSUPPORTED;
  apt_config_t c = (cfg == nullptr || cfg->route == APT_ROUTE_AUTO) ? select_config(M, N, K, p, q)
                                                                      : *cfg;
  // the activation row sums come from this call; the weights' from the caller
  const apt_status_t st = check_config(c, M, N, K, p, q, w_rowsum != nullptr);
  if (st != APT_OK) return st;
  *resolved = c;
  *layout = act_layout(M, N, K, p, q, fp16, c);
  return APT_OK;
}

}  // namespace apt

using apt::gemm_common;

extern "C" {

apt_status_t apt_gemm(int M, int N, int K, int p, int q, const void* a_packed, const void* w_packed,
                      const int32_t* a_rowsum, const int32_t* w_rowsum, int32_t* c_int32,
                      const uint16_t* a_scale, const uint16_t* w_scale, uint16_t* c_fp16,
                      const apt_config_t* cfg, void* workspace, size_t workspace_bytes,
                      void* stream) {
  return gemm_common(M, N, K, p, q, a_packed, w_packed, a_rowsum, w_rowsum, c_int32, a_scale,
                     w_scale, c_fp16, nullptr, nullptr, cfg, workspace, workspace_bytes, stream);
}

apt_status_t apt_gemm_affine(int M, int N, int K, int p, int q, const void* a_packed,
                             const void* w_packed, const int32_t* a_rowsum,
                             const int32_t* w_rowsum, const uint16_t* a_scale,
                             const uint16_t* a_zero, const uint16_t* w_scale,
                             const uint16_t* w_zero, uint16_t* c_fp16, int32_t* c_int32,
                             const apt_config_t* cfg, void* workspace, size_t workspace_bytes,
                             void* stream) {
  if (a_rowsum == nullptr || w_rowsum == nullptr || a_scale == nullptr || a_zero == nullptr ||
      w_scale == nullptr || w_zero == nullptr || c_fp16 == nullptr)
    return APT_ERR_INVALID_ARG;
  return gemm_common(M, N, K, p, q, a_packed, w_packed, a_rowsum, w_rowsum, c_int32, a_scale,
                     w_scale, c_fp16, a_zero, w_zero, cfg, workspace, workspace_bytes, stream);
}

size_t apt_gemm_act_workspace_bytes(int M, int N, int K, int p, int q, int a_kind,
                                    const apt_config_t* cfg) {
  if (M < 1 || N < 1 || K < 1 || !bits_ok(p) || !bits_ok(q)) return 0;
  if (a_kind != APT_ACT_CODES && a_kind != APT_ACT_FP16) return 0;
  const apt_config_t c = (cfg == nullptr || cfg->route == APT_ROUTE_AUTO)
                             ? apt::select_config(M, N, K, p, q)
                             : *cfg;
  if (check_config(c, M, N, K, p, q, true) != APT_OK) return 0;
  return apt::act_layout(M, N, K, p, q, a_kind == APT_ACT_FP16, c).total;
}

apt_status_t apt_gemm_act(int M, int N, int K, int p, int q, const void* a_src, int a_kind,
                          const void* w_packed, const int32_t* w_rowsum, int32_t* c_int32,
                          const uint16_t* a_scale, const uint16_t* w_scale, uint16_t* c_fp16,
                          uint16_t* a_scale_out, const apt_config_t* cfg, void* workspace,
                          size_t workspace_bytes, void* stream) {
  apt_config_t c;
  apt::ActLayout L;
  const apt_status_t st = apt::act_check(M, N, K, p, q, a_src, a_kind, w_packed, w_rowsum, c_int32,
                                         a_scale, w_scale, c_fp16, a_scale_out, cfg, &c, &L);
  if (st != APT_OK) return st;
  if (L.total > 0) {
    if (workspace == nullptr || workspace_bytes < L.total) return APT_ERR_WORKSPACE;
    if (!aligned16(workspace)) return APT_ERR_INVALID_ARG;
  }
  const bool fp16 = a_kind == APT_ACT_FP16;
  hipStream_t s = static_cast<hipStream_t>(stream);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  apt::GemmArgs g;
  g.M = M; g.N = N; g.K = K; g.p = p; g.q = q;
  g.a_packed = nullptr;
  g.w_packed = static_cast<const uint32_t*>(w_packed);
  g.a_rowsum = nullptr;
  g.w_rowsum = w_rowsum;
  g.c_int32 = c_int32;
  g.a_scale = reinterpret_cast<const __half*>(a_scale);
  g.w_scale = reinterpret_cast<const __half*>(w_scale);
  g.c_fp16 = reinterpret_cast<__half*>(c_fp16);
  g.a_zero = nullptr;
  g.w_zero = nullptr;
  if (L.plan == apt::ActPlan::kFusedXor)
    return hip_status(apt::launch_gemm_xor_act(g, a_src, fp16, a_scale_out, c, s));
  int32_t* rowsum = reinterpret_cast<int32_t*>(ws + L.rowsum_off);
  uint16_t* scale = reinterpret_cast<uint16_t*>(ws + L.scale_off);
  g.a_rowsum = rowsum;
  if (fp16) g.a_scale = reinterpret_cast<const __half*>(scale);
  if (L.plan == apt::ActPlan::kFragments) {
    const apt::ActSource src{a_src, fp16, rowsum, scale, a_scale_out};
    return hip_status(apt::launch_gemm_int8(g, c, ws, s, &src));
  }
  // the packer into the workspace, then the route on the packed rows (an fp16
  // source's scales go straight to the caller's array when there is one)
  uint32_t* planes = reinterpret_cast<uint32_t*>(ws + L.planes_off);
  if (a_scale_out != nullptr) scale = a_scale_out;
  const hipError_t e =
      fp16 ? apt::launch_quantize_pack(static_cast<const uint16_t*>(a_src), M, K, q, planes, rowsum,
                                       scale, s)
           : apt::launch_pack(static_cast<const int8_t*>(a_src), M, K, q, planes, rowsum, s);
  if (e != hipSuccess) return hip_status(e);
  return apt::gemm_launch(M, N, K, p, q, planes, w_packed, rowsum, w_rowsum, c_int32,
                          fp16 ? scale : a_scale, w_scale, c_fp16, nullptr, nullptr, c, ws,
                          L.route_bytes, stream);
}

apt_status_t apt_gemm_decode(int M, int N, int K, int p, int q, const void* a_src, int a_kind,
                             const void* w_packed, int32_t* c_int32, const uint16_t* a_scale,
                             const uint16_t* w_scale, uint16_t* c_fp16, uint16_t* a_scale_out,
                             const apt_config_t* cfg, void* stream) {
  if (M < 1 || M > APT_DECODE_MAX_M || N < 1 || K < 1 || !bits_ok(p) || !bits_ok(q))
    return APT_ERR_INVALID_ARG;
  if (a_kind != APT_ACT_CODES && a_kind != APT_ACT_FP16) return APT_ERR_INVALID_ARG;
  const bool fp16_src = a_kind == APT_ACT_FP16;
  if (a_src == nullptr || w_packed == nullptr || !aligned16(w_packed)) return APT_ERR_INVALID_ARG;
  if (fp16_src && (reinterpret_cast<uintptr_t>(a_src) & 1u) != 0) return APT_ERR_INVALID_ARG;
  if (c_int32 == nullptr && c_fp16 == nullptr) return APT_ERR_INVALID_ARG;
  if (c_fp16 != nullptr && (w_scale == nullptr || (!fp16_src && a_scale == nullptr)))
    return APT_ERR_INVALID_ARG;
  if (fp16_src ? a_scale != nullptr : a_scale_out != nullptr) return APT_ERR_INVALID_ARG;
  if (!fits_int32(K, p, q)) return APT_ERR_UNSUPPORTED;
  apt_config_t c{};
  c.route = APT_ROUTE_XOR;
  if (cfg != nullptr && cfg->route != APT_ROUTE_AUTO) {
    if (cfg->route != APT_ROUTE_XOR || !apt::xor_config_ok(*cfg)) return APT_ERR_INVALID_ARG;
    c = *cfg;
  }
  if (!apt::xor_act_sizes_ok(M, N, K, p, q, c, fp16_src)) return APT_ERR_UNSUPPORTED;
  apt::GemmArgs g;
  g.M = M; g.N = N; g.K = K; g.p = p; g.q = q;
  g.a_packed = nullptr;
  g.w_packed = static_cast<const uint32_t*>(w_packed);
  g.a_rowsum = nullptr;
  g.w_rowsum = nullptr;
  g.c_int32 = c_int32;
  g.a_scale = reinterpret_cast<const __half*>(a_scale);
  g.w_scale = reinterpret_cast<const __half*>(w_scale);
  g.c_fp16 = reinterpret_cast<__half*>(c_fp16);
  g.a_zero = nullptr;
  g.w_zero = nullptr;
  return hip_status(apt::launch_gemm_xor_act(g, a_src, fp16_src, a_scale_out, c,
                                             static_cast<hipStream_t>(stream)));
}

size_t apt_search_workspace_bytes(int M, int N, int K, int p, int q) {
  if (M < 1 || N < 1 || K < 1 || !bits_ok(p) || !bits_ok(q)) return 0;
  apt_config_t cand[apt::kMaxCandidates];
  const int n = apt::candidate_configs(M, N, K, p, q, cand, apt::kMaxCandidates);
  size_t most = 0;
  for (int i = 0; i < n; ++i)
    if (apt::mfma_route(cand[i].route) &&
        apt::int8_config_ok(cand[i], N))
      most = std::max(most, apt::int8_workspace_bytes(M, N, K, q, cand[i]));
  return most;
}

apt_status_t apt_search_config(int M, int N, int K, int p, int q, const void* a_packed,
                               const void* w_packed, const int32_t* a_rowsum,
                               const int32_t* w_rowsum, int32_t* c_int32, void* workspace,
                               size_t workspace_bytes, void* stream, apt_config_t* best,
                               float* best_us) {
  if (M < 1 || N < 1 || K < 1 || !bits_ok(p) || !bits_ok(q)) return APT_ERR_INVALID_ARG;
  if (a_packed == nullptr || w_packed == nullptr || !aligned16(a_packed) || !aligned16(w_packed) ||
      a_rowsum == nullptr || w_rowsum == nullptr || c_int32 == nullptr || best == nullptr)
    return APT_ERR_INVALID_ARG;
  if (!fits_int32(K, p, q)) return APT_ERR_UNSUPPORTED;
  const size_t need = apt_search_workspace_bytes(M, N, K, p, q);
  if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return APT_ERR_WORKSPACE;
  if (workspace != nullptr && !aligned16(workspace)) return APT_ERR_INVALID_ARG;

  apt_config_t cand[apt::kMaxCandidates];
  const int n = apt::candidate_configs(M, N, K, p, q, cand, apt::kMaxCandidates);
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipEvent_t e0 = nullptr, e1 = nullptr;
  hipError_t he = hipEventCreate(&e0);
  if (he != hipSuccess) return hip_status(he);
  he = hipEventCreate(&e1);
  if (he != hipSuccess) {
    (void)hipEventDestroy(e0);
    return hip_status(he);
  }
  constexpr int kWarm = 2, kTimed = 5;
  apt_status_t st = APT_OK;
  int best_i = -1;
  float best_t = 0.f;
  auto call = [&](const apt_config_t& c) {
    return gemm_common(M, N, K, p, q, a_packed, w_packed, a_rowsum, w_rowsum, c_int32, nullptr,
                       nullptr, nullptr, nullptr, nullptr, &c, workspace, workspace_bytes, stream);
  };
  for (int i = 0; i < n && st == APT_OK; ++i) {
    apt_status_t r = call(cand[i]);
    if (r == APT_ERR_HIP) {
      st = r;
      break;
    }
    if (r != APT_OK) continue;  // a candidate this problem cannot take
    for (int w = 1; w < kWarm && st == APT_OK; ++w) st = call(cand[i]);
    if (st != APT_OK) break;
    if ((he = hipEventRecord(e0, s)) != hipSuccess) {
      st = hip_status(he);
      break;
    }
    for (int t = 0; t < kTimed && st == APT_OK; ++t) st = call(cand[i]);
    float ms = 0.f;
    if (st != APT_OK) break;
    if ((he = hipEventRecord(e1, s)) != hipSuccess || (he = hipEventSynchronize(e1)) != hipSuccess ||
        (he = hipEventElapsedTime(&ms, e0, e1)) != hipSuccess) {
      st = hip_status(he);
      break;
    }
    const float us = ms * 1000.f / kTimed;
    if (best_i < 0 || us < best_t) {
      best_i = i;
      best_t = us;
    }
  }
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (st != APT_OK) return st;
  if (best_i < 0) return APT_ERR_UNSUPPORTED;
  apt::table_store(M, N, K, p, q, cand[best_i]);
  *best = cand[best_i];
  if (best_us != nullptr) *best_us = best_t;
  return APT_OK;
}

void apt_config_table_clear(void) { apt::table_clear(); }

int apt_config_table_size(void) { return apt::table_size(); }

int apt_last_hip_error(void) { return apt::t_last_hip_error; }

const char* apt_status_string(apt_status_t status) {
  switch (status) {
    case APT_OK: return "ok";
    case APT_ERR_INVALID_ARG: return "invalid argument";
    case APT_ERR_UNSUPPORTED: return "unsupported problem or configuration";
    case APT_ERR_HIP: return "HIP runtime error";
    case APT_ERR_WORKSPACE: return "workspace missing or too small";
  }
  return "unknown status";
}

}  // extern "C"
