// noalloc.hip - apt_gemm_noalloc: apt_gemm with its workspace in a fixed
// device array of the library instead of a caller buffer, for callers that
// cannot allocate device memory.
//
// `scratch` is a file-scope device array: each GPU the library runs on holds
// its own copy, at its own address, until the process ends.  In host code its
// name is only a host-side stand-in, so the device address is looked up once
// per device (hipGetSymbolAddress, with that device current) and that address
// is what the kernels receive.  Every call on a GPU shares that GPU's copy and
// leaves the last call's contents in it: the kernels overwrite the activation
// fragments, and the activation expansion clears the stream-K arrival
// counters, before anything reads them, so nothing carries over from one call
// to the next.  Calls that overlap in time on one GPU race on it.
#include <mutex>

#include "apt_internal.h"

namespace {

static_assert(APT_NOALLOC_SCRATCH_BYTES % 256 == 0, "whole 256-byte blocks");
static __device__ __align__(256) uint8_t scratch[APT_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices];  // device address of `scratch` per device ordinal

// Device address of `scratch` on the device `stream` runs on (the current
// device for the null stream), looked up on the first call for that device.
apt_status_t scratch_for(hipStream_t stream, void** out) {
  int cur = 0;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return apt::hip_status(e);
  int dev = cur;
  if (stream != nullptr) {
    e = hipStreamGetDevice(stream, &dev);
    if (e != hipSuccess) return apt::hip_status(e);
  }
  if (dev < 0 || dev >= kMaxDevices) return APT_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_scratch[dev] == nullptr) {
    // the lookup needs the stream's device current
    if (dev != cur && (e = hipSetDevice(dev)) != hipSuccess) return apt::hip_status(e);
    void* p = nullptr;
    const hipError_t le = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur && (e = hipSetDevice(cur)) != hipSuccess) return apt::hip_status(e);
    if (le != hipSuccess) return apt::hip_status(le);
    if (p == nullptr) return APT_ERR_HIP;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return APT_OK;
}

}  // namespace

extern "C" apt_status_t apt_gemm_noalloc(int M, int N, int K, int p, int q, const void* a_packed,
                                         const void* w_packed, const int32_t* a_rowsum,
                                         const int32_t* w_rowsum, int32_t* c_int32,
                                         const uint16_t* a_scale, const uint16_t* w_scale,
                                         uint16_t* c_fp16, const apt_config_t* cfg, void* stream) {
  apt_config_t c;
  apt_status_t st = apt::gemm_check(M, N, K, p, q, a_packed, w_packed, a_rowsum, w_rowsum, c_int32,
                                    a_scale, w_scale, c_fp16, cfg, &c);
  if (st != APT_OK) return st;
  size_t need = apt::gemm_workspace_need(M, N, K, q, c);
  const bool selected = cfg == nullptr || cfg->route == APT_ROUTE_AUTO;
  if (need > APT_NOALLOC_SCRATCH_BYTES && selected && (c.grid != 0 || c.tail_grid != 0)) {
    // The selected decomposition's stream-K partial tiles do not fit: the same
    // tiles with one workgroup per tile need only the activation fragments.
    c.grid = 0;
    c.tail_grid = 0;
    need = apt::gemm_workspace_need(M, N, K, q, c);
  }
  if (need > APT_NOALLOC_SCRATCH_BYTES) return APT_ERR_WORKSPACE;
  void* ws = nullptr;
  if (need > 0) {
    st = scratch_for(static_cast<hipStream_t>(stream), &ws);
    if (st != APT_OK) return st;
  }
  return apt::gemm_launch(M, N, K, p, q, a_packed, w_packed, a_rowsum, w_rowsum, c_int32, a_scale,
                          w_scale, c_fp16, nullptr, nullptr, c, ws, ws ? APT_NOALLOC_SCRATCH_BYTES : 0,
                          stream);
}
