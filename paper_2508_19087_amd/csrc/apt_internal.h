// apt_internal.h - definitions shared by the gfx950 kernels and the C ABI of
// the WpAq bipolar-INT GEMM library.  Not part of the public interface.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

#include <tuple>
#include <utility>

#include "../../include/apt.h"

namespace apt {

// Packed layout (fixed in apt.h): 128 elements per chunk, 4 uint32 words per
// plane per chunk; rows in groups of 8, and for each group and chunk the b
// planes follow each other, each plane holding the 8 rows' 4 words.
constexpr int kChunk = 128;
constexpr int kWordsPerPlane = 4;
constexpr int kRowGroup = 8;
constexpr int kPlaneStride = kRowGroup * kWordsPerPlane;  // words from plane i to plane i+1

inline int num_chunks(int K) { return (K + kChunk - 1) / kChunk; }

// Launches kernel k on `stream` and returns the status of this launch alone.
// (A launch followed by hipGetLastError would also report an error that an
// earlier, unrelated runtime call of the thread left behind.)  The arguments
// are converted to the kernel's parameter types and passed by address.
template <typename... P, typename... A>
inline hipError_t launch_kernel(void (*k)(P...), dim3 grid, dim3 block, size_t lds,
                                hipStream_t stream, A&&... args) {
  static_assert(sizeof...(P) == sizeof...(A), "one argument per kernel parameter");
  std::tuple<P...> vals(std::forward<A>(args)...);
  void* ptrs[sizeof...(P) > 0 ? sizeof...(P) : 1];
  std::apply([&ptrs](auto&... v) {
    int i = 0;
    ((ptrs[i++] = static_cast<void*>(&v)), ...);
  }, vals);
  return hipLaunchKernel(reinterpret_cast<const void*>(k), grid, block, ptrs, lds, stream);
}

// The FP4 MFMA route applies to (p, q) over K: E2M1 holds bipolar weights of
// at most 2 bits, E2M1 (q <= 2) or E4M3 (q <= 4) the activations, and the
// fp32 sums stay exact while no partial sum can reach 2^24 in magnitude.  The
// MFMAs also sum the padding elements of the last chunk (each -(2^p - 1)
// times -(2^q - 1)), so the bound is on the padded K.
inline bool fp4_route_ok(int K, int p, int q) {
  return p <= 2 && q <= 4 &&
         (int64_t)num_chunks(K) * kChunk * ((1 << p) - 1) * ((1 << q) - 1) < ((int64_t)1 << 24);
}
// The FP6 MFMA route applies to (p, q) over K: E2M3 holds bipolar values of
// at most 3 bits, and the fp32 sums stay exact as for the FP4 route.
inline bool fp6_route_ok(int K, int p, int q) {
  return p <= 3 && q <= 3 &&
         (int64_t)num_chunks(K) * kChunk * ((1 << p) - 1) * ((1 << q) - 1) < ((int64_t)1 << 24);
}
// The FP8 MFMA route applies to (p, q) over K: E4M3 holds bipolar values of
// at most 4 bits, and the fp32 sums stay exact as for the FP4 route.
inline bool fp8_route_ok(int K, int p, int q) {
  return p <= 4 && q <= 4 &&
         (int64_t)num_chunks(K) * kChunk * ((1 << p) - 1) * ((1 << q) - 1) < ((int64_t)1 << 24);
}
// Routes that run the reassembled MFMA kernels (operand formats int8, FP4, FP6, FP8).
inline bool mfma_route(int route) {
  return route == APT_ROUTE_INT8_MFMA || route == APT_ROUTE_FP4_MFMA || route == APT_ROUTE_FP6_MFMA ||
         route == APT_ROUTE_FP8_MFMA;
}
inline int padded_rows(int R) { return (R + kRowGroup - 1) / kRowGroup * kRowGroup; }

// Word offset of the 4 words of plane i, chunk c, row r.
__host__ __device__ __forceinline__ int64_t plane_words(int r, int c, int i, int nchunks, int bits) {
  return ((int64_t)(r / kRowGroup) * nchunks + c) * bits * kPlaneStride + i * kPlaneStride +
         (r % kRowGroup) * kWordsPerPlane;
}

// Launch of the converter + bit-plane packer (pack.hip).
hipError_t launch_pack(const int8_t* codes, int rows, int K, int bits, uint32_t* packed,
                       int32_t* rowsum, hipStream_t stream);
// Per-row quantization of fp16 rows to b-bit bipolar codes, then the same
// packing; writes the fp16 bits of each row's bipolar scale to scale[row]
// (pack.hip).
hipError_t launch_quantize_pack(const uint16_t* x, int rows, int K, int bits, uint32_t* packed,
                                int32_t* rowsum, uint16_t* scale, hipStream_t stream);

// Arguments every GEMM route receives (device pointers; validated by the ABI).
struct GemmArgs {
  int M, N, K, p, q;
  const uint32_t* a_packed;
  const uint32_t* w_packed;
  const int32_t* a_rowsum;
  const int32_t* w_rowsum;
  int32_t* c_int32;
  const __half* a_scale;
  const __half* w_scale;
  __half* c_fp16;
  // Zero-points of the fp16 epilogue (both set or both NULL); with them the
  // row sums are required.
  const __half* a_zero;
  const __half* w_zero;
};

// fp16 epilogue value (float32 arithmetic; the caller rounds to fp16) of an
// output C of two linear quantizers in bipolar form (Sec. III-A: scale s/2,
// zero z - s/2): s_a s_w C + s_a z_w R_a + z_a (s_w R_w + K z_w), with
// `colterm` = s_w R_w + K z_w precomputed per output column.
__device__ __forceinline__ float affine_value(int32_t c, float sa, float sw, float zw, float ra,
                                              float za, float colterm) {
  return sa * (sw * (float)c + zw * ra) + za * colterm;
}

// XOR + popcount route (gemm_xor.hip).  Any shape.
hipError_t launch_gemm_xor(const GemmArgs& g, const apt_config_t& cfg, hipStream_t stream);
bool xor_config_ok(const apt_config_t& cfg);
bool xor_sizes_ok(int M, int N, int K, int p, int q, const apt_config_t& cfg);
// XOR route with the activation rows converted inside the kernel from int8
// codes or (fp16_src) fp16 values; a_scale_out receives the fp16 source's
// per-row scales (or NULL).  The rows' LDS copy must fit (xor_act_sizes_ok).
hipError_t launch_gemm_xor_act(const GemmArgs& g, const void* a_src, bool fp16_src,
                               uint16_t* a_scale_out, const apt_config_t& cfg, hipStream_t stream);
bool xor_act_sizes_ok(int M, int N, int K, int p, int q, const apt_config_t& cfg, bool fp16_src);

// Activations given unpacked (int8 codes, or fp16 values quantized per row)
// to a route that builds its operand bytes itself: the int8-format MFMA route
// writes its fragments, row sums (and fp16 scales) straight from them
// (act_frag.hip).
struct ActSource {
  const void* data;    // [M][K] int8 codes or fp16 bits
  bool fp16;
  int32_t* rowsum;     // device [M]: receives the row sums
  uint16_t* scale;     // device [M]: receives the fp16 source's scales
  uint16_t* scale_out; // device [M] or NULL: a copy of them for the caller
};
hipError_t launch_act_frag(const void* src, bool fp16, int M, int K, int q, int nsteps, void* frag,
                           int32_t* rowsum, uint16_t* scale, uint16_t* scale_out, int* counters,
                           int ncounters, hipStream_t s);

// Reassembled int8 MFMA route (gemm_int8.hip).  The workspace holds the
// activations expanded into MFMA fragments (int8_workspace_bytes): from the
// packed planes (src NULL), or, with the int8 operand format only, from an
// unpacked source (g.a_rowsum and g.a_scale must then name src's outputs).
hipError_t launch_gemm_int8(const GemmArgs& g, const apt_config_t& cfg, void* workspace,
                            hipStream_t stream, const ActSource* src = nullptr);
// Operand format of the activations in a config of the MFMA routes (0: int8).
int int8_operand_format(const apt_config_t& cfg, int q);
constexpr int kMaxGrid = 4096;  // persistent workgroups of the int8 route, at most
bool int8_config_ok(const apt_config_t& cfg, int N);
bool int8_sizes_ok(int M, int N, int K, int p, int q, const apt_config_t& cfg);
size_t int8_workspace_bytes(int M, int N, int K, int q, const apt_config_t& cfg);

// Plane-pair +-1 MFMA route (gemm_pm1.hip).
hipError_t launch_gemm_pm1(const GemmArgs& g, const apt_config_t& cfg, hipStream_t stream);
bool pm1_config_ok(const apt_config_t& cfg, int p, int q);
bool pm1_sizes_ok(int M, int N);

// Maps a runtime status to the library's (APT_OK or APT_ERR_HIP, recording
// the code for apt_last_hip_error) (api.hip).
apt_status_t hip_status(hipError_t e);

// The GEMM entry points' common steps (api.hip).  gemm_check validates
// everything but the workspace (sizes, bit widths, pointers, outputs, the
// int32 bound, the config) and resolves the config (cfg NULL or AUTO: the
// selected one); gemm_workspace_need gives the workspace bytes of a
// resolved config; gemm_launch checks the workspace and launches;
// gemm_common is the three in a row.  a_zero / w_zero NULL for the scale
// epilogue.
apt_status_t gemm_check(int M, int N, int K, int p, int q, const void* a_packed,
                        const void* w_packed, const int32_t* a_rowsum, const int32_t* w_rowsum,
                        const int32_t* c_int32, const uint16_t* a_scale, const uint16_t* w_scale,
                        const uint16_t* c_fp16, const apt_config_t* cfg, apt_config_t* resolved);
size_t gemm_workspace_need(int M, int N, int K, int q, const apt_config_t& c);
apt_status_t gemm_launch(int M, int N, int K, int p, int q, const void* a_packed,
                         const void* w_packed, const int32_t* a_rowsum, const int32_t* w_rowsum,
                         int32_t* c_int32, const uint16_t* a_scale, const uint16_t* w_scale,
                         uint16_t* c_fp16, const uint16_t* a_zero, const uint16_t* w_zero,
                         const apt_config_t& c, void* workspace, size_t workspace_bytes,
                         void* stream);
apt_status_t gemm_common(int M, int N, int K, int p, int q, const void* a_packed,
                         const void* w_packed, const int32_t* a_rowsum, const int32_t* w_rowsum,
                         int32_t* c_int32, const uint16_t* a_scale, const uint16_t* w_scale,
                         uint16_t* c_fp16, const uint16_t* a_zero, const uint16_t* w_zero,
                         const apt_config_t* cfg, void* workspace, size_t workspace_bytes,
                         void* stream);

// Host-side selector (select.hip): the search module's table first, then the
// model.
apt_config_t select_config(int M, int N, int K, int p, int q);
bool table_lookup(int M, int N, int K, int p, int q, apt_config_t* out);
// The shipped table of searched configs with approximate matching.
bool shipped_lookup(int M, int N, int K, int p, int q, apt_config_t* out);
int shipped_table_size();
void table_store(int M, int N, int K, int p, int q, const apt_config_t& c);
void table_clear();
int table_size();
// Configs the search module times for a problem (at most max_out of them).
constexpr int kMaxCandidates = 64;  // bound checked in select.hip
int candidate_configs(int M, int N, int K, int p, int q, apt_config_t* out, int max_out);

}  // namespace apt
