// read_stream.hip - measurement probe (not part of libapt.so): a read-only
// reference for the decode GEMMs' weight streams.  Every byte of a buffer is
// read once with 16-byte loads, V per lane (lane t of the grid reads vectors
// t, t + T, ..., t + (V-1) T, T = threads in the grid, so a wave reads whole
// 1 KB segments), and folded with XOR into one word per workgroup, so that
// the loads cannot be dropped and the host can check the result (the XOR of
// the out words equals the XOR of every 32-bit word of the buffer).  With NT
// the loads carry the non-temporal hint.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kBlock = 256;
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

template <int V, bool NT>
__global__ __launch_bounds__(kBlock) void read_xor_kernel(const uint4* __restrict__ src, int64_t nvec,
                                                          uint32_t* __restrict__ out) {
  const int64_t T = (int64_t)gridDim.x * kBlock;
  const int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  uint4 v[V];
#pragma unroll
  for (int i = 0; i < V; ++i) {
    const int64_t idx = t + i * T;
    if (idx < nvec) {
      if (NT) {
        const v4u x = __builtin_nontemporal_load(reinterpret_cast<const v4u*>(src) + idx);
        v[i] = make_uint4(x[0], x[1], x[2], x[3]);
      } else {
        v[i] = src[idx];
      }
    } else
      v[i] = make_uint4(0u, 0u, 0u, 0u);
  }
  uint32_t x = 0u;
#pragma unroll
  for (int i = 0; i < V; ++i) x ^= v[i].x ^ v[i].y ^ v[i].z ^ v[i].w;
  for (int off = 32; off > 0; off >>= 1) x ^= __shfl_xor(x, off);
  __shared__ uint32_t red[kBlock / 64];
  if (threadIdx.x % 64 == 0) red[threadIdx.x / 64] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = 0u;
    for (int w = 0; w < kBlock / 64; ++w) r ^= red[w];
    out[blockIdx.x] = r;
  }
}

int64_t blocks_for(int64_t nvec, int v) { return (nvec + (int64_t)kBlock * v - 1) / ((int64_t)kBlock * v); }

template <int V, bool NT>
int launch(const void* src, int64_t nvec, uint32_t* out, hipStream_t s) {
  const uint4* a0 = static_cast<const uint4*>(src);
  void* args[] = {&a0, &nvec, &out};
  // the status of this launch alone (not an earlier call's leftover error)
  const hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(read_xor_kernel<V, NT>),
                                       dim3((unsigned)blocks_for(nvec, V)), dim3(kBlock), args, 0, s);
  return e == hipSuccess ? 0 : 3;
}

}  // namespace

// Workgroups (= out words) of apt_probe_read_xor for `bytes` bytes and v
// vectors per lane; 0 if bytes is not a positive multiple of 16.
extern "C" int64_t apt_probe_read_blocks(int64_t bytes, int v) {
  if (bytes <= 0 || bytes % 16 != 0 || v < 1) return 0;
  return blocks_for(bytes / 16, v);
}

// Enqueues the read of `bytes` bytes at device pointer src (16-byte aligned,
// bytes a multiple of 16) on `stream`, v = 1, 2, 4 or 8 vectors per lane, nt
// = 1 for non-temporal loads; out receives apt_probe_read_blocks(bytes, v)
// words.  Returns 0, 1 for bad arguments, or 3 on a launch error.
extern "C" int apt_probe_read_xor(const void* src, int64_t bytes, int v, int nt, uint32_t* out,
                                  void* stream) {
  if (src == nullptr || out == nullptr || bytes <= 0 || bytes % 16 != 0 ||
      (reinterpret_cast<uintptr_t>(src) & 15u) != 0)
    return 1;
  const int64_t nvec = bytes / 16;
  if (blocks_for(nvec, v) > 0x7fffffff) return 1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  switch (v * 2 + (nt ? 1 : 0)) {
    case 2: return launch<1, false>(src, nvec, out, s);
    case 3: return launch<1, true>(src, nvec, out, s);
    case 4: return launch<2, false>(src, nvec, out, s);
    case 5: return launch<2, true>(src, nvec, out, s);
    case 8: return launch<4, false>(src, nvec, out, s);
    case 9: return launch<4, true>(src, nvec, out, s);
    case 16: return launch<8, false>(src, nvec, out, s);
    case 17: return launch<8, true>(src, nvec, out, s);
  }
  return 1;
}
