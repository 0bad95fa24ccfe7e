// mfma_issue.hip - measurement probe (not part of libapt.so): how much each
// part of the MFMA GEMM loop's instruction pattern costs in MFMA issue on
// gfx950.  Every wave runs `chunks` chunks of 4 k-steps; a k-step issues 16
// independent v_mfma_i32_32x32x32_i8 (4 A x 4 B fragments, 16 accumulators)
// on top of which each mode adds one part of the prefill kernel's loop:
//   0  nothing (registers only)
//   1  4 LDS reads of the next k-step's A fragments (double-buffered)
//   2  mode 1 + one workgroup barrier per chunk
//   3  mode 2 + 4 buffer loads of 16 bytes per lane per k-step into the B
//      fragments, a chunk ahead of their use (the activation fragments)
//   4  mode 2 + 4 buffer loads of 4 bytes per lane per k-step
//   5  mode 2 + 2 buffer loads of 16 bytes per lane per k-step
//   6  mode 2 + 4 buffer loads of 16 bytes per lane per k-step straight into
//      LDS, read back one k-step ahead
// Modes 0-6 run one wave per SIMD (256 workgroups of 4 waves, accumulators in
// AGPRs).  Mode 7 is mode 3's per-SIMD pattern on two waves per SIMD (8 waves
// per workgroup, each with 2 B fragments: 8 MFMAs and 2 loads per k-step).
// Lane 0 of each wave reads the shader clock counter (s_memtime) and the
// 100 MHz constant counter (s_memrealtime) around its loop; the host averages
// them into cycles per MFMA per SIMD and the shader clock.
// Operands come from one host-generated buffer (registers, LDS and the load
// buffer) of pseudo-random bytes, sparse bytes, 4-bit bipolar values or 4-bit
// codes: the shader clock under dense MFMA work depends on how many operand
// bits switch.  Each wave ends by summing every element of each
// accumulator over its lanes; for mode 0, whose operands never change, the
// host checks every wave's sums against a closed form: the sum of all
// elements of A.B is sum_k colsum_A(k) * rowsum_B(k), and in the operand
// layout of v_mfma_i32_32x32x32_i8 byte j of lane l holds the same k in both
// operands, shared by the 32 lanes of one half of the wave, so
// sum(C) = sum over halves h and bytes j of (sum of A's byte j over half h) *
// (sum of B's byte j over half h), whatever k each (h, j) stands for.  The
// accumulators and sums wrap modulo 2^32 on both sides.
#include <hip/hip_runtime.h>

#include <vector>

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kLdsVecs = 512 + 4 * 2 * 16 * 64;  // A fragments + the mode-6 ring (136 KB)

template <int MODE, int FM, int WAVES>
__global__ __launch_bounds__(WAVES * 64, 1) void issue_kernel(int chunks, const v4i* __restrict__ src,
                                                              int nvec, unsigned long long* out,
                                                              int* sums) {
  extern __shared__ v4i dyn[];
  v4i* al = dyn + 512;
  const int lane = threadIdx.x % 64, wave = threadIdx.x / 64;
  const int wu = __builtin_amdgcn_readfirstlane(wave);  // uniform in the wave
  for (int i = threadIdx.x; i < 512; i += blockDim.x) dyn[i] = src[i];
  __syncthreads();
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<v4i*>(src), 0, nvec * 16, 0x00020000);
  v16i acc[4][FM];
  for (int b = 0; b < 4; ++b)
    for (int a = 0; a < FM; ++a)
      for (int v = 0; v < 16; ++v) acc[b][a][v] = 0;
  v4i wf[2][4], af[4][FM], an[2][FM];
  // initial operands: vectors [0, 512) of the buffer for wf, [512, 1024) for af, then an
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int b = 0; b < 4; ++b) wf[x][b] = src[(x * 4 + b) * 64 + lane];
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int a = 0; a < FM; ++a) af[k][a] = src[512 + (k * FM + a) * 64 + lane];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int a = 0; a < FM; ++a) an[x][a] = src[1024 + (x * FM + a) * 64 + lane];
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  for (int c = 0; c < chunks; ++c) {
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int cur = ks & 1, nxt = cur ^ 1;
      if (MODE >= 1) {
#pragma unroll
        for (int b = 0; b < 4; ++b) wf[nxt][b] = dyn[(b * 128 + ((ks + 1) & 1) * 64 + lane) & 511];
      }
      if (MODE == 6) {
        const int slot = (c + (ks + 1) / 4) & 1, kn = (ks + 1) & 3;
#pragma unroll
        for (int a = 0; a < FM; ++a) an[nxt][a] = al[((wave * 2 + slot) * 16 + kn * 4 + a) * 64 + lane];
      }
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int a = 0; a < FM; ++a)
          acc[b][a] = __builtin_amdgcn_mfma_i32_32x32x32_i8(wf[cur][b], MODE == 6 ? an[cur][a] : af[ks][a],
                                                            acc[b][a], 0, 0, 0);
      // wave-uniform byte offset of this k-step's B fragments, inside the first half of the buffer
      const uint32_t base = ((uint32_t)(((c + 1) * 16 + ks * 4 + (wu & 1) * 2) * 64) & (uint32_t)(nvec / 2 - 1)) * 16u;
      if (MODE == 3 || MODE == 7) {
#pragma unroll
        for (int a = 0; a < FM; ++a)
          af[ks][a] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(rs, lane * 16, base + a * 1024, 0));
      } else if (MODE == 4) {
#pragma unroll
        for (int a = 0; a < FM; ++a)
          af[ks][a][0] = (int)__builtin_amdgcn_raw_buffer_load_b32(rs, lane * 16, base + a * 1024, 0);
      } else if (MODE == 5) {
#pragma unroll
        for (int a = 0; a < FM / 2; ++a)
          af[ks][a] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(rs, lane * 16, base + a * 1024, 0));
      } else if (MODE == 6) {
        const int slot = (c + 1) & 1;
#pragma unroll
        for (int a = 0; a < FM; ++a)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              rs, (__attribute__((address_space(3))) void*)(al + ((wave * 2 + slot) * 16 + ks * 4 + a) * 64), 16,
              lane * 16, base + a * 1024, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if (MODE == 6) __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    if (MODE >= 2) __syncthreads();
  }
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
  const int w = blockIdx.x * WAVES + wave;
  // fully unrolled: an index into acc that is not a constant would put it in scratch memory
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int a = 0; a < FM; ++a) {
      uint32_t s = 0;
#pragma unroll
      for (int v = 0; v < 16; ++v) s += (uint32_t)acc[b][a][v];
#pragma unroll
      for (int m = 32; m >= 1; m /= 2) s += (uint32_t)__shfl_xor((int)s, m);
      if (lane == 0) sums[w * 16 + b * 4 + a] = (int)s;
    }
  if (lane == 0) {
    out[4 * w + 0] = t0;
    out[4 * w + 1] = t1;
    out[4 * w + 2] = r0;
    out[4 * w + 3] = r1;
  }
}

// Mode 0's closed form (see the header): the sum of every element of
// accumulator (b, a) after `chunks` chunks, modulo 2^32, from the buffer's
// bytes.  Operand A of k-step ks is wf[ks % 2][b] (vectors (ks % 2) * 4 + b),
// operand B is af[ks][a] (vectors 512 + (ks * FM + a) * 64).
template <int FM>
uint32_t mode0_sum(const std::vector<int8_t>& bytes, int b, int a, int chunks) {
  auto half_col = [&](int vec0, int h, int j) {  // sum of byte j over lanes 32h .. 32h + 31
    int64_t s = 0;
    for (int l = 32 * h; l < 32 * h + 32; ++l) s += bytes[(size_t)(vec0 + l) * 16 + j];
    return s;
  };
  int64_t per_chunk = 0;
  for (int ks = 0; ks < 4; ++ks)
    for (int h = 0; h < 2; ++h)
      for (int j = 0; j < 16; ++j)
        per_chunk += half_col(((ks % 2) * 4 + b) * 64, h, j) * half_col(512 + (ks * FM + a) * 64, h, j);
  return (uint32_t)((uint64_t)per_chunk * (uint64_t)chunks);
}

template <int MODE, int FM, int WAVES>
int run(int blocks, int chunks, int data, double* res) {
  constexpr int nvec = 1 << 16;  // 1 MB of B fragments (cache-resident); a power of two
  v4i* src = nullptr;
  unsigned long long* out = nullptr;
  int* sums = nullptr;
  const int waves = blocks * WAVES;
  std::vector<int8_t> bytes((size_t)nvec * 16);
  uint64_t x = 0x9E3779B97F4A7C15ull;  // xorshift64
  for (size_t i = 0; i < bytes.size(); ++i) {
    x ^= x << 13;
    x ^= x >> 7;
    x ^= x << 17;
    // 1: one small byte per dword, the rest zero (few bits switch); 2: odd values in
    // [-15, 15], 4-bit bipolar values as int8; 3: bytes in [0, 15], the 4-bit
    // codes the reassembled int8 route multiplies; 0: any byte
    bytes[i] = data == 1   ? (int8_t)(i % 4 == 0 ? (x >> 58) : 0)
               : data == 2 ? (int8_t)(2 * (int)(x >> 60) - 15)
               : data == 3 ? (int8_t)(x >> 60)
                           : (int8_t)(x >> 56);
  }
  int rc = 0;
  if (hipMalloc(&src, sizeof(v4i) * nvec) != hipSuccess ||
      hipMalloc(&out, sizeof(unsigned long long) * 4 * waves) != hipSuccess ||
      hipMalloc(&sums, sizeof(int) * 16 * waves) != hipSuccess ||
      hipMemcpy(src, bytes.data(), bytes.size(), hipMemcpyHostToDevice) != hipSuccess)
    rc = 1;
  const size_t lds = (size_t)kLdsVecs * 16;
  auto kern = issue_kernel<MODE, FM, WAVES>;
  if (!rc && hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                 hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    rc = 2;
  std::vector<unsigned long long> h(4 * (size_t)waves);
  for (int rep = 0; rep < 2 && !rc; ++rep) {  // the first run warms up; the second is reported
    hipLaunchKernelGGL(kern, dim3(blocks), dim3(WAVES * 64), lds, 0, chunks, src, nvec, out, sums);
    if (hipGetLastError() != hipSuccess || hipDeviceSynchronize() != hipSuccess) rc = 3;
  }
  if (!rc && hipMemcpy(h.data(), out, h.size() * 8, hipMemcpyDeviceToHost) != hipSuccess) rc = 4;
  std::vector<int> hs(16 * (size_t)waves);
  if (!rc && hipMemcpy(hs.data(), sums, hs.size() * sizeof(int), hipMemcpyDeviceToHost) != hipSuccess) rc = 4;
  res[3] = 0.0;  // 1: every wave's sums checked against the closed form (mode 0)
  if (!rc && MODE == 0) {
    for (int w = 0; w < waves && !rc; ++w)
      for (int b = 0; b < 4; ++b)
        for (int a = 0; a < FM; ++a)
          if ((uint32_t)hs[w * 16 + b * 4 + a] != mode0_sum<FM>(bytes, b, a, chunks)) rc = 5;
    if (!rc) res[3] = 1.0;
  }
  if (!rc) {
    double cyc = 0, real = 0;
    for (int w = 0; w < waves; ++w) {
      cyc += (double)(h[4 * w + 1] - h[4 * w]);
      real += (double)(h[4 * w + 3] - h[4 * w + 2]);
    }
    cyc /= waves;
    real /= waves;
    const double mfmas_per_simd = (double)chunks * 4 * 4 * FM * (WAVES / 4);
    res[0] = cyc / mfmas_per_simd;          // shader cycles per MFMA per SIMD
    res[1] = cyc / (real / 100e6) / 1e9;     // shader clock, GHz
    res[2] = real / 100.0 / chunks;          // microseconds per chunk
  }
  (void)hipFree(src);
  (void)hipFree(out);
  (void)hipFree(sums);
  return rc;
}

}  // namespace

// Runs probe mode `mode` (0-7) for `chunks` chunks on `blocks` workgroups,
// on pseudo-random operand bytes (data = 0), on bytes of which only the low
// byte of each dword is nonzero and small (data = 1), on random odd bytes in
// [-15, 15] (data = 2: 4-bit bipolar values) or on random bytes in [0, 15]
// (data = 3: the 4-bit codes the reassembled int8 route multiplies), and writes cycles
// per MFMA per SIMD, the shader clock (GHz) and microseconds per chunk to
// res[0..2], and to res[3] 1 if the accumulators were checked (mode 0) and 0
// otherwise.  Returns 0, a nonzero step number on a HIP error, or 5 if mode
// 0's sums differ from the closed form.
extern "C" int apt_probe_mfma_issue(int mode, int blocks, int chunks, int data, double* res) {
  switch (mode) {
    case 0: return run<0, 4, 4>(blocks, chunks, data, res);
    case 1: return run<1, 4, 4>(blocks, chunks, data, res);
    case 2: return run<2, 4, 4>(blocks, chunks, data, res);
    case 3: return run<3, 4, 4>(blocks, chunks, data, res);
    case 4: return run<4, 4, 4>(blocks, chunks, data, res);
    case 5: return run<5, 4, 4>(blocks, chunks, data, res);
    case 6: return run<6, 4, 4>(blocks, chunks, data, res);
    case 7: return run<7, 2, 8>(blocks, chunks, data, res);
  }
  return 99;
}
