// gemm_int8.h - the reassembled-int8 MFMA route of the WpAq bipolar-INT
// GEMM for gfx950 (APT-LLM, arXiv 2508.19087, Sec. III-B and IV-B).
//
// The bit-planes of each operand are merged back into one byte per element
// before the multiply (reassemble.h), so one v_mfma_i32_32x32x32_i8 covers
// every plane pair of an element pair; the paper's Sec. III-B sum over plane
// products is the same number by distributivity.
//
// Kernels:
//   expand_a_kernel  once per call, the activations' planes are reassembled
//                    into operand bytes laid out as ready-made MFMA fragments
//                    (a workspace buffer), so the main kernel loads them with
//                    whole-line 1 KB reads straight into registers;
//   gemm_int8_kernel persistent workgroups walking whole tiles and stream-K
//                    shares of tiles (gemm_int8_body); a tile part covers
//                    every plane pair of its outputs, as the paper's
//                    recovery-oriented scheduling does (Sec. IV-B);
//   gemm_int8_pair_kernel two such launches (main and tail tile shapes) in
//                    one grid.
// In the body, K advances one 128-element chunk per pipeline step over a
// 3-stage LDS ring: while the matrix cores work on chunk c, the weight planes
// of chunk c+2 (fetched one step earlier) are reassembled into the free
// stage, those of chunk c+3 are fetched, the activation fragments of chunk
// c+1 are fetched k-step by k-step behind the MFMAs, and the first weight
// fragments of chunk c+1 are read from LDS before the step's barrier.
// Only the weights pass through LDS: staging both operands there would need
// as many LDS bytes per chunk as the MFMAs take cycles, and LDS would bound
// the kernel.
//
// Operand bytes are y = u (b <= 7) or u - 128 (b == 8) with bipolar value
// v = 2y + c.  Expanding sum_k v_a v_w over the real K gives the epilogue
//   C = 4 D - 4 (K_pad - K) y_pad,a y_pad,w + c_w R_a[m] + c_a R_w[n] - c_a c_w K,
// where D is the MFMA sum over K_pad = 128 NC, y_pad the operand byte of a
// padding element, and R the row sums of bipolar values from the packers.
// The main loop runs an even number of chunks; a last odd chunk has all-zero
// activation bytes, so whatever weight bytes meet it add nothing to D.  The
// arithmetic is done modulo 2^32; the true C fits in int32 (checked by the
// host), so the wrapped result is exact.
#pragma once

#include <algorithm>

#include "apt_internal.h"
#include "reassemble.h"

namespace apt {
namespace int8 {

constexpr int kWave = 64;
constexpr int kStepBytes = 32;                  // operand bytes per row and MFMA k-step
constexpr int kFragVecs = kWave;                // one 32x32 fragment = 64 lanes x 16 bytes

// Operand format of the contraction (template parameter F):
//   F = 0: int8 operand bytes, one v_mfma_i32_32x32x32_i8 per 32 elements of k;
//   F = 1: FP4 (E2M1) operand nibbles for weights and activations of at most 2
//          bits, one v_mfma_scale_f32_32x32x64_f8f6f4 (unit scales) per 64
//          elements of k: the same operand bytes and issue cycles per MFMA as
//          int8 for twice the multiply-adds;
//   F = 2: FP4 weights (at most 2 bits) with FP8 (E4M3) activation bytes (at
//          most 4 bits: every odd value up to 15 is exact in E4M3), the same
//          MFMA with a mixed operand format, 64 elements of k per MFMA at
//          about 1.15x the int8 multiply-add rate (register-only loop).
// With F > 0 the fp32 sums are exact integers while K_pad (2^p - 1)(2^q - 1)
// < 2^24, K_pad = K rounded up to a chunk (the host checks).
// Per chunk, k-step ks of lane half h holds (F = 0) half h of word ks's bytes,
// or (F > 0) word 2 ks + h's weight nibbles; nibble 8 t + f is element 4 f + t
// of the word.  The FP8 operand covers k in 16-element blocks: lane half h
// holds elements 16 h .. 16 h + 15 of the k-step's first 32 in bytes 0..15
// and of its second 32 in bytes 16..31, which puts nibble n of word 2 ks + x
// (n = 16 h + j) against byte 16 x + j of lane half h.
//   F = 3: FP6 (E2M3) weights and activations of at most 3 bits, the same
//          MFMA with both operands in the six-bit format (24 operand bytes per
//          lane and k-step, 64 elements of k per MFMA).  Each lane half's 24
//          bytes sit in a 32-byte slot of the LDS row and in two 16-byte
//          fragment vectors (the second half-used).
//   F = 4: FP8 (E4M3) weights and activations of at most 4 bits, the same
//          MFMA with both operands in E4M3 (32 operand bytes per lane and
//          k-step, 64 elements of k per MFMA, the int8 multiply-add rate):
//          lane half h of k-step ks holds the 32 bytes of word 2 ks + h in the
//          order of the int8 byte tree, on both sides, so equal elements meet.
template <int F>
struct Fmt {
  static constexpr int kStepK = F ? 64 : 32;                   // k per MFMA
  static constexpr int kSteps = kChunk / kStepK;               // k-steps per chunk
  static constexpr int kStepRowBytes = F >= 3 ? 2 * kStepBytes : kStepBytes;  // LDS row bytes per k-step
  static constexpr int kHalfBytes = kStepRowBytes / 2;         // per lane half
  static constexpr int kRowBytes = kSteps * kStepRowBytes + 16;  // padded LDS row of a chunk
  static constexpr int kAVecs = F >= 2 ? 2 : 1;                // 16-byte activation vectors per lane and k-step
};
constexpr int kStages = 3;                      // weight LDS ring depth

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v2i __attribute__((ext_vector_type(2)));
typedef float v16f __attribute__((ext_vector_type(16)));

typedef uint32_t v2u __attribute__((ext_vector_type(2)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

// One 16-byte streaming global store of output bytes (written once, not
// re-read).  As a plain store the compiler shares the first element's store
// with the element-wise edge path and splits the vector into 12 + 4 bytes.
__device__ __forceinline__ void store16(int32_t* p, v4i v) {
  __builtin_nontemporal_store(v, reinterpret_cast<v4i*>(p));
}

// An empty instruction that reads x: code computing x cannot be moved past it.
__device__ __forceinline__ void keep_here(const v16i& x) { asm volatile("" ::"v"(x)); }
__device__ __forceinline__ void keep_here(const v4i& x, uint32_t y) { asm volatile("" ::"v"(x), "v"(y)); }

// Buffer resource over [base, base + bytes) for raw buffer loads: a
// wave-uniform base in SGPRs plus a per-lane 32-bit offset and a uniform
// offset, so the loop's address arithmetic is a scalar add per chunk.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, 0x00020000);
}

struct Int8Params {
  GemmArgs g;
  int nchunks;        // NC, chunks of K
  int nsteps;         // k-steps in the activation fragment buffer (even chunk count x 4)
  int mblocks;        // 32-row blocks of the activation fragment buffer
  const v4i* a_frag;  // activation fragments (workspace)
  uint32_t a_bytes;   // bytes of the activation fragment buffer
  uint32_t w_bytes;   // bytes of the packed weights
  int n_begin;        // first output column of this launch's tile grid
  int tiles_n;        // tiles per row of the tile grid
  int tiles;          // BM x BN tiles
  int dp_tiles;       // whole tiles per workgroup (the first dp_tiles * G tiles)
  int sk_pairs;       // chunk pairs of the stream-K tiles (the last ones), shared evenly
  int sk_grid;        // workgroups [0, sk_grid) share them
  v4i* partial;       // stream-K: two partial tiles per workgroup (workspace)
  uint32_t partial_bytes;
  int* counters;      // stream-K: arrivals per stream-K tile (workspace, zeroed per call)
  int vec_out;        // outputs take 16-byte (int32) / 8-byte (fp16) row stores
};

// Bytes of the activation fragment buffer for M rows and K in operand format
// fmt (F = 1: nibbles, otherwise bytes).
inline size_t a_frag_bytes(int M, int K, int fmt = 0) {
  const int nce = (num_chunks(K) + 1) & ~1;
  return (size_t)((M + 31) / 32) * 32 * nce * (fmt == 1 ? kChunk / 2 : kChunk);
}

// E4M3 bits of the bipolar value 2u - (2^Q - 1) (Q <= 4: odd, |v| <= 15).
template <int Q>
__device__ __forceinline__ uint32_t e4m3_bipolar(uint32_t u) {
  static_assert(Q <= 4, "E4M3 holds bipolar values of at most 4 bits exactly");
  const int v = 2 * (int)u - ((1 << Q) - 1);
  const int a = v < 0 ? -v : v;
  // |v| = 1, 3, ..., 15: exponent field 7 + floor(log2 |v|), 3 mantissa bits
  const int e = a >= 8 ? 3 : a >= 4 ? 2 : a >= 2 ? 1 : 0;
  const uint32_t bits = (uint32_t)(((e + 7) << 3) | (((a << 3) >> e) & 7));
  return v < 0 ? bits | 0x80u : bits;
}

// ---- activation expansion ---------------------------------------------------
// Fragment (mb, ks) holds k-step ks of rows 32 mb .. 32 mb + 31 in MFMA operand
// order: lane l (vector index ((mb * nsteps + ks) * 64 + l)) carries 16 bytes of
// row 32 mb + l mod 32, namely bytes 16 (l / 32) .. 16 (l / 32) + 15 of the
// k-step's 32 reassembled bytes (F = 1: the 16 nibble bytes of one plane
// word).  F = 2: two 16-byte vectors per lane, ((mb * nsteps + ks) * 2 + x) *
// 64 + l, with the E4M3 bytes of word 2 ks + x that lane half l / 32 meets
// (Fmt).  Rows past M are expanded from all-zero planes (padding elements); a
// chunk past the last one (the odd chunk that makes the count even) is
// all-zero bytes, which are 0 in every format.
template <int Q, int F>
__global__ __launch_bounds__(256) void expand_a_kernel(const uint32_t* __restrict__ a_packed, int M,
                                                       int nchunks, int nsteps, int mblocks,
                                                       v4i* __restrict__ out, int* __restrict__ counters,
                                                       int ncounters) {
  // One thread per (word w, row) of chunk blockIdx.y, w fastest: 4 threads
  // read one row's 16 contiguous bytes of a plane, so a wave reads whole
  // 128-byte lines.  (A two-dimensional grid keeps the index arithmetic in
  // 32 bits: no division by the row count per thread.)
  const int rows = mblocks * 32;
  const int t = blockIdx.x * (int)blockDim.x + threadIdx.x;
  // The stream-K arrival counters of this call start cleared (the GEMM
  // launch follows in stream order).
  if (blockIdx.y == 0)
    for (int i = t; i < ncounters; i += gridDim.x * blockDim.x) counters[i] = 0;
  if (t >= rows * kWordsPerPlane) return;
  const int w = t % kWordsPerPlane;
  const int row = t / kWordsPerPlane;
  const int chunk = blockIdx.y;
  constexpr int kSteps = Fmt<F>::kSteps;
  uint32_t pw[Q];
  if (row < M && chunk < nchunks) {
    const uint32_t* src = a_packed + plane_words(row, chunk, 0, nchunks, Q) + w;
#pragma unroll
    for (int j = 0; j < Q; ++j) pw[j] = __builtin_nontemporal_load(src + j * kPlaneStride);
  } else {
#pragma unroll
    for (int j = 0; j < Q; ++j) pw[j] = 0u;
  }
  const int mb = row / 32, l = row % 32;
  if (F == 4) {
    // word w -> k-step w / 2, lane half w mod 2; vector 0 holds operand dwords
    // 0..3, vector 1 dwords 4..7
    uint32_t o[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
    if (chunk < nchunks) fp8_word<(Q <= 4 ? Q : 4)>(pw, o);
    v4i* f = out + ((int64_t)mb * nsteps + chunk * kSteps + w / 2) * 2 * kFragVecs;
    f[(w % 2) * 32 + l] = v4i{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
    f[kFragVecs + (w % 2) * 32 + l] = v4i{(int)o[4], (int)o[5], (int)o[6], (int)o[7]};
  } else if (F == 3) {
    // word w -> k-step w / 2, lane half w mod 2; vector 0 holds operand dwords
    // 0..3, vector 1 dwords 4..5
    uint32_t o[6] = {0u, 0u, 0u, 0u, 0u, 0u};
    if (chunk < nchunks) fp6_word<(Q <= 3 ? Q : 3)>(pw, o);
    v4i* f = out + ((int64_t)mb * nsteps + chunk * kSteps + w / 2) * 2 * kFragVecs;
    f[(w % 2) * 32 + l] = v4i{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
    f[kFragVecs + (w % 2) * 32 + l] = v4i{(int)o[4], (int)o[5], 0, 0};
  } else if (F == 2) {
    // word w -> k-step w / 2, vector w mod 2; byte j of lane half h is element
    // 4 (j mod 8) + 2 h + j / 8 of the word
    uint32_t o[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
    if (chunk < nchunks) {
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int e = 4 * (j % 8) + 2 * h + j / 8;
          uint32_t u = 0u;
#pragma unroll
          for (int i = 0; i < Q; ++i) u |= ((pw[i] >> e) & 1u) << i;
          o[4 * h + j / 4] |= e4m3_bipolar<(Q <= 4 ? Q : 4)>(u) << (8 * (j % 4));
        }
    }
    v4i* f = out + (((int64_t)mb * nsteps + chunk * kSteps + w / 2) * 2 + w % 2) * kFragVecs;
    f[l] = v4i{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
    f[l + 32] = v4i{(int)o[4], (int)o[5], (int)o[6], (int)o[7]};
  } else if (F) {
    // word w -> k-step w / 2, lane half w mod 2
    uint32_t o[4] = {0u, 0u, 0u, 0u};
    if (chunk < nchunks) fp4_word<(Q <= 2 ? Q : 2)>(pw, o);
    v4i* f = out + ((int64_t)mb * nsteps + chunk * kSteps + w / 2) * kFragVecs;
    f[(w % 2) * 32 + l] = v4i{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
  } else {
    uint32_t o[8];
    reassemble_word<Q>(pw, o);
    if (chunk >= nchunks)
#pragma unroll
      for (int i = 0; i < 8; ++i) o[i] = 0u;
    v4i* f = out + ((int64_t)mb * nsteps + chunk * kSteps + w) * kFragVecs;
    f[l] = v4i{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
    f[l + 32] = v4i{(int)o[4], (int)o[5], (int)o[6], (int)o[7]};
  }
}

// ---- weight staging -----------------------------------------------------------
// ROWS weight rows of a tile, each split into SPLIT items of 128/SPLIT elements
// (4/SPLIT words per plane).  Consecutive threads take consecutive rows of the
// same part, so a wave's LDS writes hit distinct banks.  Rows past the matrix
// edge are clamped to its last row: their products only reach outputs that are
// never stored, and the code stays branch-free so the scheduler can interleave
// it with the MFMAs.  Chunks past the last one are clamped to it; they meet
// all-zero activation bytes.
template <int B, int ROWS, int SPLIT, int T, int F>
struct Stage {
  static constexpr int kRowBytes = Fmt<F>::kRowBytes;
  static constexpr int kWpi = kWordsPerPlane / SPLIT;
  static constexpr int kItems = ROWS * SPLIT / T;
  static_assert(ROWS * SPLIT % T == 0 && kItems >= 1, "items must divide evenly");
  static constexpr int kWords = kItems * kWpi;  // words reassembled per thread per chunk
  uint32_t raw[kItems][B][kWpi];

  // Byte offset of item `it`'s plane-0 words of chunk 0 in the packed weights.
  static __device__ __forceinline__ uint32_t item_offset(int row0, int rows, int nchunks, int tid,
                                                         int it) {
    const int item = tid + T * it;
    const int r = min(row0 + item % ROWS, rows - 1);
    const int sub = item / ROWS;
    return (uint32_t)(plane_words(r, 0, 0, nchunks, B) + sub * kWpi) * 4u;
  }

  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rsrc, const uint32_t* voff,
                                       int nchunks, int chunk) {
    const uint32_t soff = (uint32_t)min(chunk, nchunks - 1) * (uint32_t)(B * kPlaneStride * 4);
#pragma unroll
    for (int it = 0; it < kItems; ++it) {
#pragma unroll
      for (int i = 0; i < B; ++i) {
        const uint32_t vo = voff[it] + i * kPlaneStride * 4;
        if (kWpi == 4) {
          v4u v = __builtin_amdgcn_raw_buffer_load_b128(rsrc, vo, soff, 0);
          raw[it][i][0] = v.x; raw[it][i][1] = v.y; raw[it][i][2] = v.z; raw[it][i][3] = v.w;
        } else if (kWpi == 2) {
          v2u v = __builtin_amdgcn_raw_buffer_load_b64(rsrc, vo, soff, 0);
          raw[it][i][0] = v.x; raw[it][i][1] = v.y;
        } else {
          raw[it][i][0] = __builtin_amdgcn_raw_buffer_load_b32(rsrc, vo, soff, 0);
        }
      }
    }
  }

  // Half h (0: output dwords 0..3, 1: 4..7) of word u (0 <= u < kWords) of
  // this thread's items, reassembled and written to LDS.  The low half
  // leaves the tree's middle level in mid[] for the high half.  FP4: the
  // whole word's 16 nibble bytes in half 0, nothing in half 1.
  __device__ __forceinline__ void store_half(uint8_t* lds_tile, int tid, int u, int h,
                                             uint32_t mid[8]) const {
    const int it = u / kWpi, w = u % kWpi;
    const int item = tid + T * it;
    const int r = item % ROWS;
    const int sub = item / ROWS;
    uint32_t o[4];
    if (F == 4) {
      if (h != 0) return;
      uint32_t pw[B], o8[8];
#pragma unroll
      for (int i = 0; i < B; ++i) pw[i] = raw[it][i][w];
      fp8_word<(B <= 4 ? B : 4)>(pw, o8);
      const int wc = sub * kWpi + w;  // word of the chunk -> k-step wc / 2, lane half wc mod 2
      uint8_t* d = lds_tile + r * kRowBytes + (wc / 2) * Fmt<F>::kStepRowBytes + (wc % 2) * Fmt<F>::kHalfBytes;
      *reinterpret_cast<uint4*>(d) = make_uint4(o8[0], o8[1], o8[2], o8[3]);
      *reinterpret_cast<uint4*>(d + 16) = make_uint4(o8[4], o8[5], o8[6], o8[7]);
      return;
    }
    if (F == 3) {
      if (h != 0) return;
      uint32_t pw[B], o6[6];
#pragma unroll
      for (int i = 0; i < B; ++i) pw[i] = raw[it][i][w];
      fp6_word<(B <= 3 ? B : 3)>(pw, o6);
      const int wc = sub * kWpi + w;  // word of the chunk -> k-step wc / 2, lane half wc mod 2
      uint8_t* d = lds_tile + r * kRowBytes + (wc / 2) * Fmt<F>::kStepRowBytes + (wc % 2) * Fmt<F>::kHalfBytes;
      *reinterpret_cast<uint4*>(d) = make_uint4(o6[0], o6[1], o6[2], o6[3]);
      *reinterpret_cast<uint2*>(d + 16) = make_uint2(o6[4], o6[5]);
      return;
    }
    if (F) {
      if (h != 0) return;
      uint32_t pw[B];
#pragma unroll
      for (int i = 0; i < B; ++i) pw[i] = raw[it][i][w];
      fp4_word<(B <= 2 ? B : 2)>(pw, o);
      const int wc = sub * kWpi + w;  // word of the chunk -> k-step wc / 2, lane half wc mod 2
      *reinterpret_cast<uint4*>(lds_tile + r * kRowBytes + (wc / 2) * kStepBytes + (wc % 2) * 16) =
          make_uint4(o[0], o[1], o[2], o[3]);
      return;
    }
    if (h == 0) {
      uint32_t pw[B];
#pragma unroll
      for (int i = 0; i < B; ++i) pw[i] = raw[it][i][w];
      reassemble_lo<B>(pw, mid, o);
    } else {
      reassemble_hi<B>(mid, o);
    }
    uint4* d4 = reinterpret_cast<uint4*>(lds_tile + r * kRowBytes + (sub * kWpi + w) * kStepBytes);
    d4[h] = make_uint4(o[0], o[1], o[2], o[3]);
  }

  __device__ __forceinline__ void store(uint8_t* lds_tile, int tid) const {
    uint32_t mid[8];
#pragma unroll
    for (int u = 0; u < kWords; ++u) {
      store_half(lds_tile, tid, u, 0, mid);
      store_half(lds_tile, tid, u, 1, mid);
    }
  }
};

__host__ __device__ constexpr int offset_of(int b) { return b == 8 ? 1 : 1 - (1 << b); }
__host__ __device__ constexpr int pad_of(int b) { return b == 8 ? -128 : 0; }

// ---- main kernel --------------------------------------------------------------
// Work decomposition.  The output is cut into T tiles of BM x BN (row-major
// tile order) and each tile's K into NCE/2 pairs of chunks.  A launch of G
// persistent workgroups gives workgroup w the whole tiles w, w + G, ...,
// (dp_tiles - 1) G + w, and splits the chunk pairs of the remaining
// T - dp_tiles G tiles evenly among the first G' <= G workgroups: workgroup
// w < G' takes pairs [w S / G', (w+1) S / G') of them (S = sk_pairs), i.e. the
// end of one tile, possibly whole tiles, and the start of another
// (stream-K).  The host keeps G' at most twice the stream-K tile count, so a
// tile has about two parts (every further part costs a partial tile written
// and read back), or G' equal to it, so that each leftover tile is one
// workgroup's whole part (see sk_parts).  A workgroup walks its stream-K pairs
// first and its whole tiles after, as one continuous chunk stream: the
// software pipeline runs across tile boundaries, and at the end of each part
// of a tile the accumulators are flushed:
//   whole tile        epilogue;
//   producer part     (starts after the tile's first pair) int32 partial to
//                     the workspace, then an arrival on the tile's counter;
//   owner part        (starts at the first pair, ends early) usually finds
//                     every producer arrived, adds their partials and runs
//                     the epilogue; otherwise it publishes its own partial
//                     and arrives as well.
// Whoever arrives last finishes the tile, so no workgroup ever waits for
// another.  Partials and counters use device-coherent (sc1) accesses, so the
// hand-off needs no cache flush: the workgroups of one tile sit on different
// XCDs, behind different L2s.

// Position in a workgroup's chunk-pair stream.  Every field is uniform.
struct Cursor {
  int tile;      // tile index (>= T past the end of the stream)
  int m0, n0;    // tile origin (a valid tile's past the end)
  int pair;      // pair within the tile
  int pend;      // end of this part (exclusive pair)
  int pbeg;      // first pair of this part
  int sk_left;   // stream-K pairs after this part
  int dp_next;   // next whole-tile round
};

// Walks the stream; tile origins are updated incrementally (no division in
// the loop): the next stream-K tile is the next tile in row-major order, the
// next whole tile is G tiles further.
struct Stream {
  int G, w, pairs, dp_tiles, sk_base, sk_lo, sk_hi, sk_g, tiles;
  int n_begin, n_end;    // output columns of the tile grid: [n_begin, n_begin + tiles_n BN)
  int bm, bn;
  int g_m, g_n;           // G tiles as (rows, columns) of the tile grid: G = g_m tiles_n + g_n
  int dp_m0, dp_n0;       // origin of tile w

  __device__ __forceinline__ void step_origin(Cursor& c, int dm, int dn) const {
    c.n0 += dn * bn;
    c.m0 += dm * bm;
    if (c.n0 >= n_end) {
      c.n0 -= n_end - n_begin;
      c.m0 += bm;
    }
  }
  __device__ __forceinline__ void begin_dp(Cursor& c, int round) const {
    if (round == 0) {
      c.m0 = dp_m0;
      c.n0 = dp_n0;
    } else if (round < dp_tiles) {
      step_origin(c, g_m, g_n);
    }
    c.tile = round < dp_tiles ? round * G + w : 0x7fffffff;  // past the end
    c.pair = c.pbeg = 0;
    c.pend = pairs;
    c.dp_next = round + 1;
    c.sk_left = 0;
  }
  __device__ __forceinline__ Cursor first(int tiles_n) const {
    // (tile origins are absolute output coordinates)
    Cursor c;
    if (sk_hi > sk_lo) {
      c.tile = sk_base + sk_lo / pairs;
      c.m0 = c.tile / tiles_n * bm;
      c.n0 = n_begin + c.tile % tiles_n * bn;
      c.pair = c.pbeg = sk_lo % pairs;
      c.pend = min(pairs, c.pair + (sk_hi - sk_lo));
      c.sk_left = (sk_hi - sk_lo) - (c.pend - c.pair);
      c.dp_next = 0;
    } else {
      begin_dp(c, 0);
    }
    return c;
  }
  __device__ __forceinline__ void advance(Cursor& c) const {
    if (++c.pair < c.pend) return;
    if (c.sk_left > 0) {
      ++c.tile;
      step_origin(c, 0, 1);
      c.pair = c.pbeg = 0;
      c.pend = min(pairs, c.sk_left);
      c.sk_left -= c.pend;
    } else {
      begin_dp(c, c.dp_next);
    }
  }
  // Workgroup whose stream-K range holds stream-K pair u of S (G' = sk_g).
  __device__ __forceinline__ int range_of(int u, int S) const {
    return (int)((((int64_t)u + 1) * sk_g - 1) / S);
  }
};

// The MFMA takes the weight fragment as its first operand, so the accumulator
// of lane l holds D[n][m] for m = l mod 32 and four consecutive n: each lane
// stores 16 contiguous output bytes.
// The whole work of workgroup w of G for one tile shape (the kernels below
// call it; `lds` is the dynamic LDS of the launch).
template <int P, int F, int BM, int BN, int WM, int WN, int SPLIT>
__device__ __forceinline__ void gemm_int8_body(const Int8Params& prm, uint8_t* lds, int w, int G) {
  static_assert(F == 0 || P <= (F == 4 ? 4 : F == 3 ? 3 : 2),
                "FP4 operands hold weights of at most 2 bits, FP6 at most 3, FP8 at most 4");
  constexpr int kSteps = Fmt<F>::kSteps;
  constexpr int kAVecs = Fmt<F>::kAVecs;
  constexpr int kRowBytes = Fmt<F>::kRowBytes;
  constexpr int T = WM * WN * kWave;
  constexpr int WTM = BM / WM, WTN = BN / WN;  // wave tile
  constexpr int FM = WTM / 32, FN = WTN / 32;  // 32x32 fragments per wave
  constexpr int kStageBytes = BN * kRowBytes;
  static_assert(FM >= 1 && FN >= 1, "wave tile too small");
  __shared__ int s_bcast;

  const GemmArgs& g = prm.g;
  const int NC = prm.nchunks;
  const int NCE = (NC + 1) & ~1;  // even chunk count; a last odd chunk is all padding
  const int tid = threadIdx.x;
  const int lane = tid % kWave;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);  // uniform in the wave
  const int wm = wave / WN, wn = wave % WN;
  // Epilogue terms of the tile being finished, staged in LDS after the ring:
  // c_a R_w[n] and the scale s_w[n] per column, c_w R_a[m] - const and s_a[m]
  // per row; with zero-points also z_w[n] and s_w R_w[n] + K z_w[n] per
  // column, float(R_a[m]) and z_a[m] per row.
  uint32_t* const lds_wt = reinterpret_cast<uint32_t*>(lds + kStages * kStageBytes);
  uint32_t* const lds_at = lds_wt + BN;
  float* const lds_ws = reinterpret_cast<float*>(lds_at + BM);
  float* const lds_as = lds_ws + BN;
  float* const lds_zt = lds_as + BM;   // z_w[n] | float(R_a[m])
  float* const lds_zc = lds_zt + BN + BM;  // s_w R_w[n] + K z_w[n] | z_a[m]
  constexpr int kEpiStride = 32 * 4 + 16;  // bytes per row of a 32x32 int32 block in LDS
  uint8_t* const epi_slot = lds + kStages * kStageBytes + (BN + BM) * 16 + wave * 32 * kEpiStride;

  Stream st;
  st.G = G;
  st.w = w;
  st.pairs = NCE / 2;
  st.dp_tiles = prm.dp_tiles;
  st.sk_base = prm.dp_tiles * st.G;
  st.sk_g = prm.sk_grid;
  st.sk_lo = st.w < st.sk_g ? (int)((int64_t)st.w * prm.sk_pairs / st.sk_g) : 0;
  st.sk_hi = st.w < st.sk_g ? (int)((int64_t)(st.w + 1) * prm.sk_pairs / st.sk_g) : 0;
  st.tiles = prm.tiles;
  st.n_begin = prm.n_begin;
  st.n_end = prm.n_begin + prm.tiles_n * BN;
  st.bm = BM;
  st.bn = BN;
  st.g_m = st.G / prm.tiles_n;
  st.g_n = st.G % prm.tiles_n;
  st.dp_m0 = st.w / prm.tiles_n * BM;
  st.dp_n0 = prm.n_begin + st.w % prm.tiles_n * BN;
  if (prm.dp_tiles == 1 && prm.sk_pairs == 0 && prm.tiles % 8 == 0 && G == prm.tiles) {
    // One round of whole tiles: workgroups are dealt round-robin to the 8
    // XCDs (w mod 8), so give each XCD a contiguous run of row-major tiles;
    // its L2 then holds fewer activation bands.
    const int t = (w % 8) * (prm.tiles / 8) + w / 8;
    st.dp_m0 = t / prm.tiles_n * BM;
    st.dp_n0 = prm.n_begin + t % prm.tiles_n * BN;
  }

  // ---- operand sources
  using SW = Stage<P, BN, SPLIT, T, F>;
  SW rw0, rw1;
  const __amdgpu_buffer_rsrc_t w_rsrc = make_rsrc(g.w_packed, prm.w_bytes);
  const __amdgpu_buffer_rsrc_t a_rsrc = make_rsrc(prm.a_frag, prm.a_bytes);
  // Uniform byte offset of this wave's 32-row fragment block a of a tile.
  // Offsets are unsigned 32-bit: the host admits fragment buffers below 4 GiB.
  auto a_block = [&](int m0, int a) __attribute__((always_inline)) -> uint32_t {
    const int mb = min((m0 + wm * WTM) / 32 + a, prm.mblocks - 1);
    return (uint32_t)mb * (uint32_t)prm.nsteps * (uint32_t)(kAVecs * kFragVecs * 16);
  };
  const uint32_t a_lane = lane * 16;
  // vector x (F = 2: 0 or 1) of k-step ks of the fragment block
  auto load_a = [&](int m0, int chunk, int ks, int a, int x = 0) __attribute__((always_inline)) -> v4i {
    const uint32_t soff =
        a_block(m0, a) +
        ((uint32_t)(min(chunk, NCE - 1) * kSteps + ks) * kAVecs + x) * (uint32_t)(kFragVecs * 16);
    return __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(a_rsrc, a_lane, soff, 0));
  };
  auto w_offsets = [&](int n0, uint32_t* voff) __attribute__((always_inline)) {
#pragma unroll
    for (int it = 0; it < SW::kItems; ++it) voff[it] = SW::item_offset(n0, g.N, NC, tid, it);
  };

  v16i acc[FN][FM];
  auto zero_acc = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int b = 0; b < FN; ++b)
#pragma unroll
      for (int a = 0; a < FM; ++a)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[b][a][v] = 0;
  };
  zero_acc();
  v4i afr[kSteps * kAVecs][FM];  // vector x of k-step ks at ks * kAVecs + x

  const int lrow = lane % 32;
  const int lk = (lane / 32) * Fmt<F>::kHalfBytes;
  const int w_lane = (wn * WTN + lrow) * kRowBytes + lk;
  v4i wf[2][FN];
  v2i wf6[2][F == 3 ? FN : 1];  // FP6: operand dwords 4..5
  v4i wf8[2][F == 4 ? FN : 1];  // FP8: operand dwords 4..7
  auto read_wf = [&](const uint8_t* stage, int ks, int sl) __attribute__((always_inline)) {
#pragma unroll
    for (int b = 0; b < FN; ++b) {
      const uint8_t* src = stage + w_lane + b * 32 * kRowBytes + ks * Fmt<F>::kStepRowBytes;
      wf[sl][b] = *reinterpret_cast<const v4i*>(src);
      if constexpr (F == 3) wf6[sl][b] = *reinterpret_cast<const v2i*>(src + 16);
      if constexpr (F == 4) wf8[sl][b] = *reinterpret_cast<const v4i*>(src + 16);
    }
  };

  // One pipeline step: the MFMAs of one chunk from stage `cst`.  During
  // k-step ks the weight fragments of ks+1 are read (for the last k-step:
  // those of the next chunk's first k-step from `nst`, complete since the
  // previous barrier), a slice of the reassembly of the chunk after next
  // from `rw` goes to stage `sst`, and the activation registers of ks are
  // refilled with the next chunk (tile origin a_m0, chunk a_chunk).  A
  // scheduling fence closes every k-step.
  constexpr int kHalves = 2 * SW::kWords;
  auto step = [&](const uint8_t* cst, uint8_t* sst, const uint8_t* nst, const SW& rw, int a_m0,
                  int a_chunk) __attribute__((always_inline)) {
    uint32_t mid[8];
#pragma unroll
    for (int ks = 0; ks < kSteps; ++ks) {
      const int cur = ks & 1, nxt = cur ^ 1;
      if (ks + 1 < kSteps)
        read_wf(cst, ks + 1, nxt);
      else
        read_wf(nst, 0, nxt);
#pragma unroll
      for (int hu = 0; hu < kHalves; ++hu)
        if (hu * kSteps / kHalves == ks) rw.store_half(sst, tid, hu / 2, hu % 2, mid);
#pragma unroll
      for (int b = 0; b < FN; ++b)
#pragma unroll
        for (int a = 0; a < FM; ++a)
          if constexpr (F == 4) {
            // E4M3 weights and activations (format code 0), unit E8M0 scales (127)
            const v8i wa = {wf[cur][b][0], wf[cur][b][1], wf[cur][b][2], wf[cur][b][3],
                            wf8[cur][b][0], wf8[cur][b][1], wf8[cur][b][2], wf8[cur][b][3]};
            const v4i a0 = afr[2 * ks][a], a1 = afr[2 * ks + 1][a];
            const v8i ab = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
            acc[b][a] = __builtin_bit_cast(
                v16i, __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                          wa, ab, __builtin_bit_cast(v16f, acc[b][a]), 0, 0, 0, 127, 0, 127));
          } else if constexpr (F == 3) {
            // E2M3 weights and activations (format code 2), unit E8M0 scales (127)
            const v8i wa = {wf[cur][b][0], wf[cur][b][1], wf[cur][b][2], wf[cur][b][3],
                            wf6[cur][b][0], wf6[cur][b][1], 0, 0};
            const v4i a0 = afr[2 * ks][a], a1 = afr[2 * ks + 1][a];
            const v8i ab = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], 0, 0};
            acc[b][a] = __builtin_bit_cast(
                v16i, __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                          wa, ab, __builtin_bit_cast(v16f, acc[b][a]), 2, 2, 0, 127, 0, 127));
          } else if constexpr (F == 2) {
            // E2M1 weights (format code 4) x E4M3 activations (code 0), unit E8M0 scales (127)
            const v8i wa = {wf[cur][b][0], wf[cur][b][1], wf[cur][b][2], wf[cur][b][3], 0, 0, 0, 0};
            const v4i a0 = afr[2 * ks][a], a1 = afr[2 * ks + 1][a];
            const v8i ab = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
            acc[b][a] = __builtin_bit_cast(
                v16i, __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                          wa, ab, __builtin_bit_cast(v16f, acc[b][a]), 4, 0, 0, 127, 0, 127));
          } else if constexpr (F == 1) {
            // E2M1 x E2M1 (format code 4 for both), unit E8M0 scales (127)
            const v8i wa = {wf[cur][b][0], wf[cur][b][1], wf[cur][b][2], wf[cur][b][3], 0, 0, 0, 0};
            const v8i ab = {afr[ks][a][0], afr[ks][a][1], afr[ks][a][2], afr[ks][a][3], 0, 0, 0, 0};
            acc[b][a] = __builtin_bit_cast(
                v16i, __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                          wa, ab, __builtin_bit_cast(v16f, acc[b][a]), 4, 4, 0, 127, 0, 127));
          } else {
            acc[b][a] = __builtin_amdgcn_mfma_i32_32x32x32_i8(wf[cur][b], afr[ks][a], acc[b][a], 0, 0, 0);
          }
#pragma unroll
      for (int a = 0; a < FM; ++a)
#pragma unroll
        for (int x = 0; x < kAVecs; ++x) afr[ks * kAVecs + x][a] = load_a(a_m0, a_chunk, ks, a, x);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // ---- epilogue constants
  // F = 0: C = 4 D + c_w R_a + c_a R_w - c_a c_w K - pad_term (kernel header).
  // F > 0: the operands are the bipolar values themselves, so C = D less the
  // padding elements inside the last real chunk: their all-zero planes stand
  // for -(2^p - 1) and -(2^q - 1), whose products add (K_pad - K)(2^p-1)(2^q-1).
  const int q = g.q;
  constexpr uint32_t kMul = F ? 1u : 4u;
  const uint32_t ca = F ? 0u : (uint32_t)(q == 8 ? 1 : 1 - (1 << q));
  const uint32_t cw = F ? 0u : (uint32_t)offset_of(P);
  const uint32_t pad_term =
      F ? (uint32_t)(NC * kChunk - g.K) * ((1u << P) - 1u) * ((1u << q) - 1u)
        : 4u * (uint32_t)(NC * kChunk - g.K) * (uint32_t)((q == 8 ? -128 : 0) * pad_of(P));
  const uint32_t const_term = ca * cw * (uint32_t)g.K + pad_term;
  const bool fp16 = g.c_fp16 != nullptr;
  const bool vec_ok = prm.vec_out != 0;

  // Epilogue terms of tile (m0, n0): one value per thread, fetched a pair of
  // chunks before the tile's flush and written to LDS before that pair's
  // last barrier (the loads are issued before any output store, so waiting
  // for them never waits for stores).
  // The loaded words are kept as they arrive and combined only when they are
  // staged, a chunk later: arithmetic right after the loads would make the
  // wave wait for every load in flight (the loads complete in order).
  constexpr int kTermsPerThread = (BN + BM + T - 1) / T;
  uint32_t rowsum[kTermsPerThread];
  uint16_t scale_bits[kTermsPerThread];
  auto fetch_terms = [&](int m0, int n0) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < kTermsPerThread; ++k) {
      const int i = tid + k * T;
      rowsum[k] = 0;
      scale_bits[k] = 0;
      if (i < BN) {
        const int n = min(n0 + i, g.N - 1);
        rowsum[k] = (uint32_t)g.w_rowsum[n];
        if (fp16) scale_bits[k] = __half_as_ushort(g.w_scale[n]);
      } else if (i < BN + BM) {
        const int m = min(m0 + i - BN, g.M - 1);
        rowsum[k] = (uint32_t)g.a_rowsum[m];
        if (fp16) scale_bits[k] = __half_as_ushort(g.a_scale[m]);
      }
    }
  };
  // With zero-points the extra terms are read here, just before they are
  // staged: once per tile, off the main loop's register budget.
  const bool affine = g.a_zero != nullptr;
  auto stage_terms = [&](int m0, int n0) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < kTermsPerThread; ++k) {
      const int i = tid + k * T;
      if (i < BN + BM) {
        // c_a R_w[n] per column, c_w R_a[m] - const per row; lds_at follows lds_wt
        lds_wt[i] = i < BN ? ca * rowsum[k] : cw * rowsum[k] - const_term;
        lds_ws[i] = __half2float(__ushort_as_half(scale_bits[k]));
      }
    }
    if (affine) {
#pragma unroll
      for (int k = 0; k < kTermsPerThread; ++k) {
        const int i = tid + k * T;
        if (i < BN) {
          const int n = min(n0 + i, g.N - 1);
          const float zw = __half2float(g.w_zero[n]);
          lds_zt[i] = zw;
          lds_zc[i] = __half2float(g.w_scale[n]) * (float)g.w_rowsum[n] + (float)g.K * zw;
        } else if (i < BN + BM) {
          const int m = min(m0 + i - BN, g.M - 1);
          lds_zt[i] = (float)g.a_rowsum[m];
          lds_zc[i] = __half2float(g.a_zero[m]);
        }
      }
    }
  };

  // Stream-K partial tiles: two slots per workgroup, each in accumulator
  // order (lane-contiguous 16-byte vectors), with device-coherent (sc1)
  // accesses.
  constexpr int kAccVecs = FN * FM * 4;  // v4i per lane
  constexpr uint32_t kSlotBytes = (uint32_t)BM * BN * 4;
  const __amdgpu_buffer_rsrc_t p_rsrc = make_rsrc(prm.partial, prm.partial_bytes);
  const uint32_t p_lane = (uint32_t)((wave * kAccVecs * kWave + lane) * 16);
  auto partial_off = [&](int b, int a, int j) __attribute__((always_inline)) -> uint32_t {
    return p_lane + (uint32_t)(((b * FM + a) * 4 + j) * kWave * 16);
  };

  // Final values of tile (m0, n0): each 32x32 accumulator block goes through
  // the wave's LDS slot and comes back row by row, so that every store
  // instruction writes 8 whole 128-byte output rows; the affine correction
  // and the optional fp16 scaling are applied on the way out.  A tile shared
  // by workgroups [pv_first, pv_last] first adds, block by block, the
  // partials of every sharing workgroup except this one (the first one's
  // in its second slot, the others' in their first): the four loads of a
  // block leave together, where one load per round trip is all the
  // registers of the main loop leave room for over a whole tile.
  auto epilogue = [&](int m0, int n0, int pv_first, int pv_last) __attribute__((always_inline)) {
    const int er = lane / 8, ec = (lane % 8) * 4;  // read-back row (+8 i) and first column
#pragma unroll
    for (int a = 0; a < FM; ++a) {
#pragma unroll
      for (int b = 0; b < FN; ++b) {
        for (int v = pv_first; v <= pv_last; ++v) {
          if (v == st.w) continue;
          const uint32_t so = (uint32_t)(v == pv_first ? 2 * v + 1 : 2 * v) * kSlotBytes;
          v4i pv[4];
#pragma unroll
          for (int j = 0; j < 4; ++j)
            pv[j] = __builtin_bit_cast(
                v4i, __builtin_amdgcn_raw_buffer_load_b128(p_rsrc, partial_off(b, a, j), so, 16 /* sc1 */));
          __builtin_amdgcn_sched_barrier(0);  // all four loads leave before the first add waits
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[b][a][4 * j + i] += pv[j][i];
        }
        // acc[b][a][4 gi + j] = D[n = 8 gi + 4 (lane / 32) + j][m = lane mod 32]
#pragma unroll
        for (int gi = 0; gi < 4; ++gi) {
          v4i v = {acc[b][a][gi * 4 + 0], acc[b][a][gi * 4 + 1], acc[b][a][gi * 4 + 2],
                   acc[b][a][gi * 4 + 3]};
          *reinterpret_cast<v4i*>(epi_slot + lrow * kEpiStride + (gi * 8 + (lane / 32) * 4) * 4) = v;
        }
        __builtin_amdgcn_s_waitcnt(0xc07f);  // LDS writes of this wave done (lgkmcnt 0)
        __builtin_amdgcn_wave_barrier();
        const int nl = wn * WTN + b * 32 + ec;  // column in the tile
        const int ncol = n0 + nl;
        const bool full = vec_ok && ncol + 3 < g.N;
        const v4u wt = *reinterpret_cast<const v4u*>(lds_wt + nl);
        const v4f ws = *reinterpret_cast<const v4f*>(lds_ws + nl);
        // the block's four rows and their row terms are read together, before
        // any of the (uniform) edge and format branches below, which would
        // otherwise take one LDS round trip each
        v4i dv[4];
        uint32_t atv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          dv[i] = *reinterpret_cast<const v4i*>(epi_slot + (er + 8 * i) * kEpiStride + ec * 4);
          atv[i] = lds_at[wm * WTM + a * 32 + er + 8 * i];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) keep_here(dv[i], atv[i]);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int ml = wm * WTM + a * 32 + er + 8 * i;  // row in the tile
          const int m = m0 + ml;
          const v4i d = dv[i];
          const uint32_t at = atv[i];
          int32_t cv[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) cv[j] = (int32_t)(kMul * (uint32_t)d[j] + at + wt[j]);
          if (m < g.M && ncol < g.N) {
            const int64_t o = (int64_t)m * g.N + ncol;
            if (g.c_int32) {
              if (full)
                store16(g.c_int32 + o, v4i{cv[0], cv[1], cv[2], cv[3]});
              else
                for (int j = 0; j < 4 && ncol + j < g.N; ++j) g.c_int32[o + j] = cv[j];
            }
            if (fp16) {
              const float sa = lds_as[ml];
              float f[4];
              if (affine) {
                const v4f zw = *reinterpret_cast<const v4f*>(lds_zt + nl);
                const v4f col = *reinterpret_cast<const v4f*>(lds_zc + nl);
                const float ra = lds_zt[BN + ml], za = lds_zc[BN + ml];
#pragma unroll
                for (int j = 0; j < 4; ++j) f[j] = affine_value(cv[j], sa, ws[j], zw[j], ra, za, col[j]);
              } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) f[j] = (float)cv[j] * sa * ws[j];
              }
              uint32_t hb[2];
#pragma unroll
              for (int j = 0; j < 4; j += 2) {
                const uint32_t h0 = __half_as_ushort(__float2half_rn(f[j]));
                const uint32_t h1 = __half_as_ushort(__float2half_rn(f[j + 1]));
                hb[j / 2] = h0 | (h1 << 16);
              }
              if (full)
                *reinterpret_cast<uint2*>(g.c_fp16 + o) = make_uint2(hb[0], hb[1]);
              else
                for (int j = 0; j < 4 && ncol + j < g.N; ++j)
                  g.c_fp16[o + j] = __ushort_as_half((unsigned short)(hb[j / 2] >> (16 * (j % 2))));
            }
          }
        }
        __builtin_amdgcn_s_waitcnt(0xc07f);  // reads done before the slot is rewritten
        __builtin_amdgcn_wave_barrier();
      }
    }
  };

  // ---- stream-K partial tiles
  auto store_partial = [&](int slot) __attribute__((always_inline)) {
#pragma unroll
    for (int b = 0; b < FN; ++b)
#pragma unroll
      for (int a = 0; a < FM; ++a)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const v4i v = {acc[b][a][4 * j], acc[b][a][4 * j + 1], acc[b][a][4 * j + 2],
                         acc[b][a][4 * j + 3]};
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u, v), p_rsrc, partial_off(b, a, j),
                                                 slot * kSlotBytes, 16 /* sc1 */);
        }
  };
  // Publishes this workgroup's partial of stream-K tile u in `slot` and
  // counts its arrival; true when it is the last of the tile's parts.
  auto arrive = [&](int slot, int* counter, int parts) __attribute__((always_inline)) {
    store_partial(slot);
    __builtin_amdgcn_s_waitcnt(0);  // the partial is at device scope before the arrival
    __syncthreads();
    if (tid == 0)
      s_bcast = __hip_atomic_fetch_add(counter, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1;
    __syncthreads();
    return s_bcast == parts;
  };

  // End of a part of tile c.tile: epilogue, or the stream-K hand-off.
  // The workgroups sharing this workgroup's first and last stream-K tiles
  // (the only ones it can share): [first, last] workgroup of each.
  int sh_tile[2] = {-1, -1}, sh_first[2] = {0, 0}, sh_last[2] = {0, 0};
  if (st.sk_hi > st.sk_lo) {
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int u = (e == 0 ? st.sk_lo : st.sk_hi - 1) / st.pairs;
      sh_tile[e] = st.sk_base + u;
      sh_first[e] = st.range_of(u * st.pairs, prm.sk_pairs);
      sh_last[e] = st.range_of(u * st.pairs + st.pairs - 1, prm.sk_pairs);
    }
  }

  auto flush = [&](const Cursor& c) __attribute__((always_inline)) {
    if (F) {
      // FP4: the fp32 sums are exact integers; partials and the epilogue
      // work on their int32 values.  Converted as whole vectors: a bit cast
      // of one vector element is taken from element 0 by this compiler.
#pragma unroll
      for (int b = 0; b < FN; ++b)
#pragma unroll
        for (int a = 0; a < FM; ++a)
          acc[b][a] = __builtin_convertvector(__builtin_bit_cast(v16f, acc[b][a]), v16i);
    }
    bool finish = true;
    int w_first = 0, w_last = -1;  // the workgroups sharing the tile (none: whole)
    if (__builtin_expect(c.pbeg != 0 || c.pend != st.pairs, 0)) {
      const int e = c.tile == sh_tile[0] ? 0 : 1;
      w_first = sh_first[e];
      w_last = sh_last[e];
      const int parts = w_last - w_first + 1;
      int* counter = prm.counters + (c.tile - st.sk_base);
      if (c.pbeg == 0) {  // owner: the first pairs of the tile, at the end of its range
        if (tid == 0)
          s_bcast = __hip_atomic_load(counter, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __syncthreads();
        finish = s_bcast == parts - 1;
        __syncthreads();
        if (!finish) finish = arrive(2 * st.w + 1, counter, parts);
      } else {            // producer: later pairs, at the start of its range
        finish = arrive(2 * st.w, counter, parts);
      }
    }
    if (finish) epilogue(c.m0, c.n0, w_first, w_last);
  };

  // ---- pipeline over the chunk stream.  Chunk 2p+e of the stream is chunk
  // 2 cur.pair + e of tile cur.tile, for the cursor of pair p.
  Cursor cp = st.first(prm.tiles_n);
  Cursor c1 = cp;
  st.advance(c1);
  Cursor c2 = c1;
  st.advance(c2);
  uint32_t wv0[SW::kItems], wv1[SW::kItems], wv2[SW::kItems];  // weight offsets of cp, c1, c2
  w_offsets(cp.n0, wv0);
  w_offsets(c1.n0, wv1);
  w_offsets(c2.n0, wv2);

  // Prologue: pair cp into stages 0 and 1, the first chunk of c1 in
  // registers, activation fragments and the first weight fragments of the
  // first chunk.  The loads leave in the loop's own order (weight words of
  // the next chunk, then activation fragments), so that the wait counts the
  // compiler derives at the loop head, which cover both ways in, only wait
  // for the loads each k-step needs.
  rw0.load(w_rsrc, wv0, NC, 2 * cp.pair);
  rw1.load(w_rsrc, wv0, NC, 2 * cp.pair + 1);
  rw0.store(lds, tid);
  rw1.store(lds + kStageBytes, tid);
  rw0.load(w_rsrc, wv1, NC, 2 * c1.pair);
#pragma unroll
  for (int ks = 0; ks < kSteps; ++ks)
#pragma unroll
    for (int a = 0; a < FM; ++a)
#pragma unroll
      for (int x = 0; x < kAVecs; ++x) afr[ks * kAVecs + x][a] = load_a(cp.m0, 2 * cp.pair, ks, a, x);
  __syncthreads();
  read_wf(lds, 0, 0);

  int s0 = 0;  // stage of the current pair's first chunk
  while (cp.tile < prm.tiles) {
    const int s1 = s0 == 2 ? 0 : s0 + 1, s2 = s1 == 2 ? 0 : s1 + 1;
    const bool part_end = cp.pair + 1 == cp.pend;
    if (part_end) fetch_terms(cp.m0, cp.n0);
    rw1.load(w_rsrc, wv1, NC, 2 * c1.pair + 1);
    step(lds + s0 * kStageBytes, lds + s2 * kStageBytes, lds + s1 * kStageBytes, rw0,
         cp.m0, 2 * cp.pair + 1);
    __syncthreads();
    rw0.load(w_rsrc, wv2, NC, 2 * c2.pair);
    step(lds + s1 * kStageBytes, lds + s0 * kStageBytes, lds + s2 * kStageBytes, rw1,
         c1.m0, 2 * c1.pair);
    if (F) {
      // An empty use of every accumulator here keeps the scaled MFMAs in
      // their k-steps: without one, the machine code sinker moves all of the
      // pair's MFMAs past the conditional blocks below, and the next
      // chunk's activation registers then spill.  (No instruction is emitted.)
#pragma unroll
      for (int b = 0; b < FN; ++b)
#pragma unroll
        for (int a = 0; a < FM; ++a) keep_here(acc[b][a]);
    }
    if (part_end) stage_terms(cp.m0, cp.n0);
    __syncthreads();
    if (__builtin_expect(part_end, 0)) {
      flush(cp);
      zero_acc();
    }
    s0 = s2;
    cp = c1;
    c1 = c2;
#pragma unroll
    for (int it = 0; it < SW::kItems; ++it) { wv0[it] = wv1[it]; wv1[it] = wv2[it]; }
    const int old_tile = c2.tile;
    st.advance(c2);
    if (c2.tile != old_tile) w_offsets(c2.n0, wv2);
  }
}

template <int P, int F, int BM, int BN, int WM, int WN, int SPLIT>
__global__ __launch_bounds__(WM* WN* kWave, (WM * WN == 4) ? 2 : 1) void gemm_int8_kernel(Int8Params prm) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  gemm_int8_body<P, F, BM, BN, WM, WN, SPLIT>(prm, lds, blockIdx.x, gridDim.x);
}

// Two launches' work in one grid: workgroups [0, g0) do shape A over prm_a,
// the rest shape B over prm_b (same wave count).  Workgroups are dispatched
// in index order, so B's start on the compute units that A's release, while
// A's last tiles and output stores are still in flight.
template <int P, int F, int BMA, int BNA, int WMA, int WNA, int SA, int BMB, int BNB, int WMB,
          int WNB, int SB>
__global__ __launch_bounds__(WMA* WNA* kWave, (WMA * WNA == 4) ? 2 : 1) void gemm_int8_pair_kernel(Int8Params prm_a,
                                                                         Int8Params prm_b, int g0) {
  static_assert(WMA * WNA == WMB * WNB, "both shapes need the same workgroup size");
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  if ((int)blockIdx.x < g0)
    gemm_int8_body<P, F, BMA, BNA, WMA, WNA, SA>(prm_a, lds, blockIdx.x, g0);
  else
    gemm_int8_body<P, F, BMB, BNB, WMB, WNB, SB>(prm_b, lds, blockIdx.x - g0, gridDim.x - g0);
}

struct TileShape {
  int bm, bn, wm, wn, split;
};
constexpr TileShape kShapes[] = {
    {256, 256, 4, 2, 2},
    {256, 256, 2, 4, 2},
    {256, 128, 4, 2, 4},
    {128, 128, 2, 2, 2},
    {512, 128, 8, 1, 4},
    {256, 128, 4, 1, 2},
};
constexpr int kNumShapes = sizeof(kShapes) / sizeof(kShapes[0]);

// LDS of shape S: the weight ring, the epilogue terms and one 32x32 int32
// epilogue slot per wave.
template <int F>
constexpr size_t lds_bytes(const TileShape& sh) {
  return kStages * (size_t)sh.bn * Fmt<F>::kRowBytes + (size_t)(sh.bn + sh.bm) * 16 +
         (size_t)sh.wm * sh.wn * 32 * (32 * 4 + 16);
}

// Launches shape S with `grid` persistent workgroups (prm holds the
// decomposition).
template <int P, int F, int S>
hipError_t launch_shape(const Int8Params& prm, int grid, hipStream_t stream) {
  constexpr TileShape sh = kShapes[S];
  const size_t lds = lds_bytes<F>(sh);
  auto kern = gemm_int8_kernel<P, F, sh.bm, sh.bn, sh.wm, sh.wn, sh.split>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  return launch_kernel(kern, dim3(grid), dim3(sh.wm * sh.wn * kWave), lds, stream, prm);
}

template <int P, int F>
inline hipError_t launch_p_shape(int shape, const Int8Params& prm, int grid, hipStream_t stream) {
  switch (shape) {
    case 0: return launch_shape<P, F, 0>(prm, grid, stream);
    case 1: return launch_shape<P, F, 1>(prm, grid, stream);
    case 2: return launch_shape<P, F, 2>(prm, grid, stream);
    case 3: return launch_shape<P, F, 3>(prm, grid, stream);
    case 4: return launch_shape<P, F, 4>(prm, grid, stream);
    case 5: return launch_shape<P, F, 5>(prm, grid, stream);
  }
  return hipErrorInvalidValue;
}

// One launch of shapes SA (grid ga) then SB (grid gb), when they pair.
template <int P, int F, int SA, int SB>
hipError_t launch_pair_shapes(const Int8Params& pa, int ga, const Int8Params& pb, int gb,
                              hipStream_t stream) {
  constexpr TileShape a = kShapes[SA], b = kShapes[SB];
  const size_t lds = std::max(lds_bytes<F>(a), lds_bytes<F>(b));
  auto kern = gemm_int8_pair_kernel<P, F, a.bm, a.bn, a.wm, a.wn, a.split, b.bm, b.bn, b.wm, b.wn,
                                    b.split>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  return launch_kernel(kern, dim3(ga + gb), dim3(a.wm * a.wn * kWave), lds, stream, pa, pb, ga);
}

// The shape pairs built as one launch (same wave count): 256x256 or 512x128
// main tiles with 256x128 (4x2) tail tiles (8 waves); 256x128 (4x1) main
// tiles with 128x128 or 256x128 (4x1) tail tiles (4 waves).
inline bool pair_supported(int sa, int sb) {
  return ((sa == 0 || sa == 4) && sb == 2) || (sa == 5 && (sb == 3 || sb == 5));
}

template <int P, int F>
inline hipError_t launch_p_pair(int sa, const Int8Params& pa, int ga, int sb, const Int8Params& pb,
                                int gb, hipStream_t stream) {
  if (sa == 0 && sb == 2) return launch_pair_shapes<P, F, 0, 2>(pa, ga, pb, gb, stream);
  if (sa == 4 && sb == 2) return launch_pair_shapes<P, F, 4, 2>(pa, ga, pb, gb, stream);
  if (sa == 5 && sb == 3) return launch_pair_shapes<P, F, 5, 3>(pa, ga, pb, gb, stream);
  if (sa == 5 && sb == 5) return launch_pair_shapes<P, F, 5, 5>(pa, ga, pb, gb, stream);
  return hipErrorInvalidValue;
}

// Launches for weight bits P (main kernel) and activation bits Q (expansion)
// in operand format fmt (0 int8; 1 FP4, P and Q <= 2; 2 FP4 weights with FP8
// activations, P <= 2, Q <= 4; other combinations return hipErrorInvalidValue);
// the explicit instantiations live in gemm_int8_inst.hip, built once per width.
template <int P>
hipError_t launch_for_p(int fmt, int shape, const Int8Params& prm, int grid, hipStream_t stream);
template <int P>
hipError_t launch_pair_for_p(int fmt, int sa, const Int8Params& pa, int ga, int sb,
                             const Int8Params& pb, int gb, hipStream_t stream);
template <int Q>
hipError_t launch_expand_for_q(int fmt, const uint32_t* a_packed, int M, int nchunks, int nsteps,
                               int mblocks, v4i* out, int* counters, int ncounters,
                               hipStream_t stream);

}  // namespace int8
}  // namespace apt
