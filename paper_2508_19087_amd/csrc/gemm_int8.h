// gemm_int8.h - the reassembled-int8 MFMA route of the WpAq bipolar-INT
// GEMM for gfx950 (APT-LLM, arXiv 2508.19087, Sec. III-B and IV-B).
//
// The bit-planes of each operand are merged back into one byte per element
// before the multiply (reassemble.h), so one v_mfma_i32_32x32x32_i8 covers
// every plane pair of an element pair; the paper's Sec. III-B sum over plane
// products is the same number by distributivity.
//
// Two kernels:
//   expand_a_kernel  once per call, the activations' planes are reassembled
//                    into operand bytes laid out as ready-made MFMA fragments
//                    (a workspace buffer), so the main kernel loads them with
//                    whole-line 1 KB reads straight into registers;
//   gemm_int8_kernel each workgroup owns one BM x BN output tile and every
//                    plane pair of it, as the paper's recovery-oriented
//                    scheduling does (Sec. IV-B).  K advances one 128-element
//                    chunk per pipeline step: the weight planes of the tile
//                    are fetched two chunks ahead, reassembled into a
//                    double-buffered LDS tile while the matrix cores work on
//                    the previous chunk, and the activation fragments of the
//                    next chunk are fetched k-step by k-step behind the MFMAs.
// Only the weights pass through LDS: staging both operands there would need
// as many LDS bytes per chunk as the MFMAs take cycles, and LDS would bound
// the kernel.
//
// Operand bytes are y = u (b <= 7) or u - 128 (b == 8) with bipolar value
// v = 2y + c.  Expanding sum_k v_a v_w over the real K gives the epilogue
//   C = 4 D - 4 (K_pad - K) y_pad,a y_pad,w + c_w R_a[m] + c_a R_w[n] - c_a c_w K,
// where D is the MFMA sum over K_pad, y_pad the operand byte of a padding
// element, and R the row sums of bipolar values from the packers.  The
// arithmetic is done modulo 2^32; the true C fits in int32 (checked by the
// host), so the wrapped result is exact.
#pragma once

#include "apt_internal.h"
#include "reassemble.h"

namespace apt {
namespace int8 {

constexpr int kWave = 64;
constexpr int kRowBytes = kChunk + 16;          // padded LDS row: 128 operand bytes + 16
constexpr int kStepBytes = 32;                  // K bytes per MFMA k-step
constexpr int kSteps = kChunk / kStepBytes;     // k-steps per chunk
constexpr int kFragVecs = kWave;                // one 32x32 fragment = 64 lanes x 16 bytes

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

// All-zero plane words: the weight planes of a chunk past the end (the main
// loop always runs an even number of chunks) are read from here, which makes
// them padding elements.  Large enough for any in-group offset of 8 planes.
static __device__ __attribute__((aligned(16))) uint32_t kZeroPlanes[512] = {};

struct Int8Params {
  GemmArgs g;
  int nchunks;        // NC, chunks of K
  int nsteps;         // k-steps in the activation fragment buffer (even chunk count x 4)
  int n_begin;        // first output column of this launch
  int tiles_n;
  int mblocks;        // 32-row blocks of the activation fragment buffer
  const v4i* a_frag;  // activation fragments (workspace)
  int ksplit;         // 1, or 2: each tile's K range is split between two workgroups
  v4i* partial;       // ksplit 2: one int32 partial tile per tile (workspace)
  int* flags;         // ksplit 2: partial-ready flag per tile (workspace, zeroed per call)
};

// Bytes of the activation fragment buffer for M rows and K.
inline size_t a_frag_bytes(int M, int K) {
  const int nce = (num_chunks(K) + 1) & ~1;
  return (size_t)((M + 31) / 32) * 32 * nce * kChunk;
}

// ---- activation expansion ---------------------------------------------------
// Fragment (mb, ks) holds k-step ks of rows 32 mb .. 32 mb + 31 in MFMA operand
// order: lane l (vector index ((mb * nsteps + ks) * 64 + l)) carries 16 bytes of
// row 32 mb + l mod 32, namely bytes 16 (l / 32) .. 16 (l / 32) + 15 of the
// k-step's 32 reassembled bytes.  Rows past M and chunks past the last one are
// expanded from all-zero planes (padding elements).
template <int Q>
__global__ __launch_bounds__(256) void expand_a_kernel(const uint32_t* __restrict__ a_packed, int M,
                                                       int nchunks, int nsteps, int mblocks,
                                                       v4i* __restrict__ out, int* __restrict__ flags,
                                                       int nflags) {
  const int rows = mblocks * 32;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  // The split-K flags of this call start cleared (the GEMM launches follow in
  // stream order).
  if (t < nflags) flags[t] = 0;
  if (t >= (int64_t)rows * (nsteps / kSteps)) return;
  const int row = (int)(t % rows);
  const int chunk = (int)(t / rows);
  uint32_t pw[kWordsPerPlane][Q];
  if (row < M && chunk < nchunks) {
    const uint32_t* src = a_packed + plane_words(row, chunk, 0, nchunks, Q);
#pragma unroll
    for (int j = 0; j < Q; ++j) {
      uint4 v = *reinterpret_cast<const uint4*>(src + j * kPlaneStride);
      pw[0][j] = v.x; pw[1][j] = v.y; pw[2][j] = v.z; pw[3][j] = v.w;
    }
  } else {
#pragma unroll
    for (int w = 0; w < kWordsPerPlane; ++w)
#pragma unroll
      for (int j = 0; j < Q; ++j) pw[w][j] = 0u;
  }
  const int mb = row / 32, l = row % 32;
#pragma unroll
  for (int w = 0; w < kWordsPerPlane; ++w) {
    uint32_t o[8];
    reassemble_word<Q>(pw[w], o);
    v4i* f = out + ((int64_t)mb * nsteps + chunk * kSteps + w) * kFragVecs;
    f[l] = v4i{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
    f[l + 32] = v4i{(int)o[4], (int)o[5], (int)o[6], (int)o[7]};
  }
}

// ---- weight staging -----------------------------------------------------------
// ROWS weight rows of a tile, each split into SPLIT items of 128/SPLIT elements
// (4/SPLIT words per plane).  Consecutive threads take consecutive rows of the
// same part, so a wave's LDS writes hit distinct banks.  Rows past the matrix
// edge are clamped to its last
// row: their products only reach outputs that are never stored, and the code
// stays branch-free so the scheduler can interleave it with the MFMAs.
template <int B, int ROWS, int SPLIT, int T>
struct Stage {
  static constexpr int kWpi = kWordsPerPlane / SPLIT;
  static constexpr int kItems = ROWS * SPLIT / T;
  static_assert(ROWS * SPLIT % T == 0 && kItems >= 1, "items must divide evenly");
  uint32_t raw[kItems][B][kWpi];

  // Loads chunk `chunk` of the item rows; a chunk at or past the end reads the
  // zero planes, i.e. padding elements.
  __device__ __forceinline__ void load(const uint32_t* __restrict__ packed, int row0, int rows,
                                       int nchunks, int chunk, int tid) {
    const bool real = chunk < nchunks;
#pragma unroll
    for (int it = 0; it < kItems; ++it) {
      const int item = tid + T * it;
      const int r = min(row0 + item % ROWS, rows - 1);
      const int sub = item / ROWS;
      const uint32_t* src = real ? packed + plane_words(r, chunk, 0, nchunks, B) + sub * kWpi
                                 : kZeroPlanes + (r % kRowGroup) * kWordsPerPlane + sub * kWpi;
#pragma unroll
      for (int i = 0; i < B; ++i) {
        if (kWpi == 4) {
          uint4 v = *reinterpret_cast<const uint4*>(src + i * kPlaneStride);
          raw[it][i][0] = v.x; raw[it][i][1] = v.y; raw[it][i][2] = v.z; raw[it][i][3] = v.w;
        } else if (kWpi == 2) {
          uint2 v = *reinterpret_cast<const uint2*>(src + i * kPlaneStride);
          raw[it][i][0] = v.x; raw[it][i][1] = v.y;
        } else {
          raw[it][i][0] = src[i * kPlaneStride];
        }
      }
    }
  }

  // Reassembles word u (0 <= u < kWords) of this thread's items into LDS.
  static constexpr int kWords = kItems * kWpi;
  __device__ __forceinline__ void store_word(uint8_t* lds_tile, int tid, int u) const {
    const int it = u / kWpi, w = u % kWpi;
    const int item = tid + T * it;
    const int r = item % ROWS;
    const int sub = item / ROWS;
    uint32_t pw[B];
#pragma unroll
    for (int i = 0; i < B; ++i) pw[i] = raw[it][i][w];
    uint32_t o[8];
    reassemble_word<B>(pw, o);
    uint4* d4 = reinterpret_cast<uint4*>(lds_tile + r * kRowBytes + (sub * kWpi + w) * kStepBytes);
    d4[0] = make_uint4(o[0], o[1], o[2], o[3]);
    d4[1] = make_uint4(o[4], o[5], o[6], o[7]);
  }

  __device__ __forceinline__ void store(uint8_t* lds_tile, int tid) const {
#pragma unroll
    for (int u = 0; u < kWords; ++u) store_word(lds_tile, tid, u);
  }
};

__host__ __device__ constexpr int offset_of(int b) { return b == 8 ? 1 : 1 - (1 << b); }
__host__ __device__ constexpr int pad_of(int b) { return b == 8 ? -128 : 0; }

// Scheduling hint for one k-step with N MFMAs: DS reads of the next k-step
// first, then each MFMA followed by VALU_PER vector instructions of the weight
// reassembly, with the LDS writes and the activation-fragment loads spread
// between the MFMAs.  Masks: 0x008 MFMA, 0x002 VALU, 0x100 DS read,
// 0x200 DS write, 0x020 VMEM read.
template <int I, int N, int READS, int WRITES, int VMEM, int VALU_PER>
struct Interleave {
  static __device__ __forceinline__ void run() {
    if constexpr (I < READS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if constexpr (VALU_PER > 0) __builtin_amdgcn_sched_group_barrier(0x002, VALU_PER, 0);
    if constexpr (WRITES > 0 && I >= N - 2 * WRITES && (I - (N - 2 * WRITES)) % 2 == 1)
      __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
    if constexpr (I < VMEM) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    Interleave<I + 1, N, READS, WRITES, VMEM, VALU_PER>::run();
  }
};
template <int N, int READS, int WRITES, int VMEM, int VALU_PER>
struct Interleave<N, N, READS, WRITES, VMEM, VALU_PER> {
  static __device__ __forceinline__ void run() {}
};

// ---- main kernel --------------------------------------------------------------
// The MFMA takes the weight fragment as its first operand, so the accumulator
// of lane l holds D[n][m] for m = l mod 32 and four consecutive n: each lane
// stores 16 contiguous output bytes.
template <int P, int BM, int BN, int WM, int WN, int SPLIT, bool HINTS>
__global__ __launch_bounds__(WM* WN* kWave) void gemm_int8_kernel(Int8Params prm) {
  constexpr int T = WM * WN * kWave;
  constexpr int WTM = BM / WM, WTN = BN / WN;  // wave tile
  constexpr int FM = WTM / 32, FN = WTN / 32;  // 32x32 fragments per wave
  constexpr int kStageBytes = BN * kRowBytes;
  static_assert(FM >= 1 && FN >= 1, "wave tile too small");
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];

  const GemmArgs& g = prm.g;
  const int NC = prm.nchunks;
  const int NCE = (NC + 1) & ~1;  // even chunk count; a last odd chunk is all padding
  const int c_mid = ((NCE / 2) + 1) & ~1;  // split point of the two K halves (even)
  const int tid = threadIdx.x;
  const int lane = tid % kWave;
  const int wave = tid / kWave;
  const int wm = wave / WN, wn = wave % WN;

  // Workgroups are dealt round-robin to the 8 XCDs, each with its own L2.
  // When the tile grid splits into 4 x 8 blocks of tiles, block k of XCD x
  // takes tile k of the x-th such block (one block fills the XCD's 32 CUs),
  // so concurrently running tiles share 4 activation bands and 8 weight
  // column blocks in that L2.  Otherwise each XCD takes a contiguous run of
  // row-major tiles.
  // With ksplit 2, workgroups 2t and 2t+1 share tile t: the even one takes
  // the first half of K and publishes its partial sums, the odd one takes the
  // second half, adds the partial and stores the tile.  Workgroups are
  // dispatched in index order, so a waiting odd workgroup's partner is
  // always already resident or done.
  const bool split = prm.ksplit == 2;
  const int half = split ? (int)(blockIdx.x & 1) : 0;
  const int bid = split ? (int)(blockIdx.x >> 1) : (int)blockIdx.x;
  const int ntiles = split ? (int)gridDim.x / 2 : (int)gridDim.x;
  const int tiles_m = ntiles / prm.tiles_n;
  int tm, tn;
  constexpr int kXcds = 8, kSM = 4, kSN = 8;
  if (split) {
    tm = bid / prm.tiles_n;
    tn = bid % prm.tiles_n;
  } else if (tiles_m % kSM == 0 && prm.tiles_n % kSN == 0 && ntiles % (kXcds * kSM * kSN) == 0) {
    const int xcd = blockIdx.x % kXcds, k = blockIdx.x / kXcds;
    const int super = (k / (kSM * kSN)) * kXcds + xcd, in = k % (kSM * kSN);
    const int supers_n = prm.tiles_n / kSN;
    tm = (super / supers_n) * kSM + in % kSM;
    tn = (super % supers_n) * kSN + in / kSM;
  } else {
    int tile = bid;
    if (ntiles % kXcds == 0) tile = (bid % kXcds) * (ntiles / kXcds) + bid / kXcds;
    tm = tile / prm.tiles_n;
    tn = tile % prm.tiles_n;
  }
  const int m0 = tm * BM, n0 = prm.n_begin + tn * BN;

  using SW = Stage<P, BN, SPLIT, T>;
  SW rw0, rw1;
  uint8_t* buf0 = lds;
  uint8_t* buf1 = lds + kStageBytes;

  v16i acc[FN][FM];
#pragma unroll
  for (int b = 0; b < FN; ++b)
#pragma unroll
    for (int a = 0; a < FM; ++a)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[b][a][v] = 0;

  // Activation fragments of this wave: 32-row blocks clamped to the buffer.
  const v4i* a_ptr[FM];
#pragma unroll
  for (int a = 0; a < FM; ++a) {
    const int mb = min((m0 + wm * WTM) / 32 + a, prm.mblocks - 1);
    a_ptr[a] = prm.a_frag + (int64_t)mb * prm.nsteps * kFragVecs + lane;
  }
  v4i afr[kSteps][FM];

  const int lrow = lane % 32;
  const int lk = (lane / 32) * 16;

  // One pipeline phase: the MFMAs of chunk c from LDS buffer `cst`, k-step by
  // k-step.  During k-step ks the weight fragments of ks+1 are read, one slice
  // of the next chunk's weight reassembly goes to LDS buffer `sst`, and the
  // activation fragment registers of ks are refilled with chunk c+1.  A
  // scheduling fence closes every k-step.
  auto phase = [&](const uint8_t* cst, uint8_t* sst, const SW& rw, int c) {
    const uint8_t* w_t = cst + (wn * WTN + lrow) * kRowBytes + lk;
    const int next_step = min(c + 1, NCE - 1) * kSteps;
    v4i wf[2][FN];
#pragma unroll
    for (int b = 0; b < FN; ++b) wf[0][b] = *reinterpret_cast<const v4i*>(w_t + b * 32 * kRowBytes);
#pragma unroll
    for (int ks = 0; ks < kSteps; ++ks) {
      const int cur = ks & 1, nxt = cur ^ 1;
      if (ks + 1 < kSteps) {
#pragma unroll
        for (int b = 0; b < FN; ++b)
          wf[nxt][b] = *reinterpret_cast<const v4i*>(w_t + b * 32 * kRowBytes + (ks + 1) * kStepBytes);
      }
#pragma unroll
      for (int u = ks * SW::kWords / kSteps; u < (ks + 1) * SW::kWords / kSteps; ++u)
        rw.store_word(sst, tid, u);
#pragma unroll
      for (int b = 0; b < FN; ++b)
#pragma unroll
        for (int a = 0; a < FM; ++a)
          acc[b][a] = __builtin_amdgcn_mfma_i32_32x32x32_i8(wf[cur][b], afr[ks][a], acc[b][a], 0, 0, 0);
#pragma unroll
      for (int a = 0; a < FM; ++a) afr[ks][a] = a_ptr[a][(int64_t)(next_step + ks) * kFragVecs];
      if constexpr (HINTS) {
        constexpr int words = (SW::kWords + kSteps - 1) / kSteps;  // at most, per k-step
        constexpr int valu = words * 40;
        Interleave<0, FN * FM, FN, 2 * words, FM, (valu + FN * FM - 1) / (FN * FM)>::run();
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  const int c_begin = (split && half == 1) ? c_mid : 0;
  const int c_end = (split && half == 0) ? c_mid : NCE;

  // Prologue: weight chunk c_begin into LDS buffer 0, the next one in
  // registers, activation fragments of chunk c_begin in registers.
  rw0.load(g.w_packed, n0, g.N, NC, c_begin, tid);
  rw1.load(g.w_packed, n0, g.N, NC, c_begin + 1, tid);
#pragma unroll
  for (int ks = 0; ks < kSteps; ++ks)
#pragma unroll
    for (int a = 0; a < FM; ++a) afr[ks][a] = a_ptr[a][(int64_t)(c_begin * kSteps + ks) * kFragVecs];
  rw0.store(buf0, tid);
  __syncthreads();

  // Two chunks per trip.  While the MFMAs of chunk c run, weight chunk c+1
  // (already in registers) is reassembled into the other LDS buffer and
  // weight chunk c+2 is fetched into the register set just consumed.
  for (int c = c_begin; c < c_end; c += 2) {
    rw0.load(g.w_packed, n0, g.N, NC, c + 2, tid);
    phase(buf0, buf1, rw1, c);
    __syncthreads();
    rw1.load(g.w_packed, n0, g.N, NC, c + 3, tid);
    phase(buf1, buf0, rw0, c + 1);
    __syncthreads();
  }

  if (split) {
    // Partial tile in accumulator order: vector ((wave * FN * FM * 4 + f) * 64 + lane).
    v4i* part = prm.partial + (int64_t)bid * (BM * BN / 4) + wave * (FN * FM * 4) * kWave + lane;
    if (half == 0) {
#pragma unroll
      for (int b = 0; b < FN; ++b)
#pragma unroll
        for (int a = 0; a < FM; ++a)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            part[((b * FM + a) * 4 + j) * kWave] =
                v4i{acc[b][a][4 * j], acc[b][a][4 * j + 1], acc[b][a][4 * j + 2], acc[b][a][4 * j + 3]};
      // Every wave's stores reach device scope (the partner runs on another
      // XCD, behind another L2) before one thread raises the flag.
      __threadfence();
      __syncthreads();
      if (tid == 0) __hip_atomic_store(prm.flags + bid, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
      return;
    }
    if (tid == 0) {
      // Bounded wait: the partner is resident or done, so the flag arrives.
      for (long spin = 0; spin < (1L << 28); ++spin) {
        if (__hip_atomic_load(prm.flags + bid, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) == 1) break;
        __builtin_amdgcn_s_sleep(2);
      }
    }
    __syncthreads();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
#pragma unroll
    for (int b = 0; b < FN; ++b)
#pragma unroll
      for (int a = 0; a < FM; ++a)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const v4i pv = __builtin_nontemporal_load(part + ((b * FM + a) * 4 + j) * kWave);
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[b][a][4 * j + i] += pv[i];
        }
  }

  // Epilogue.  Each 32x32 accumulator block goes through a private LDS slot
  // of the wave and comes back row by row, so that every store instruction
  // writes 8 whole 128-byte output rows; the affine correction and the
  // optional fp16 scaling are applied on the way out.
  const int q = g.q;
  const uint32_t ca = (uint32_t)(q == 8 ? 1 : 1 - (1 << q)), cw = (uint32_t)offset_of(P);
  const uint32_t pad_term =
      4u * (uint32_t)(NCE * kChunk - g.K) * (uint32_t)((q == 8 ? -128 : 0) * pad_of(P));
  const uint32_t const_term = ca * cw * (uint32_t)g.K + pad_term;
  constexpr int kEpiStride = 32 * 4 + 16;  // bytes per row of a 32x32 int32 block in LDS
  uint8_t* slot = lds + wave * 32 * kEpiStride;
  const int er = lane / 8, ec = (lane % 8) * 4;  // read-back row (+8 i) and first column
  const bool vec_ok = (g.N % 4) == 0;
  uint32_t wterm[FN][4];
#pragma unroll
  for (int b = 0; b < FN; ++b)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = min(n0 + wn * WTN + b * 32 + ec + j, g.N - 1);
      wterm[b][j] = ca * (uint32_t)g.w_rowsum[n];
    }
#pragma unroll
  for (int a = 0; a < FM; ++a) {
    const int mrow0 = m0 + wm * WTM + a * 32;
    uint32_t aterm[4];
    float sa[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = min(mrow0 + er + 8 * i, g.M - 1);
      aterm[i] = cw * (uint32_t)g.a_rowsum[m] - const_term;
      sa[i] = g.c_fp16 ? __half2float(g.a_scale[m]) : 0.f;
    }
#pragma unroll
    for (int b = 0; b < FN; ++b) {
      // acc[b][a][4 gi + j] = D[n = 8 gi + 4 (lane / 32) + j][m = lane mod 32]
#pragma unroll
      for (int gi = 0; gi < 4; ++gi) {
        v4i v = {acc[b][a][gi * 4 + 0], acc[b][a][gi * 4 + 1], acc[b][a][gi * 4 + 2],
                 acc[b][a][gi * 4 + 3]};
        *reinterpret_cast<v4i*>(slot + lrow * kEpiStride + (gi * 8 + (lane / 32) * 4) * 4) = v;
      }
      __builtin_amdgcn_s_waitcnt(0xc07f);  // LDS writes of this wave done (lgkmcnt 0)
      __builtin_amdgcn_wave_barrier();
      const int ncol = n0 + wn * WTN + b * 32 + ec;
      const bool full = vec_ok && ncol + 3 < g.N;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = mrow0 + er + 8 * i;
        const v4i d = *reinterpret_cast<const v4i*>(slot + (er + 8 * i) * kEpiStride + ec * 4);
        int32_t cv[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) cv[j] = (int32_t)(4u * (uint32_t)d[j] + aterm[i] + wterm[b][j]);
        if (m < g.M && ncol < g.N) {
          const int64_t o = (int64_t)m * g.N + ncol;
          if (g.c_int32) {
            if (full)
              *reinterpret_cast<int4*>(g.c_int32 + o) = make_int4(cv[0], cv[1], cv[2], cv[3]);
            else
              for (int j = 0; j < 4 && ncol + j < g.N; ++j) g.c_int32[o + j] = cv[j];
          }
          if (g.c_fp16) {
            __half h[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const int n = min(ncol + j, g.N - 1);
              h[j] = __float2half_rn((float)cv[j] * sa[i] * __half2float(g.w_scale[n]));
            }
            if (full)
              *reinterpret_cast<uint2*>(g.c_fp16 + o) = *reinterpret_cast<const uint2*>(h);
            else
              for (int j = 0; j < 4 && ncol + j < g.N; ++j) g.c_fp16[o + j] = h[j];
          }
        }
      }
      __builtin_amdgcn_s_waitcnt(0xc07f);  // reads done before the slot is rewritten
      __builtin_amdgcn_wave_barrier();
    }
  }
}

struct TileShape {
  int bm, bn, wm, wn, split;
  bool hints;
};
constexpr TileShape kShapes[] = {
    {256, 256, 4, 2, 2, false},
    {256, 256, 2, 4, 2, false},
    {256, 128, 4, 2, 4, false},
    {128, 128, 2, 2, 2, false},
    {256, 256, 4, 2, 2, true},
    {256, 256, 2, 2, 1, false},
};
constexpr int kNumShapes = sizeof(kShapes) / sizeof(kShapes[0]);

// Launches shape S over output columns [prm.n_begin, prm.n_begin + n_count).
template <int P, int S>
hipError_t launch_shape(const Int8Params& prm0, int n_count, hipStream_t stream) {
  constexpr TileShape sh = kShapes[S];
  Int8Params prm = prm0;
  prm.tiles_n = (n_count + sh.bn - 1) / sh.bn;
  const int tiles_m = (prm.g.M + sh.bm - 1) / sh.bm;
  const size_t lds = 2 * (size_t)sh.bn * kRowBytes;
  auto kern = gemm_int8_kernel<P, sh.bm, sh.bn, sh.wm, sh.wn, sh.split, sh.hints>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const int blocks = tiles_m * prm.tiles_n * (prm.ksplit == 2 ? 2 : 1);
  hipLaunchKernelGGL(kern, dim3(blocks), dim3(sh.wm * sh.wn * kWave), lds, stream, prm);
  return hipGetLastError();
}

template <int P>
inline hipError_t launch_p_shape(int shape, const Int8Params& prm, int n_count, hipStream_t stream) {
  switch (shape) {
    case 0: return launch_shape<P, 0>(prm, n_count, stream);
    case 1: return launch_shape<P, 1>(prm, n_count, stream);
    case 2: return launch_shape<P, 2>(prm, n_count, stream);
    case 3: return launch_shape<P, 3>(prm, n_count, stream);
    case 4: return launch_shape<P, 4>(prm, n_count, stream);
    case 5: return launch_shape<P, 5>(prm, n_count, stream);
  }
  return hipErrorInvalidValue;
}

// Launches for weight bits P (main kernel) and activation bits Q (expansion);
// the explicit instantiations live in gemm_int8_inst.hip, built once per width.
template <int P>
hipError_t launch_for_p(int shape, const Int8Params& prm, int n_count, hipStream_t stream);
template <int Q>
hipError_t launch_expand_for_q(const uint32_t* a_packed, int M, int nchunks, int nsteps,
                               int mblocks, v4i* out, int* flags, int nflags, hipStream_t stream);

}  // namespace int8
}  // namespace apt
