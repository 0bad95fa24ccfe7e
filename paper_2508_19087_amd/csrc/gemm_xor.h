// gemm_xor.h - the XOR + popcount route of the WpAq bipolar-INT GEMM for
// gfx950 (APT-LLM, arXiv 2508.19087, Sec. III-B).
//
// For bipolar bits a, w in {0,1} standing for 2a-1 and 2w-1,
// (2a-1)(2w-1) = 1 - 2 (a XOR w), so the plane product over K elements is
// Y(i,j) = K - 2 popc(W_i XOR A_j).  Recovery (Sec. III-B) then gives
//     C = sum_{i,j} 2^(i+j) Y(i,j) = K (2^p-1)(2^q-1) - 2 sum_{i,j} 2^(i+j) popc(W_i XOR A_j).
// Padding bits are zero in both operands, so they XOR to zero and the true K
// enters the constant term.
//
// This route streams the weight planes once, so it is the decode route
// (M <= 8, bound by HBM) and the route of small problems.
//
// Work split: every wave owns one whole 8-row group of weight rows and its
// whole K, for MT activation rows (MT = 1: one row, MT = 8: the 8 rows of an
// activation row group).  Lane l takes weight row slot l mod 8 and the chunks
// c = l / 8 + 8 t, so the 8 lanes that share a chunk read one 128-byte line
// per plane.  The chunks are walked in batches of kB per lane with two batches
// of weight words in flight: the loads of batch t + 2 are issued before batch
// t + 1 is used, so a lane keeps up to 2 kB P 16-byte loads outstanding
// (with one activation row, every load of a lane up to K = 16384 is issued
// before the first is used) and the latency of HBM is paid about once per
// wave, not once per batch; the popcounts consume the loads in the order
// they complete.  The weight loads carry the non-temporal hint: each weight byte is
// read once per call, and the hint measured 10-15% faster cold streaming
// than plain loads.  All 1-bit products of an output stay in
// registers (the register analogue of the paper's fragment-level recovery,
// Sec. IV-B); the 8 chunk lanes of a row meet through three lane shuffles, and
// nothing intermediate goes to memory.  A workgroup is W such waves side by
// side (W = 1, 2 or 4); they share only the copy of the activation chunks in
// LDS, so no wave waits for another after that copy.  With few row groups
// (short N, long K) the W waves of a workgroup instead share one row group
// and take every W-th chunk round (K split), so that more waves share the
// popcount work; their sums meet through LDS at the end.
#include "apt_internal.h"
#include "rowcode.h"

namespace apt {
namespace xorpop {

constexpr int kWave = 64;
constexpr int kMaxWaves = 4;                 // waves per workgroup, at most
constexpr int kChunkLanes = kWave / kRowGroup;  // lanes per row slot (8)
// LDS of the staged activation chunks, at most (bytes).
constexpr size_t kMaxActLds = 64 * 1024;

struct XorParams {
  GemmArgs g;
  int nchunks;   // NC, chunks of K
  int groups;    // row groups of the packed weights (padded N / 8)
  int ksplit;    // 1: each wave owns a row group; W > 1: the W waves of a
                 // workgroup share one and take every W-th chunk round
  // Fused activation source (SRC 1: int8 codes, 2: fp16 values, [M][K]),
  // converted per workgroup into the LDS copy; a_vec: 16-byte loads allowed
  // (K % 16 == 0 and a 16-byte aligned base).  SRC 2 writes each row's
  // bipolar scale to a_scale_out (if not NULL) from the first column block.
  const void* a_src;
  int a_vec;
  uint16_t* a_scale_out;
};

// Source of the activations: the packed planes, or (one activation row per
// block row) int8 codes or fp16 values converted inside the kernel.
enum { kSrcPacked = 0, kSrcCodes = 1, kSrcHalf = 2 };
// Rounds of 16 source elements per lane that the fused form holds in
// registers (requested before the weights); a longer row loads the rest after.
constexpr int kSrcHeld = 4;

// Activation chunk vectors per chunk in LDS: MT = 8 stages all 8 rows of each
// plane plus one pad vector (so that the 8 chunk lanes of a wave, which read
// 8 consecutive chunks at once, start 32 Q + 4 dwords apart and fall in
// different banks); MT = 1 stages the one row's Q vectors.  The copy covers
// the chunks rounded up to a multiple of 8 (one chunk per lane and round),
// the chunks past K as zeros.
template <int Q, int MT>
__host__ __device__ constexpr int act_chunk_vecs() { return MT == 8 ? Q * kRowGroup + 1 : Q; }
__host__ __device__ constexpr int staged_chunks(int nchunks) {
  return (nchunks + kChunkLanes - 1) / kChunkLanes * kChunkLanes;
}

// Chunks per lane per batch: about 8 16-byte weight loads per batch, or 16
// in the deep form (one activation row and K past one plain batch per lane:
// with two batches in flight every load of a lane up to K = 16384 at p = 2
// is issued before the first is used).
template <int P, bool DEEP>
__host__ __device__ constexpr int batch_chunks() {
  return DEEP ? (P >= 16 ? 1 : 16 / P) : (P >= 8 ? 1 : 8 / P);
}
// Activation vectors each thread loads into registers before the weight
// loads are issued (the rest of a larger copy is loaded after them).
constexpr int kStagePre = 4;
// Cache policy of the weight loads: non-temporal.
constexpr int kNT = 2;

typedef uint32_t v4u __attribute__((ext_vector_type(4)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t xor_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, 0x00020000);
}

// Every load below is a buffer load whose offset is past the resource's end
// when its element does not exist (a chunk past K, a row group past N, a
// vector past the copy): such loads return zeros without touching memory.
// The loads are therefore unconditional (no branch) and their waits count
// exactly; a zero weight word meets a zero activation word in the chunks
// between K and the end of the last round, which adds nothing to any
// popcount.
template <int P, int Q, int MT, bool DEEP, bool kALds, int SRC = kSrcPacked>
__global__ __launch_bounds__(kWave* kMaxWaves) void gemm_xor_kernel(XorParams prm) {
  static_assert(SRC == kSrcPacked || kALds, "the fused source builds the LDS copy");
  extern __shared__ uint4 a_lds[];
  const GemmArgs& g = prm.g;
  const int NC = prm.nchunks;
  const int m0 = blockIdx.y * MT;
  const int mrows = min(MT, g.M - m0);
  const int lane = threadIdx.x % kWave;
  const int wave = threadIdx.x / kWave;
  const int slot = lane % kRowGroup;
  const int cl = lane / kRowGroup;
  const int KW = prm.ksplit;
  const int kv = KW > 1 ? wave : 0;  // this wave's share of the chunk rounds
  const int rg = __builtin_amdgcn_readfirstlane(KW > 1 ? (int)blockIdx.x
                                                       : blockIdx.x * (int)(blockDim.x / kWave) + wave);
  const bool rv = rg < prm.groups;

  // ---- activation chunks: rows m0 .. m0 + MT - 1 (all in the row group
  // m0 / 8), ordered (chunk, plane, row) in the packed buffer.  The first
  // vectors of the LDS copy are requested before the weight loads: loads
  // complete in order, so a copy requested after them would wait for the
  // whole weight stream before the first popcount could start.
  constexpr int kAV = act_chunk_vecs<Q, MT>();
  const uint4* a_src = reinterpret_cast<const uint4*>(g.a_packed) +
                       (int64_t)(m0 / kRowGroup) * NC * Q * kRowGroup;
  const __amdgpu_buffer_rsrc_t a_rsrc = xor_rsrc(a_src, (uint32_t)NC * Q * kRowGroup * 16u);
  const int a_row = MT == 1 ? m0 % kRowGroup : 0;
  const int NS = staged_chunks(NC);
  const int n_vec = MT == 8 ? NS * Q * kRowGroup : NS * Q;  // staged vectors
  // vector t of the copy (zeros past chunk NC)
  auto a_at = [&](int t) __attribute__((always_inline)) -> uint4 {
    const uint32_t v = MT == 8 ? (uint32_t)t : (uint32_t)t * kRowGroup + a_row;
    const uint32_t off = t < n_vec ? v * 16u : 0xFFFFFFF0u;
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(a_rsrc, off, 0, 0));
  };
  auto lds_at = [&](int t) __attribute__((always_inline)) -> int {
    return MT == 8 ? t + t / (Q * kRowGroup) : t;
  };
  uint4 pre[kStagePre];
  if (kALds && SRC == kSrcPacked) {
#pragma unroll
    for (int k = 0; k < kStagePre; ++k) pre[k] = a_at(threadIdx.x + k * (int)blockDim.x);
  }
  // Fused source: for each of the block row's activation rows, lane t takes
  // elements 16 t + 16 L r, r = 0, 1, ... (L lanes in the workgroup) up to the
  // padded row length 128 NS.  The first kHeld rounds of every row are
  // requested here, before the weights.
  using CodeSrc = rowcode::CodeRow<false, Q>;
  using CodeVec = rowcode::CodeRow<true, Q>;
  using HalfSrc = rowcode::HalfRow<false, Q>;
  using HalfVec = rowcode::HalfRow<true, Q>;
  constexpr int kSrcDwords = SRC == kSrcHalf ? HalfSrc::kDwords : CodeSrc::kDwords;
  constexpr int kElemBytes = SRC == kSrcHalf ? 2 : 1;
  constexpr int kSrcRows = SRC != kSrcPacked ? MT : 1;
  constexpr int kHeld = MT == 1 ? kSrcHeld : 1;
  const int src_step = (int)blockDim.x * rowcode::kLaneElems;
  const int src_rounds = (NS * kChunk + src_step - 1) / src_step;  // per row, uniform
  // row m of the block row: its K elements (reads past them return zeros)
  auto s_rsrc = [&](int m) __attribute__((always_inline)) {
    return xor_rsrc(static_cast<const uint8_t*>(prm.a_src) + (int64_t)(m0 + m) * g.K * kElemBytes,
                    (uint32_t)g.K * kElemBytes);
  };
  auto src_load = [&](__amdgpu_buffer_rsrc_t rs, int r, uint32_t* d) __attribute__((always_inline)) {
    const int k0 = r * src_step + (int)threadIdx.x * rowcode::kLaneElems;
    if (SRC == kSrcHalf) {
      if (prm.a_vec) HalfVec::load(rs, k0, d); else HalfSrc::load(rs, k0, d);
    } else {
      if (prm.a_vec) CodeVec::load(rs, k0, d); else CodeSrc::load(rs, k0, d);
    }
  };
  uint32_t sd[kSrcRows][kHeld][kSrcDwords];
  if (SRC != kSrcPacked) {
#pragma unroll
    for (int m = 0; m < kSrcRows; ++m) {
      if (m >= mrows) break;  // uniform
      const __amdgpu_buffer_rsrc_t rs = s_rsrc(m);
#pragma unroll
      for (int r = 0; r < kHeld; ++r)
        if (r < src_rounds) src_load(rs, r, sd[m][r]);
    }
  }

  // ---- weight batches
  constexpr int kB = batch_chunks<P, DEEP>();
  // chunk rounds of this wave: t = kv + KW u, u < T (round t holds chunks
  // 8 t .. 8 t + 7, one per chunk lane)
  const int T = (NS / kChunkLanes - kv + KW - 1) / KW;
  const uint32_t w_bytes = rv ? (uint32_t)NC * P * kRowGroup * 16u : 0u;
  const __amdgpu_buffer_rsrc_t w_rsrc =
      xor_rsrc(reinterpret_cast<const uint4*>(g.w_packed) + (int64_t)(rv ? rg : 0) * NC * P * kRowGroup,
               w_bytes);
  v4u wcur[kB][P], wnxt[kB][P];
  auto load = [&](v4u (&wv)[kB][P], int t0) __attribute__((always_inline)) {
#pragma unroll
    for (int b = 0; b < kB; ++b) {
      const int c = cl + kChunkLanes * (kv + KW * (t0 + b));
      // (the plane offset is added to it, so the offset of a missing chunk
      // stays below 2^32 - 2^12; a row group holds at most 2^31 bytes)
      const uint32_t off = c < NC ? (uint32_t)((c * P) * kRowGroup + slot) * 16u : 0x80000000u;
#pragma unroll
      for (int i = 0; i < P; ++i)
        wv[b][i] = __builtin_amdgcn_raw_buffer_load_b128(w_rsrc, off, i * kRowGroup * 16, kNT);
    }
  };
  load(wcur, 0);
  if (kB < T) load(wnxt, kB);

  // fused fp16 source: each row's bipolar scale, and the quotient constants
  __shared__ float s_row[SRC == kSrcHalf ? 3 * MT : 1];
  if (kALds && SRC == kSrcPacked) {
#pragma unroll
    for (int k = 0; k < kStagePre; ++k) {
      const int t = threadIdx.x + k * (int)blockDim.x;
      if (t < n_vec) a_lds[lds_at(t)] = pre[k];
    }
    for (int t = threadIdx.x + kStagePre * (int)blockDim.x; t < n_vec; t += blockDim.x)
      a_lds[lds_at(t)] = a_at(t);
    __syncthreads();
  }
  if (SRC != kSrcPacked) {
    // The conversion of the packer (Sec. III-A, and for fp16 the bipolar form
    // of the per-row linear quantizer), with the plane words stored in the
    // LDS layout of act(): word w of plane j of chunk c of row m at dword
    // 4 (c kAV + j) + w (MT = 1) or 4 (c kAV + 8 j + m) + w (MT = 8).  Rounds
    // past kHeld are loaded (again) here.
    uint32_t* lds32 = reinterpret_cast<uint32_t*>(a_lds);
    if (SRC == kSrcHalf) {
      __shared__ uint32_t s_red[MT][kMaxWaves];
      const int nw = (int)(blockDim.x / kWave);
#pragma unroll
      for (int m = 0; m < kSrcRows; ++m) {
        if (m >= mrows) break;  // uniform
        rowcode::ushort2_t mm = {0, 0};
#pragma unroll
        for (int r = 0; r < kHeld; ++r)
          if (r < src_rounds) mm = HalfSrc::fold_max(mm, sd[m][r]);
        const __amdgpu_buffer_rsrc_t rs = s_rsrc(m);
        for (int r = kHeld; r < src_rounds; ++r) {
          uint32_t d[kSrcDwords];
          src_load(rs, r, d);
          mm = HalfSrc::fold_max(mm, d);
        }
        uint32_t v = max((uint32_t)mm.x, (uint32_t)mm.y);
        for (int off = kWave / 2; off > 0; off >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, off));
        if (lane == 0) s_red[m][wave] = v;
      }
      __syncthreads();
      if ((int)threadIdx.x < mrows) {
        const int m = threadIdx.x;
        uint32_t v = 0u;
        for (int w = 0; w < nw; ++w) v = max(v, s_red[m][w]);
        float rh, s2;
        const uint16_t s16 = rowcode::row_scale<Q>(v, rh, s2);
        s_row[3 * m] = __half2float(__ushort_as_half(s16));
        s_row[3 * m + 1] = rh;
        s_row[3 * m + 2] = s2;
        if (prm.a_scale_out != nullptr && blockIdx.x == 0) prm.a_scale_out[m0 + m] = s16;
      }
      __syncthreads();
    }
    const bool odd = (lane & 1) != 0;
    // uniform in r: both lanes of a pair run every round (DPP swap)
    auto convert = [&](int m, int r, const uint32_t* d, float rh, float s2) __attribute__((always_inline)) {
      const int k0 = r * src_step + (int)threadIdx.x * rowcode::kLaneElems;
      uint32_t u[4];
      if (SRC == kSrcHalf) HalfSrc::words(d, rh, s2, u); else CodeSrc::words(d, rh, s2, u);
#pragma unroll
      for (int t = 0; t < 4; ++t) {  // elements past K: all-zero words
        const int n_valid = g.K - (k0 + 4 * t);
        u[t] &= n_valid >= 4 ? 0xFFFFFFFFu : (n_valid <= 0 ? 0u : ((1u << (8 * n_valid)) - 1u));
      }
      uint32_t alo = u[0], ahi = u[1], blo = u[2], bhi = u[3];
      rowcode::transpose8x8<Q>(alo, ahi);
      rowcode::transpose8x8<Q>(blo, bhi);
      const int c = k0 / kChunk;
      uint32_t* dst = lds32 + (c * kAV + (MT == 8 ? m : 0)) * kWordsPerPlane + (k0 % kChunk) / 32;
      constexpr int kPlaneDwords = (MT == 8 ? kRowGroup : 1) * kWordsPerPlane;
#pragma unroll
      for (int i = 0; i < Q; i += 2) {
        const uint32_t wv = rowcode::plane_word(i < 4 ? alo : ahi, i < 4 ? blo : bhi, i % 4, odd);
        if (k0 < NS * kChunk && (!odd || i + 1 < Q)) dst[(i + (odd ? 1 : 0)) * kPlaneDwords] = wv;
      }
    };
#pragma unroll
    for (int m = 0; m < kSrcRows; ++m) {
      if (m >= mrows) break;  // uniform
      const float rh = SRC == kSrcHalf ? s_row[3 * m + 1] : 0.0f;
      const float s2 = SRC == kSrcHalf ? s_row[3 * m + 2] : 0.0f;
#pragma unroll
      for (int r = 0; r < kHeld; ++r)
        if (r < src_rounds) convert(m, r, sd[m][r], rh, s2);
      const __amdgpu_buffer_rsrc_t rs = s_rsrc(m);
      for (int r = kHeld; r < src_rounds; ++r) {
        uint32_t d[kSrcDwords];
        src_load(rs, r, d);
        convert(m, r, d, rh, s2);
      }
    }
    __syncthreads();
  }
  // vector of chunk c, plane j, row m (zeros for c >= NC)
  auto act = [&](int c, int j, int m) __attribute__((always_inline)) -> uint4 {
    if (kALds) return MT == 8 ? a_lds[c * kAV + j * kRowGroup + m] : a_lds[c * kAV + j];
    const uint32_t v = (uint32_t)(c * Q + j) * kRowGroup + (MT == 8 ? m : a_row);
    return __builtin_bit_cast(
        uint4, __builtin_amdgcn_raw_buffer_load_b128(a_rsrc, c < NC ? v * 16u : 0xFFFFFFF0u, 0, 0));
  };

  // One activation row, plain batches: the first batch's activation vectors
  // are read from LDS into registers before the first weight word is awaited,
  // so that no LDS read waits behind the weight stream (cold 4096 x 4096 W2A2:
  // 3.07 against 3.19 us; at most 16 vectors, 64 registers).
  constexpr int kPre = (MT == 1 && !DEEP && kALds && kB * Q <= 16) ? kB : 0;
  uint4 apre[kPre > 0 ? kPre : 1][Q];
  if (kPre > 0) {
#pragma unroll
    for (int b = 0; b < kPre; ++b) {
      if (b >= T) break;  // uniform
      const int c = cl + kChunkLanes * (kv + KW * b);
#pragma unroll
      for (int j = 0; j < Q; ++j) apre[b][j] = act(c, j, 0);
    }
  }
  uint32_t S[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) S[m] = 0u;
  auto compute = [&](const v4u (&wv)[kB][P], int t0) __attribute__((always_inline)) {
#pragma unroll
    for (int b = 0; b < kB; ++b) {
      if (t0 + b >= T) break;  // uniform: past the last round
      const int c = cl + kChunkLanes * (kv + KW * (t0 + b));
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        if (m >= mrows) break;  // uniform
#pragma unroll
        for (int j = 0; j < Q; ++j) {
          const uint4 av = (kPre > 0 && t0 == 0) ? apre[b < kPre ? b : 0][j] : act(c, j, m);
          uint32_t s = 0u;
#pragma unroll
          for (int i = 0; i < P; ++i) {
            uint32_t cnt = __builtin_popcount(wv[b][i][0] ^ av.x);
            cnt += __builtin_popcount(wv[b][i][1] ^ av.y);
            cnt += __builtin_popcount(wv[b][i][2] ^ av.z);
            cnt += __builtin_popcount(wv[b][i][3] ^ av.w);
            s += cnt << i;
          }
          S[m] += s << j;
        }
      }
    }
  };
  for (int t0 = 0; t0 < T; t0 += kB) {
    compute(wcur, t0);
    if (t0 + kB < T) {
#pragma unroll
      for (int b = 0; b < kB; ++b)
#pragma unroll
        for (int i = 0; i < P; ++i) wcur[b][i] = wnxt[b][i];
      if (t0 + 2 * kB < T) load(wnxt, t0 + 2 * kB);
    }
  }

  // ---- sum over the 8 chunk lanes of each row slot
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    S[m] += __shfl_xor(S[m], 8);
    S[m] += __shfl_xor(S[m], 16);
    S[m] += __shfl_xor(S[m], 32);
  }

  // ---- K split: the waves' sums meet in LDS, wave 0 finishes
  if (KW > 1) {
    __shared__ uint32_t red[kMaxWaves][MT][kRowGroup];
    if (cl == 0) {
#pragma unroll
      for (int m = 0; m < MT; ++m) red[wave][m][slot] = S[m];
    }
    __syncthreads();
    if (wave != 0) return;
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      uint32_t tot = 0u;
      for (int v = 0; v < KW; ++v) tot += red[v][m][slot];
      S[m] = tot;
    }
  }

  // ---- outputs: lane (cl, slot) writes activation row m0 + cl (MT = 8) or
  // m0 (MT = 1, lanes with cl = 0) of weight row 8 rg + slot
  const int m = MT == 8 ? cl : 0;
  const int n = rg * kRowGroup + slot;
  if (m >= mrows || (MT == 1 && cl != 0) || !rv || n >= g.N) return;
  const int mg = m0 + m;
  const uint32_t kabq = (uint32_t)g.K * ((1u << P) - 1u) * ((1u << Q) - 1u);
  uint32_t tot = S[0];
#pragma unroll
  for (int mm = 1; mm < MT; ++mm)
    if (m == mm) tot = S[mm];
  const int32_t c = (int32_t)(kabq - 2u * tot);
  const int64_t o = (int64_t)mg * g.N + n;
  if (g.c_int32) g.c_int32[o] = c;
  if (g.c_fp16) {
    float f;
    if (g.a_zero) {
      const float sw = __half2float(g.w_scale[n]), zw = __half2float(g.w_zero[n]);
      f = affine_value(c, __half2float(g.a_scale[mg]), sw, zw, (float)g.a_rowsum[mg],
                       __half2float(g.a_zero[mg]), sw * (float)g.w_rowsum[n] + (float)g.K * zw);
    } else {
      f = (float)c * (SRC == kSrcHalf ? s_row[3 * m] : __half2float(g.a_scale[mg]));
      f = f * __half2float(g.w_scale[n]);
    }
    g.c_fp16[o] = __float2half_rn(f);
  }
}

// Launch shape of one XOR-route call (resolved from the config by the host).
struct XorLaunch {
  bool deep;   // deep batches (batch_chunks)
  int ksplit;  // waves sharing one row group (1 = none)
  int mt;      // activation rows per block row (1 or 8)
  int waves;   // waves per workgroup (1, 2 or 4)
  bool lds;    // activation chunks staged in LDS
  size_t lds_bytes;
  dim3 grid;
  int src;     // kSrcPacked, or a fused source (needs mt = 1 and lds)
};

// Launch with `lds` bytes of dynamic LDS; past 48 KB (with the kernel's own
// static arrays the workgroup then nears 64 KB) the kernel's limit is raised
// first.
template <class Kernel>
inline hipError_t launch_lds(Kernel kern, const XorLaunch& L, hipStream_t s, const XorParams& prm) {
  if (L.lds_bytes > 48 * 1024) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)L.lds_bytes);
    if (e != hipSuccess) return e;
  }
  return launch_kernel(kern, L.grid, dim3(kWave * L.waves), L.lds_bytes, s, prm);
}

template <int P, int Q, int MT, bool DEEP>
inline hipError_t launch_mt(const XorParams& prm, const XorLaunch& L, hipStream_t s) {
  if (L.src == kSrcCodes) return launch_lds(gemm_xor_kernel<P, Q, MT, DEEP, true, kSrcCodes>, L, s, prm);
  if (L.src == kSrcHalf) return launch_lds(gemm_xor_kernel<P, Q, MT, DEEP, true, kSrcHalf>, L, s, prm);
  if (L.lds) return launch_lds(gemm_xor_kernel<P, Q, MT, DEEP, true>, L, s, prm);
  return launch_kernel(gemm_xor_kernel<P, Q, MT, DEEP, false>, L.grid, dim3(kWave * L.waves), 0, s, prm);
}

template <int P, int Q>
inline hipError_t launch_pq(const XorParams& prm, const XorLaunch& L, hipStream_t s) {
  if (L.mt == 1) return L.deep ? launch_mt<P, Q, 1, true>(prm, L, s) : launch_mt<P, Q, 1, false>(prm, L, s);
  return launch_mt<P, Q, 8, false>(prm, L, s);
}

// Launch for weight bits P and any activation bits; one explicit
// instantiation per P lives in gemm_xor_inst.hip (built once per P).
template <int P>
hipError_t launch_for_p(int q, const XorParams& prm, const XorLaunch& L, hipStream_t s);

}  // namespace xorpop
}  // namespace apt
