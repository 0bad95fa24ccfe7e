/*
 * apt_oracle.c - plain CPU oracle for the WpAq bipolar-INT integer GEMM.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  It shares no code,
 * header, table or constant with the GPU library, and the GPU library never
 * calls it.
 *
 * Every function is the plain definition of what it computes, written for a
 * reader to check against the paper (APT-LLM, arXiv 2508.19087) by eye:
 *   - apt_oracle_convert:  the signed-INT -> bipolar-INT conversion of Sec. III-A
 *                          (flip the sign bit of the b-bit field);
 *   - apt_oracle_decode:   the bipolar-INT value equation of Sec. III-A,
 *                          (x)_D = sum_i (2 x^(i) - 1) 2^i, evaluated bit by bit;
 *   - apt_oracle_matmul*:  C = A W^T over the decoded values with 64-bit
 *                          accumulation (the product Y = WX of Sec. III-B,
 *                          which the bit-plane method reproduces exactly);
 *   - apt_oracle_rowsum:   the sum of decoded values of each row;
 *   - apt_oracle_pack / apt_oracle_unpack: the packed bit-plane layout of
 *                          Sec. IV-A as fixed by the library header (planes of
 *                          32-bit words, concatenated per 128-element chunk of
 *                          8-row groups).
 * No bit tricks, no planes, no popcounts on the multiply path.  The fp16 scale
 * epilogue is evaluated in float64 by the Python side of the oracle.
 *
 * Parity is pinned by the CPU tests: exhaustive round trips over every code at
 * b = 1..8, brute force with Python integers on tiny shapes, numpy int64
 * matmul, exhaustive 1x1x1 products, closed forms for constant inputs, the
 * XNOR-net identity at p = q = 1, and hand-derived fixtures.
 */
#include <omp.h>
#include <stddef.h>
#include <stdint.h>

/* Bipolar word from a signed b-bit code: keep the low b bits, then flip the
 * sign bit (Sec. III-A).  Returns 0, or -1 for bits outside [1, 8]. */
int apt_oracle_convert(const int8_t* x, int64_t n, int bits, uint8_t* u) {
  if (bits < 1 || bits > 8) return -1;
  unsigned mask = (1u << bits) - 1u;
  unsigned sign = 1u << (bits - 1);
  for (int64_t t = 0; t < n; ++t) {
    unsigned field = ((unsigned)(uint8_t)x[t]) & mask;
    u[t] = (uint8_t)(field ^ sign);
  }
  return 0;
}

/* Decimal value of an n-bit bipolar word, one bit at a time: each bit
 * contributes (2 bit - 1) * 2^i (Sec. III-A, value equation). */
int apt_oracle_decode(const uint8_t* u, int64_t n, int bits, int32_t* v) {
  if (bits < 1 || bits > 8) return -1;
  for (int64_t t = 0; t < n; ++t) {
    int32_t value = 0;
    for (int i = 0; i < bits; ++i) {
      int32_t bit = (u[t] >> i) & 1;
      int32_t weight = 1 << i;
      value += (2 * bit - 1) * weight;
    }
    v[t] = value;
  }
  return 0;
}

/* C[m][n] = sum_k va[m][k] * vw[n][k], accumulated in int64.  va is [M][K],
 * vw is [N][K], C is [M][N], all row-major.  Returns the number of entries
 * whose exact value does not fit in int32 (those entries are stored wrapped). */
int64_t apt_oracle_matmul(const int32_t* va, const int32_t* vw, int M, int N, int K,
                          int32_t* C) {
  int64_t overflow = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(+ : overflow)
  for (int m = 0; m < M; ++m) {
    for (int n = 0; n < N; ++n) {
      int64_t acc = 0;
      for (int k = 0; k < K; ++k)
        acc += (int64_t)va[(int64_t)m * K + k] * (int64_t)vw[(int64_t)n * K + k];
      if (acc > INT32_MAX || acc < INT32_MIN) overflow += 1;
      C[(int64_t)m * N + n] = (int32_t)(uint32_t)(uint64_t)acc;
    }
  }
  return overflow;
}

/* The same product for a list of (m, n) entries only: out[t] = C[m_idx[t]][n_idx[t]].
 * Used to check large problems on sampled outputs. */
int64_t apt_oracle_matmul_entries(const int32_t* va, const int32_t* vw, int K,
                                  const int32_t* m_idx, const int32_t* n_idx, int64_t count,
                                  int32_t* out) {
  int64_t overflow = 0;
#pragma omp parallel for schedule(static) reduction(+ : overflow)
  for (int64_t t = 0; t < count; ++t) {
    const int32_t* a = va + (int64_t)m_idx[t] * K;
    const int32_t* w = vw + (int64_t)n_idx[t] * K;
    int64_t acc = 0;
    for (int k = 0; k < K; ++k) acc += (int64_t)a[k] * (int64_t)w[k];
    if (acc > INT32_MAX || acc < INT32_MIN) overflow += 1;
    out[t] = (int32_t)(uint32_t)(uint64_t)acc;
  }
  return overflow;
}

/* out[r] = sum_k v[r][k] for v [R][K]. */
int apt_oracle_rowsum(const int32_t* v, int R, int K, int32_t* out) {
  for (int r = 0; r < R; ++r) {
    int64_t acc = 0;
    for (int k = 0; k < K; ++k) acc += v[(int64_t)r * K + k];
    out[r] = (int32_t)acc;
  }
  return 0;
}

/* Word index of (row r, chunk c, plane i, word w) in the packed layout: rows
 * in groups of 8, then chunk, then plane, then row within the group, then
 * word. */
static int64_t packed_word_index(int r, int c, int i, int w, int nchunks, int bits) {
  int64_t group = r / 8, slot = r % 8;
  return ((group * nchunks + c) * bits + i) * 32 + slot * 4 + w;
}

/* Reference packing of bipolar words u [R][K] into the documented layout:
 * plane i of element k of row r is bit (k mod 32) of word
 * packed_word_index(r, k/128, i, (k mod 128)/32).  Every other bit, including
 * all bits of the padding rows R..R_pad-1, is zero.  `packed` must hold
 * ceil(R/8)*8*NC*bits*4 words. */
int apt_oracle_pack(const uint8_t* u, int R, int K, int bits, uint32_t* packed) {
  if (bits < 1 || bits > 8 || R < 1 || K < 1) return -1;
  int nchunks = (K + 127) / 128;
  int64_t rpad = ((int64_t)R + 7) / 8 * 8;
  int64_t total = rpad * nchunks * bits * 4;
  for (int64_t t = 0; t < total; ++t) packed[t] = 0u;
  for (int r = 0; r < R; ++r) {
    for (int k = 0; k < K; ++k) {
      int c = k / 128, w = (k % 128) / 32, e = k % 32;
      for (int i = 0; i < bits; ++i) {
        uint32_t bit = (u[(int64_t)r * K + k] >> i) & 1u;
        packed[packed_word_index(r, c, i, w, nchunks, bits)] |= bit << e;
      }
    }
  }
  return 0;
}

/* Reads bipolar words u [R][K] back out of a packed buffer.  Returns the
 * number of padding elements (k >= K, or rows R..R_pad-1) with a set bit
 * (must be 0), or -1 on bad arguments. */
int64_t apt_oracle_unpack(const uint32_t* packed, int R, int K, int bits, uint8_t* u) {
  if (bits < 1 || bits > 8 || R < 1 || K < 1) return -1;
  int nchunks = (K + 127) / 128;
  int rpad = (R + 7) / 8 * 8;
  int64_t stray = 0;
  for (int r = 0; r < rpad; ++r) {
    for (int k = 0; k < nchunks * 128; ++k) {
      int c = k / 128, w = (k % 128) / 32, e = k % 32;
      unsigned value = 0;
      for (int i = 0; i < bits; ++i) {
        uint32_t bit = (packed[packed_word_index(r, c, i, w, nchunks, bits)] >> e) & 1u;
        value |= bit << i;
      }
      if (k < K && r < R)
        u[(int64_t)r * K + k] = (uint8_t)value;
      else
        stray += (value != 0);
    }
  }
  return stray;
}

/* Number of threads the parallel loops above use (built with -fopenmp). */
int apt_oracle_num_threads(void) { return omp_get_max_threads(); }
