/*
 * apt.h - C ABI of the WpAq bipolar-INT bit-plane integer GEMM for AMD gfx950.
 *
 * The library computes C = A * W^T for signed p-bit weight codes W [N][K] and
 * signed q-bit activation codes A [M][K] (1 <= p, q <= 8), the arbitrary
 * precision integer matrix multiply of APT-LLM (arXiv 2508.19087, Sec. III),
 * plus an optional fp16 per-token x per-channel scale epilogue.
 *
 * Number format (Sec. III-A, the bipolar-INT value equation): an n-bit word
 * u = u^(n-1) ... u^(0) has the value (u)_D = sum_i (2 u^(i) - 1) 2^i, so each
 * bit stands for -1 or +1.  A signed n-bit code x becomes the bipolar word by
 * flipping its sign bit, u = (x mod 2^n) XOR 2^(n-1), and then (u)_D = 2x + 1
 * (Sec. III-A, the signed-to-bipolar correspondence).  The conversion is exact;
 * a quantiser's scale s becomes s/2 in bipolar form (Sec. III-A, the rewrite of
 * the linear quantisation formula), so the scales passed to apt_gemm are the
 * bipolar ones.
 *
 * The integer result is C[m][n] = sum_{k<K} (uA[m][k])_D * (uW[n][k])_D, which
 * Sec. III-B obtains as sum_{i,j} 2^(i+j) Y^(i,j) over the 1-bit plane products.
 *
 * Conventions shared by every call:
 *   - Pointers marked "device" are device pointers owned by the caller (for
 *     example torch tensors' data_ptr()).  The library never allocates or frees
 *     memory on these paths.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     Calls that take a stream validate their arguments on the host, enqueue
 *     their kernels on that stream and return without synchronising.
 *   - No call launches anything when validation fails.
 *   - The only mutable state the library holds is the configuration table that
 *     apt_search_config fills; a lock guards it, and calls are thread-safe.
 *     Everything else a call uses lives in its arguments, so calls on
 *     different streams may run at the same time as long as they share no
 *     output or workspace (apt_gemm_noalloc, which uses the library's one
 *     fixed workspace, is the exception).
 *   - Codes outside the signed b-bit range are reduced modulo 2^b (only the low
 *     b bits of each int8 code are used).
 *
 * Packed bit-plane layout (Sec. IV-A: decompose into n 1-bit matrices, pack
 * bits into 32-bit unsigned words, concatenate the planes):
 *   K_pad = ceil(K / 128) * 128, NC = K_pad / 128 chunks per row;
 *   rows are grouped by 8, R_pad = ceil(R / 8) * 8.
 *   The buffer holds R_pad * NC * b * 4 little-endian uint32 words:
 *       word index  ((g * NC + c) * b + i) * 32 + s * 4 + w,
 *       g = r / 8, s = r mod 8, 0 <= w < 4,
 *   and bit e (LSB = 0) of that word is bit i of the bipolar word u[r][k] with
 *       k = 128 c + 32 w + e.
 *   Bits with k >= K, and all bits of rows r >= R, are zero.  A 128-byte line
 *   holds one plane of one chunk for 8 consecutive rows, and all b planes of
 *   a chunk of those rows are one contiguous b*128-byte block, so a tile of
 *   rows moves with whole-line transfers.  Buffers must be 16-byte aligned.
 *
 * Row sums: rowsum[r] = sum_{k<K} (u[r][k])_D, the sum of the bipolar values of
 * row r (= sum of 2x+1).  apt_gemm routes that contract 8-bit operands on the
 * matrix cores use them for the exact affine correction of the operand offset.
 */
#ifndef APT_H
#define APT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  APT_OK = 0,
  APT_ERR_INVALID_ARG = 1, /* bad size, bit width, pointer, alignment or combination */
  APT_ERR_UNSUPPORTED = 2, /* the int32 result cannot hold K (2^p-1) (2^q-1), or the config is not buildable */
  APT_ERR_HIP = 3,         /* the HIP runtime reported an error on launch */
  APT_ERR_WORKSPACE = 4    /* the workspace is missing or too small */
} apt_status_t;

/* GEMM routes.  All compute the same int32 result. */
enum {
  APT_ROUTE_AUTO = 0,       /* let apt_select_config decide */
  APT_ROUTE_XOR = 1,        /* XOR + popcount on packed words, cross-lane reduction (Sec. III-B, 1-bit XOR form) */
  APT_ROUTE_PM1_MFMA = 2,   /* every (i, j) plane pair as +-1 int8 operands on the int8 matrix cores */
  APT_ROUTE_INT8_MFMA = 3,  /* planes reassembled in LDS into one int8 operand, one int8 MFMA per element pair */
  APT_ROUTE_FP4_MFMA = 4,   /* as APT_ROUTE_INT8_MFMA with the bipolar values as operands of the
                               block-scaled MFMA: FP4 (E2M1) weights, p <= 2, and FP4 (q <= 2) or
                               FP8 E4M3 (q <= 4) activations; K_pad (2^p-1)(2^q-1) < 2^24,
                               K_pad = K rounded up to a multiple of 128 */
  APT_ROUTE_FP6_MFMA = 5,   /* as APT_ROUTE_FP4_MFMA with FP6 (E2M3) weights and activations,
                               p, q <= 3; K_pad (2^p-1)(2^q-1) < 2^24 */
  APT_ROUTE_FP8_MFMA = 6    /* as APT_ROUTE_FP4_MFMA with FP8 (E4M3) weights and activations,
                               p, q <= 4; K_pad (2^p-1)(2^q-1) < 2^24 */
};

/* Kernel configuration (the tunable hyperparameters of Sec. V-A in gfx950
 * terms).  Fields a route does not use are ignored.  Everything said of the
 * int8 MFMA route below holds for the FP4 MFMA route too (same tile shapes,
 * grids and split launches).
 *   route      APT_ROUTE_*
 *   bm, bn     output tile per workgroup (int8 MFMA route: 256x256 with 4x2 or
 *              2x4 waves, 512x128 with 8x1, 256x128 with 4x2 or 4x1, 128x128
 *              with 2x2; the 4-wave shapes run two workgroups per compute unit)
 *   bk         K elements staged per pipeline step (MFMA routes: 0 or 128)
 *   waves_m, waves_n   wave grid inside a workgroup (int8 MFMA route); XOR
 *              route: waves_m = waves per workgroup, each owning one 8-row
 *              group of weight rows (0 = chosen by the library, or 1, 2, 4),
 *              waves_n = K split: 2 or 4 waves of a workgroup share one row
 *              group and divide its K (1 = none, 0 = chosen by the library)
 *   grid       int8 MFMA route: persistent workgroups, 0..4096.  0 = one
 *              workgroup per tile.  Otherwise each workgroup takes
 *              floor(T / grid) whole tiles (T tiles in all) and the K chunks of
 *              the remaining tiles are divided evenly among all workgroups
 *              (stream-K); workgroups sharing a tile combine int32 partial
 *              sums through the workspace.  The result does not depend on it.
 *   lds_stages depth of the weight LDS ring (int8 MFMA route: 0 or 3; the
 *              +-1 plane route ignores it)
 *   mt         XOR route: activation rows per block row: 1, 8, or 0 =
 *              chosen by the library (1 for M = 1, for M <= 2 below 2048
 *              row groups of 8 weight rows, and below 1024 row groups unless
 *              K > 7168 and M > 2; else 8)
 *   split_n    int8 MFMA route: 0, or a multiple of bn with 0 < split_n < N
 *              and of 8: columns [0, split_n) use the tile above and columns
 *              [split_n, N) a second launch with tile tail_bm x tail_bn (of
 *              the shapes of that size, the one with the main tile's wave
 *              count, else the first) and tail_grid persistent workgroups
 *              (same meaning as grid); main and tail share one launch when
 *              their wave counts match and the pair is built
 *   reserved   ignored
 */
typedef struct {
  int32_t route;
  int32_t bm, bn, bk;
  int32_t waves_m, waves_n;
  int32_t grid;
  int32_t lds_stages;
  int32_t mt;
  int32_t split_n;
  int32_t tail_bm, tail_bn;
  int32_t tail_grid;
  int32_t reserved[3];
} apt_config_t;

/* Bytes of a packed buffer for `rows` rows of K codes at `bits` bits
 * (ceil(rows/8) * 8 * ceil(K/128) * bits * 16).  Returns 0 for rows < 1,
 * K < 1 or bits outside [1, 8]. */
size_t apt_packed_bytes(int rows, int K, int bits);

/* Converts signed p-bit weight codes to bipolar-INT and packs the bit-planes
 * (Sec. III-A conversion; Sec. IV-A steps 1-3).
 *   w_codes   device, int8 [N][K] row-major, signed p-bit codes
 *   w_packed  device, apt_packed_bytes(N, K, p) bytes, 16-byte aligned, fully written
 *   w_rowsum  device, int32 [N] or NULL; receives the row sums defined above
 * Errors: APT_ERR_INVALID_ARG for N < 1, K < 1, p outside [1, 8], NULL codes or
 * packed pointer, or a misaligned packed pointer; APT_ERR_UNSUPPORTED for
 * K > 2^30; APT_ERR_HIP on launch failure. */
apt_status_t apt_pack_weights(const int8_t* w_codes, int N, int K, int p,
                              void* w_packed, int32_t* w_rowsum, void* stream);

/* The same conversion and packing for signed q-bit activation codes
 * a_codes [M][K] (device, int8).  "Quantize" is the lossless re-quantisation of
 * signed INT codes into bipolar-INT (Sec. III-A); the codes themselves come
 * from the caller.  Arguments and errors as apt_pack_weights. */
apt_status_t apt_quantize_pack_activations(const int8_t* a_codes, int M, int K, int q,
                                           void* a_packed, int32_t* a_rowsum, void* stream);

/* Quantizes fp16 activations per row (token) to q-bit bipolar-INT codes and
 * packs them as apt_quantize_pack_activations does, in one kernel.  The paper
 * quantizes activations linearly and rewrites the quantizer in bipolar form,
 * value 2x + 1 with half the signed scale (Sec. III-A); it fixes neither the
 * scale rule nor the rounding, so this library uses, per row m:
 *   s_m = fp16(absmax_k |a[m][k]| / (2^q - 1))   (IEEE fp32 divide, then RNE)
 *   level(a) = 2 floor(t / 2) + 1 of t = a / s_m (IEEE fp32 divide), clamped
 *              to +-(2^q - 1): the nearest odd integer to t, ties upward;
 *   t = 0 (level +1, dequantizing to 0) when s_m = 0.
 * s_m is the bipolar scale the GEMM's fp16 epilogue takes as a_scale.
 *   a_fp16    device, fp16 bits [M][K] row-major; values must be finite (a NaN
 *             or infinity yields unspecified codes and scale for its row)
 *   a_packed  device, apt_packed_bytes(M, K, q) bytes, 16-byte aligned, fully written
 *   a_rowsum  device, int32 [M] or NULL; receives the row sums defined above
 *   a_scale   device, fp16 bits [M]; receives s_m
 * Errors: APT_ERR_INVALID_ARG for M < 1, K < 1, q outside [1, 8], a NULL
 * input, packed or scale pointer, or a misaligned packed pointer;
 * APT_ERR_UNSUPPORTED for K > 2^30; APT_ERR_HIP on launch failure. */
apt_status_t apt_quantize_pack_activations_fp16(const uint16_t* a_fp16, int M, int K, int q,
                                                void* a_packed, int32_t* a_rowsum,
                                                uint16_t* a_scale, void* stream);

/* Host-only.  Chooses the route and tile shape for (M, N, K, p, q) (Sec. V-B:
 * lookup table, approximate matching): the config apt_search_config recorded
 * for exactly this problem, if any; otherwise the XOR route for M <= 8, and
 * above that a model of the MI355X kernels (rounds of resident tiles per
 * compute unit, measured cycles per chunk pair of each tile shape, stream-K
 * partial traffic; the FP4 route only with FP4 activations, q <= 2; the XOR
 * route when its cost per word pair and p*q beats them on small problems),
 * which stands in for the approximate match.  The choice never changes
 * results.
 * Errors: APT_ERR_INVALID_ARG for sizes < 1, bits outside [1, 8] or out == NULL. */
apt_status_t apt_select_config(int M, int N, int K, int p, int q, apt_config_t* out);

/* Device workspace bytes apt_gemm needs for this problem and config (cfg
 * NULL or route AUTO = the selected one).  The reassembled int8 MFMA route
 * expands the activations once per call into int8 MFMA fragments
 * (ceil(M/32)*32 * K_pad' bytes, K_pad' = K_pad rounded up to a multiple of
 * 256; the FP4 MFMA route with q <= 2 stores half of that: two values per
 * byte) and,
 * for each launch with a stream-K decomposition (grid > 0 and T not a
 * multiple of grid), two int32 BM x BN partial tiles per workgroup and one
 * counter per shared tile, each region rounded up to 256 bytes; the other
 * routes need 0.  Returns 0 for invalid sizes or configs. */
size_t apt_gemm_workspace_bytes(int M, int N, int K, int p, int q, const apt_config_t* cfg);

/* C = A * W^T on packed operands, with the fused recombination of Sec. III-B
 * and the optional scale epilogue.
 *   a_packed  device, packed q-bit activations [M][K] (apt_quantize_pack_activations)
 *   w_packed  device, packed p-bit weights [N][K] (apt_pack_weights)
 *   a_rowsum, w_rowsum  device int32 [M] / [N] from the packers; required by
 *             the MFMA routes, ignored by APT_ROUTE_XOR (may be NULL there)
 *   c_int32   device int32 [M][N] row-major, or NULL
 *   a_scale   device fp16 bits [M], per-token bipolar scale, or NULL
 *   w_scale   device fp16 bits [N], per-channel bipolar scale, or NULL
 *   c_fp16    device fp16 bits [M][N] row-major, or NULL;
 *             c_fp16[m][n] = fp16_rne(float(C) * float(a_scale[m]) * float(w_scale[n]))
 *   cfg       NULL = apt_select_config, else a config to force
 *   workspace, workspace_bytes  device scratch of at least
 *             apt_gemm_workspace_bytes(...) bytes, 16-byte aligned (NULL when 0);
 *             its contents are overwritten; calls that share a workspace must
 *             not overlap in time
 * Errors: APT_ERR_INVALID_ARG for sizes < 1, bits outside [1, 8], NULL or
 * misaligned packed pointers, both outputs NULL, c_fp16 without both scales, a
 * route needing row sums without them, a misaligned workspace, or an invalid
 * cfg; APT_ERR_UNSUPPORTED when K (2^p-1)(2^q-1) >= 2^31, or when an FP4
 * route is forced with p > 2, q > 4 or K_pad (2^p-1)(2^q-1) >= 2^24; APT_ERR_WORKSPACE
 * when the workspace is missing or too small; APT_ERR_HIP on launch failure. */
apt_status_t apt_gemm(int M, int N, int K, int p, int q,
                      const void* a_packed, const void* w_packed,
                      const int32_t* a_rowsum, const int32_t* w_rowsum,
                      int32_t* c_int32,
                      const uint16_t* a_scale, const uint16_t* w_scale, uint16_t* c_fp16,
                      const apt_config_t* cfg,
                      void* workspace, size_t workspace_bytes, void* stream);

/* C = A * W^T as apt_gemm, with an fp16 epilogue for linear quantizers that
 * have a zero-point.  Sec. III-A writes a linear quantizer as X = s * x + z
 * and rewrites it for bipolar values x' = 2x + 1 as X = (s/2) x' + (z - s/2):
 * bipolar scale s' = s/2, bipolar zero z' = z - s/2.  With per-token (s'_a,
 * z'_a) and per-channel (s'_w, z'_w) bipolar parameters, the product of the
 * dequantized operands sum_k (s'_a a'[m][k] + z'_a)(s'_w w'[n][k] + z'_w) is
 *   Y[m][n] = s'_a s'_w C + s'_a z'_w R_a[m] + z'_a (s'_w R_w[n] + K z'_w),
 * with C the int32 product and R the bipolar row sums from the packers.
 *   a_packed, w_packed, cfg, workspace, workspace_bytes, stream  as apt_gemm
 *   a_rowsum, w_rowsum  device int32 [M] / [N] from the packers (required)
 *   a_scale, a_zero     device fp16 bits [M], per-token s'_a and z'_a
 *   w_scale, w_zero     device fp16 bits [N], per-channel s'_w and z'_w
 *   c_fp16    device fp16 bits [M][N] row-major: fp16_rne of Y evaluated in
 *             fp32 as s'_a (s'_w C + z'_w R_a) + z'_a (s'_w R_w + K z'_w)
 *   c_int32   device int32 [M][N] row-major (the integer product C), or NULL
 * Errors: as apt_gemm, and APT_ERR_INVALID_ARG when a row-sum, scale,
 * zero-point or the c_fp16 pointer is NULL. */
apt_status_t apt_gemm_affine(int M, int N, int K, int p, int q,
                             const void* a_packed, const void* w_packed,
                             const int32_t* a_rowsum, const int32_t* w_rowsum,
                             const uint16_t* a_scale, const uint16_t* a_zero,
                             const uint16_t* w_scale, const uint16_t* w_zero,
                             uint16_t* c_fp16, int32_t* c_int32,
                             const apt_config_t* cfg,
                             void* workspace, size_t workspace_bytes, void* stream);

/* Size of the device array apt_gemm_noalloc uses as its workspace (64 MiB). */
#define APT_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

/* apt_gemm without a caller workspace and without any device allocation, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * serving loops, harnesses that forbid hipMalloc).  The workspace is a device
 * array inside the library of APT_NOALLOC_SCRATCH_BYTES bytes; each GPU the
 * library runs on holds its own copy until the process ends (the first call
 * on a device looks up its address).  Every call on one GPU shares that GPU's
 * copy, so calls that overlap in time on one GPU (concurrent streams, or
 * several host threads) race and must be serialised by the caller; calls in
 * stream order are safe (the kernels rewrite or clear what they read).
 * Arguments, results and errors as apt_gemm without workspace and
 * workspace_bytes; the outputs are caller buffers as there.  With cfg NULL or
 * route AUTO the selected config is used, and if its stream-K partial tiles
 * do not fit, the same tiles with one workgroup per tile (the result is the
 * same).  Errors: as apt_gemm, and APT_ERR_WORKSPACE when the resolved
 * config needs more than APT_NOALLOC_SCRATCH_BYTES (activation fragments of
 * about M * K bytes on the MFMA routes, plus stream-K partial tiles of a
 * forced persistent grid); APT_ERR_UNSUPPORTED for a device ordinal of 64 or
 * more; nothing is launched in either case. */
apt_status_t apt_gemm_noalloc(int M, int N, int K, int p, int q,
                              const void* a_packed, const void* w_packed,
                              const int32_t* a_rowsum, const int32_t* w_rowsum,
                              int32_t* c_int32,
                              const uint16_t* a_scale, const uint16_t* w_scale, uint16_t* c_fp16,
                              const apt_config_t* cfg, void* stream);

/* Activation sources of apt_gemm_decode. */
enum {
  APT_ACT_CODES = 1, /* int8 [M][K], signed q-bit codes (as apt_quantize_pack_activations) */
  APT_ACT_FP16 = 2   /* fp16 bits [M][K], quantized per row as apt_quantize_pack_activations_fp16 */
};

/* Largest M apt_gemm_decode takes. */
#define APT_DECODE_MAX_M 8

/* The decode GEMM (one to eight tokens) with the activation side of the
 * conversion fused into it: C = A * W^T on the XOR + popcount route (Sec.
 * III-B), where A is given unpacked and each workgroup converts its tokens'
 * rows to bipolar-INT bit-planes (Sec. III-A conversion, Sec. IV-A steps 1-3;
 * for fp16 input after quantizing the row) into its LDS, so that neither a
 * packer launch nor a packed activation buffer sits between the token and
 * the GEMV.  Results equal those of the packer (apt_quantize_pack_activations
 * for codes, apt_quantize_pack_activations_fp16 for fp16) followed by apt_gemm
 * on the XOR route, bit for bit: the same codes, scales, int32 C and fp16
 * output.
 *   a_src     device, the activations [M][K] row-major in the a_kind format;
 *             fp16 values must be finite (as for the fp16 packer); 2-byte
 *             aligned for fp16 (16-byte alignment and K % 16 == 0 select wider
 *             loads; the result does not depend on it)
 *   a_kind    APT_ACT_CODES or APT_ACT_FP16
 *   w_packed  device, packed p-bit weights [N][K] (apt_pack_weights), 16-byte aligned
 *   c_int32   device int32 [M][N] row-major, or NULL
 *   a_scale   APT_ACT_CODES: device fp16 bits [M], per-token bipolar scale
 *             (required with c_fp16, else may be NULL); APT_ACT_FP16: must be NULL
 *             (the scale is computed from the row)
 *   w_scale   device fp16 bits [N], per-channel bipolar scale (required with c_fp16)
 *   c_fp16    device fp16 bits [M][N] row-major, or NULL; as apt_gemm's epilogue,
 *             with the computed row scale for APT_ACT_FP16
 *   a_scale_out  APT_ACT_FP16: device fp16 bits [M] receiving each row's scale
 *             s_m (as the fp16 packer's a_scale), or NULL; APT_ACT_CODES: must be NULL
 *   cfg       NULL or route AUTO: the library's XOR launch shape; else an XOR
 *             route config (mt, waves_m, waves_n as for apt_gemm)
 * Each workgroup keeps the bit-planes of its activation rows in LDS: with mt
 * = 1 one row, ceil(K / 1024) * 1024 * q / 8 bytes; with mt = 8 eight rows,
 * ceil(K / 1024) * 16 * (8 q + 1) bytes; at most 64 KB.  mt = 0 takes 1 for
 * M = 1, below 1024 row groups of 8 weight rows, and below 2048 row groups
 * for M <= 2 or an fp16 source; else 8 if that fits, else 1.
 * Errors: APT_ERR_INVALID_ARG for M outside [1, APT_DECODE_MAX_M], N or K < 1,
 * bits outside [1, 8], a bad a_kind, a NULL source or weight pointer, a
 * misaligned weight or fp16 source pointer, both outputs NULL, c_fp16 without
 * its scales, a scale pointer the a_kind does not take, or a cfg that is not
 * a valid XOR config; APT_ERR_UNSUPPORTED when K (2^p-1)(2^q-1) >= 2^31 or
 * when the rows' bit-planes do not fit in 64 KB of LDS; APT_ERR_HIP on launch
 * failure. */
apt_status_t apt_gemm_decode(int M, int N, int K, int p, int q,
                             const void* a_src, int a_kind, const void* w_packed,
                             int32_t* c_int32, const uint16_t* a_scale,
                             const uint16_t* w_scale, uint16_t* c_fp16,
                             uint16_t* a_scale_out, const apt_config_t* cfg, void* stream);

/* Device workspace bytes apt_gemm_act needs for this problem, activation
 * kind and config (cfg NULL or route AUTO = the selected one); 0 when the
 * call needs none (the fused XOR form) or for invalid arguments. */
size_t apt_gemm_act_workspace_bytes(int M, int N, int K, int p, int q, int a_kind,
                                    const apt_config_t* cfg);

/* C = A * W^T for any M with the activations given unpacked, as int8 codes
 * or fp16 values (APT_ACT_CODES / APT_ACT_FP16, quantized per row as
 * apt_quantize_pack_activations_fp16 does): the conversion to bipolar-INT
 * (Sec. III-A) runs inside this call, in the form the route needs, and the
 * results equal those of the matching packer followed by apt_gemm with the
 * same config, bit for bit (codes, scales, int32 C and fp16 output).
 *   - XOR route with M <= APT_DECODE_MAX_M whose rows fit in LDS: the rows are
 *     converted to bit-planes inside the GEMV, as apt_gemm_decode does (no
 *     workspace);
 *   - int8 MFMA route: the rows are written straight into the route's int8
 *     MFMA operand fragments, with their row sums (and fp16 scales), by one
 *     kernel (Sec. III-B's plane sum rebuilt before the multiply, as apt_gemm
 *     does from the planes), so no bit-planes are written or read;
 *   - every other route: the packer writes the bit-planes (Sec. IV-A) into the
 *     workspace, then the route runs as in apt_gemm.
 *   a_src     device, [M][K] row-major: int8 codes, or fp16 bits (2-byte
 *             aligned; values must be finite); 16-byte alignment and K % 16 == 0
 *             select wider loads (the result does not depend on it)
 *   w_packed  device, packed p-bit weights [N][K] (apt_pack_weights), 16-byte aligned
 *   w_rowsum  device int32 [N] from apt_pack_weights; required by the MFMA
 *             routes, may be NULL on the XOR and +-1 plane routes
 *   c_int32, w_scale, c_fp16, cfg   as apt_gemm
 *   a_scale   APT_ACT_CODES: per-token bipolar scale (fp16 bits [M]), required
 *             with c_fp16; APT_ACT_FP16: must be NULL
 *   a_scale_out  APT_ACT_FP16: device fp16 bits [M] receiving the row scales,
 *             or NULL; APT_ACT_CODES: must be NULL
 *   workspace, workspace_bytes  device scratch of at least
 *             apt_gemm_act_workspace_bytes(...) bytes, 16-byte aligned (NULL
 *             when 0); overwritten; calls sharing it must not overlap in time
 * Errors: as apt_gemm (a_packed and a_rowsum replaced by a_src), and
 * APT_ERR_INVALID_ARG for a bad a_kind, a misaligned fp16 source or a scale
 * pointer the a_kind does not take; APT_ERR_UNSUPPORTED also for K > 2^30. */
apt_status_t apt_gemm_act(int M, int N, int K, int p, int q,
                          const void* a_src, int a_kind, const void* w_packed,
                          const int32_t* w_rowsum, int32_t* c_int32,
                          const uint16_t* a_scale, const uint16_t* w_scale, uint16_t* c_fp16,
                          uint16_t* a_scale_out, const apt_config_t* cfg,
                          void* workspace, size_t workspace_bytes, void* stream);

/* Device workspace bytes apt_search_config needs for this problem: the most
 * that any config it times needs (apt_gemm_workspace_bytes).  Returns 0 for
 * invalid sizes or bit widths. */
size_t apt_search_workspace_bytes(int M, int N, int K, int p, int q);

/* The best-kernel search module (Sec. V-B): times every configuration the
 * library can run for (M, N, K, p, q) on the caller's operands, records the
 * fastest in the configuration table, so that apt_select_config and apt_gemm
 * with cfg NULL use it for this problem from then on, and returns it.  The
 * candidates are the XOR route, the +-1 plane route (p, q <= 7), every int8
 * tile shape with one workgroup per tile and with one persistent round of
 * workgroups, and the split launches of a main and a tail shape, each of
 * these also with FP4 operands where the FP4 route applies.  Each is
 * run twice to warm up, then timed over 5 back-to-back calls between two HIP
 * events on `stream`.  The call blocks until the timing has finished.  All
 * candidates compute the same result, so it never changes results.
 *   a_packed, w_packed, a_rowsum, w_rowsum  device, as apt_gemm (required)
 *   c_int32   device int32 [M][N]; overwritten by the timed calls
 *   workspace, workspace_bytes  device scratch of at least
 *             apt_search_workspace_bytes(...) bytes, 16-byte aligned (NULL when 0)
 *   best      host; receives the chosen config
 *   best_us   host or NULL; receives its mean time per call in microseconds
 * Errors: APT_ERR_INVALID_ARG for sizes < 1, bits outside [1, 8], a NULL or
 * misaligned operand, row-sum, output or best pointer, or a misaligned
 * workspace; APT_ERR_UNSUPPORTED when K (2^p-1)(2^q-1) >= 2^31 or no
 * candidate can run; APT_ERR_WORKSPACE when the workspace is missing or too
 * small; APT_ERR_HIP when a launch or an event call fails. */
apt_status_t apt_search_config(int M, int N, int K, int p, int q,
                               const void* a_packed, const void* w_packed,
                               const int32_t* a_rowsum, const int32_t* w_rowsum,
                               int32_t* c_int32, void* workspace, size_t workspace_bytes,
                               void* stream, apt_config_t* best, float* best_us);

/* Empties the configuration table that apt_search_config fills. */
void apt_config_table_clear(void);

/* Number of problems in the configuration table. */
int apt_config_table_size(void);

/* The hipError_t code (as an int) of the HIP runtime call that made the most
 * recent call of this thread return APT_ERR_HIP; 0 if none has.  Each launch
 * is checked through its own return status, so an error an unrelated runtime
 * call left behind is never reported as the library's.  Host-only, no
 * arguments, cannot fail. */
int apt_last_hip_error(void);

/* Static, NUL-terminated description of a status code. */
const char* apt_status_string(apt_status_t status);

#ifdef __cplusplus
}
#endif

#endif /* APT_H */
