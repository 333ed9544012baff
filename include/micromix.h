/*
 * micromix.h - C ABI of the MicroMix hot path for AMD Instinct MI355X (gfx950).
 *
 * MicroMix (arXiv 2508.02343) splits the K input channels of a linear layer
 * into three groups that are quantised with Microscaling (MX) formats of
 * different width: MXFP4 (E2M1), MXFP6 (E3M2) and MXFP8 (E4M3), each in
 * blocks of 32 elements that share one E8M0 power-of-two scale (Sec. 2.1,
 * MX quantisation equation; Appendix B, Table "tab:microscaling";
 * Sec. 4.1 "Quantization").  Channels are first gathered by a permutation
 * sigma so that channels of one precision are adjacent (Sec. 3.1,
 * "Reducing quantization error through permutation" and "Offline channel
 * assignment strategy").  The linear layer is then computed as one GEMM that
 * sums all three partitions in fp32 and writes bfloat16 (Sec. 2.1 eq. 1;
 * Sec. 3.2 "GEMM kernel").
 *
 * These calls implement that path, and mm_calibrate prepares it offline:
 *   mm_quantize_act     online fused reorder-and-quantize of activations
 *                       (Sec. 3.2 "Quantization kernel", Fig. "micromix-design" b)
 *   mm_rmsnorm_quantize_act  the same, with the layer's RMSNorm fused in
 *                       front (App. D.2, Fig. "precision-mapping")
 *   mm_quantize_weight  the same transform for weights, run once offline
 *                       with the activation's sigma and split (Sec. 3.2)
 *   mm_gemm             mixed-precision block-scaled GEMM, Y = A W^T
 *                       (Sec. 3.2 "GEMM kernel", Fig. "micromix-design" a)
 *   mm_calibrate        offline choice of sigma and the split from
 *                       calibration activations (Sec. 3.1 "Offline channel
 *                       assignment strategy"; Def. 1; Appendix C.2 "Derivations")
 *
 * Conventions shared by every call
 * --------------------------------
 * - Every data pointer is a DEVICE pointer owned by the caller.  The library
 *   allocates no memory and keeps no device state.  Descriptors are host
 *   structs read during the call only.
 * - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *   Calls only enqueue work; they never synchronise.
 * - Validation happens on the host before anything is enqueued.  On any
 *   error nothing is launched, outputs are untouched, and the status says
 *   why; mm_last_error() returns a message for the calling thread.
 * - No C++ exception crosses this boundary.
 *
 * Quantised tensor layout (mm_mx_tensor)
 * --------------------------------------
 * A quantised operand has `rows` rows of K channels in permuted order
 * X'[:, j] = X[:, sigma[j]].  Channels [0, p4) are E2M1, [p4, p4+p6) are
 * E3M2 and [p4+p6, K) are E4M3.  Each row's blocks of 32 consecutive permuted
 * channels share one scale; a block never straddles two groups.
 *
 * The packed layout is laid out for the GEMM's loads (it plays the role of the
 * tensor-core scale-factor layout the paper's quantisation kernel writes):
 *   R   = rows rounded up to a multiple of 32 (a "row group" is 32 rows);
 *   nbG = pG / 32 blocks of group G, SG = ceil(nbG / 4) "steps" of 4 blocks;
 *   RBG = bytes of one row's step: 64 (E2M1), 96 (E3M2), 128 (E4M3).
 * Codes of group G: SG steps, each R * RBG bytes; inside a step, row group q
 * (rows 32q .. 32q+31) occupies 32 * RBG bytes starting at q * 32 * RBG, and
 * within it, for row r = row % 32 and block j = 0..3 of the step:
 *   E2M1: block j of row r at  j * 512 + r * 16  (16 bytes: element 2i in
 *         the low nibble of byte i, 2i+1 in the high nibble);
 *   E3M2: block j of row r at  j * 768 + r * 24  (24 bytes: a little-endian
 *         bit stream, element i at bits 6i .. 6i+5);
 *   E4M3: bytes 16h .. 16h+15 (h = 0, 1) of block j of row r at
 *         (2j + h) * 512 + r * 16  (one code per byte).
 * So block b of row n of group G starts at byte
 *   (b/4) * R * RBG + (n/32) * 32 * RBG + [offset above with j = b%4, r = n%32].
 * Scales: (S4 + S6 + S8) steps numbered t (E2M1 steps first, then E3M2, then
 * E4M3); byte (t * R + row) * 4 + j is the E8M0 scale (2^(byte-127)) of block
 * j of that step of that row.
 * Padding: blocks past the end of a group inside its last step, and rows
 * rows .. R-1, hold zero codes and scale byte 0; the quantise calls write
 * them and mm_gemm relies on them.
 * Element codes are sign | exponent | mantissa with the OCP MX encodings:
 * E2M1 bias 1, E3M2 bias 3, E4M3 bias 7 (S.1111.111 is NaN and never written);
 * with the alternative formats (mm_formats below) the 6-bit group holds E2M3
 * codes (bias 1) and the 8-bit group E5M2 codes (bias 15; its Inf and NaN
 * codes are never written), in the same byte positions.
 * mm_mx_layout_sizes() gives each buffer's byte count.
 * Requirements: K > 0 and K % 32 == 0; p4, p6, p8 >= 0, each % 32 == 0,
 * p4 + p6 + p8 == K; every buffer of a non-empty group 16-byte aligned and
 * at least the size mm_mx_layout_sizes() reports; a buffer of an empty group
 * (p == 0) may be NULL.
 *
 * Quantisation rule (bit-exact): for a block with largest magnitude amax the
 * scale exponent is e = floor(log2 amax) - emax, with emax the format's top
 * binade exponent (E2M1 2, E3M2 4, E2M3 2, E4M3 8, E5M2 15), clamped to
 * [-127, 127], and
 * e = -127 for an all-zero block.  Each element x is coded as x * 2^-e
 * rounded to the nearest representable value, ties to the even code,
 * saturating at the largest finite value, keeping the sign of x (so -0 and
 * negative values that round to zero give the negative-zero code).
 */
#ifndef MICROMIX_H
#define MICROMIX_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MM_ABI_VERSION 6

typedef enum {
  MM_OK = 0,
  MM_ERR_NULL = 1,   /* a required pointer is NULL                          */
  MM_ERR_SHAPE = 2,  /* rows/K/ld out of range, or a/w disagree in mm_gemm  */
  MM_ERR_SPLIT = 3,  /* p4/p6/p8 not multiples of 32, negative, or sum != K */
  MM_ERR_ALIGN = 4,  /* a pointer or leading dimension is misaligned        */
  MM_ERR_FORMAT = 5, /* unknown element format, or a and w formats differ   */
  MM_ERR_DEVICE = 6, /* the HIP runtime reported an error at launch         */
  MM_ERR_WORKSPACE = 7, /* mm_calibrate: workspace smaller than required    */
  MM_ERR_VALUE = 8      /* a scalar argument out of range (eps)              */
} mm_status;

typedef struct {
  int32_t p4, p6, p8; /* channels per group: MXFP4, MXFP6, MXFP8 */
} mm_split;

/*
 * Element formats of the 6-bit and 8-bit groups (Sec. 4.1 uses E3M2 and
 * E4M3; its ablation, Table "tab:ablation-study-mxfp6-mxfp8", compares E2M3
 * and E5M2).  The zero value of each field is the default, so a
 * zero-initialised descriptor selects E3M2 and E4M3.  Any other value is
 * rejected with MM_ERR_FORMAT.
 */
typedef enum { MM_FP6_E3M2 = 0, MM_FP6_E2M3 = 1 } mm_fp6_format;
typedef enum { MM_FP8_E4M3 = 0, MM_FP8_E5M2 = 1 } mm_fp8_format;

typedef struct {
  int32_t fp6; /* mm_fp6_format of the 6-bit group */
  int32_t fp8; /* mm_fp8_format of the 8-bit group */
} mm_formats;

typedef struct {
  int64_t rows;       /* M for activations, N for weights            */
  int64_t K;          /* channels per row                            */
  mm_split split;     /* group sizes, identical for a and w in GEMM  */
  mm_formats formats; /* element formats, identical for a and w      */
  uint8_t* q4;        /* E2M1 codes (layout above)                    */
  uint8_t* q6;        /* 6-bit codes (E3M2 or E2M3)                   */
  uint8_t* q8;        /* 8-bit codes (E4M3 or E5M2)                   */
  uint8_t* sc;        /* E8M0 scales                                  */
} mm_mx_tensor;

typedef struct {
  int64_t q4, q6, q8, sc; /* bytes of each buffer */
} mm_mx_sizes;

/*
 * Byte counts of the four buffers of a quantised tensor of `rows` rows with
 * this K and split (layout above).  Host-only arithmetic, no device access.
 * Errors: MM_ERR_NULL (out is NULL), MM_ERR_SHAPE, MM_ERR_SPLIT.
 */
mm_status mm_mx_layout_sizes(int64_t rows, int64_t K, mm_split split, mm_mx_sizes* out);

/*
 * Fused reorder-and-quantize of activations (Sec. 3.2 "Quantization kernel";
 * MX rule of Sec. 2.1; groups of Sec. 3.1).
 *   x_bf16  device, bf16 [out->rows, K] row-major, row stride ldx elements
 *           (ldx >= K, ldx % 8 == 0, 16-byte aligned), finite values.
 *   perm    device, int32 [K], a permutation of [0, K) (not checked on the
 *           device: a non-permutation gives unspecified codes but stays in
 *           bounds only if every entry is in [0, K)).
 *   out     host descriptor of device buffers, filled as described above
 *           (including the padding).
 * K may be at most 32768.  Errors: MM_ERR_NULL, MM_ERR_SHAPE, MM_ERR_SPLIT,
 * MM_ERR_ALIGN, MM_ERR_FORMAT, MM_ERR_DEVICE.
 */
mm_status mm_quantize_act(const void* x_bf16, int64_t ldx, const int32_t* perm, const mm_mx_tensor* out,
                          void* stream);

/*
 * RMSNorm fused with the reorder-and-quantize of activations (App. D.2,
 * Fig. "precision-mapping": the reorder-and-quantize runs inside the layer's
 * normalisation, so the normalised bf16 activation never goes to memory).
 * Each row x is replaced by
 *   y_j = bf16( gamma_j * bf16( x_j * r ) ),  r = fp32( 1 / sqrt(mean_j x_j^2 + eps) )
 * (r evaluated in fp64 and rounded once to fp32; both products in fp32,
 * each rounded to nearest even), and y is quantised exactly as
 * mm_quantize_act would quantise it.
 *   gamma_bf16  device, bf16 [K] in the original channel order (16-byte
 *               aligned, finite).
 *   eps         finite and > 0 (MM_ERR_VALUE otherwise).
 * The other arguments, the layout and the errors are those of
 * mm_quantize_act (plus MM_ERR_VALUE; MM_ERR_NULL for a NULL gamma).
 */
mm_status mm_rmsnorm_quantize_act(const void* x_bf16, int64_t ldx, const void* gamma_bf16, float eps,
                                  const int32_t* perm, const mm_mx_tensor* out, void* stream);

/*
 * Offline reorder-and-quantize of a weight W [N, K] with the sigma and split
 * of the activation it will multiply (Sec. 3.2: weights are permuted to match
 * the reordered activations, then quantised the same way, once).  Same
 * arguments, layout and errors as mm_quantize_act with rows = N.
 */
mm_status mm_quantize_weight(const void* w_bf16, int64_t ldw, const int32_t* perm, const mm_mx_tensor* out,
                             void* stream);

/*
 * Mixed-precision GEMM (Sec. 2.1 eq. 1; Sec. 3.2 "GEMM kernel"):
 *   Y[m, n] = bf16( sum over the E2M1, E3M2 and E4M3 groups of
 *                   sum_k (2^ea[m,blk] a[m,k]) (2^ew[n,blk] w[n,k]) )
 * with one fp32 accumulator across all three groups and one round-to-
 * nearest-even conversion to bf16 at the end.
 *   a       activation descriptor, rows = M.
 *   w       weight descriptor, rows = N; same K and split as a.
 *   y_bf16  device, bf16 [M, N] row-major, row stride ldy elements
 *           (ldy >= N, ldy % 8 == 0, 16-byte aligned).
 * Errors: MM_ERR_NULL, MM_ERR_SHAPE (K or split differ, ldy below N),
 * MM_ERR_SPLIT, MM_ERR_ALIGN, MM_ERR_FORMAT (formats differ or unknown),
 * MM_ERR_DEVICE.
 */
mm_status mm_gemm(const mm_mx_tensor* a, const mm_mx_tensor* w, void* y_bf16, int64_t ldy, void* stream);

/*
 * Device workspace mm_calibrate needs for `rows` calibration rows of K
 * channels: a 2048-byte block, then (chunks + 1) * K doubles and
 * ceil(K / 256) * K int32 words, where the number of row chunks (1 .. 128)
 * depends on rows and K only.  Host-only arithmetic.  Errors: MM_ERR_NULL (bytes is NULL),
 * MM_ERR_SHAPE.
 */
mm_status mm_calibrate_workspace_size(int64_t rows, int64_t K, int64_t* bytes);

/*
 * Offline channel assignment (Sec. 3.1 "Offline channel assignment strategy";
 * Def. 1, eq. quantization-threshold; Appendix C.2 "Derivations").  From calibration
 * activations X [rows, K]:
 *   M_j    = (1/rows) sum_i |X[i, j]|, summed in fp64 (exact per term) in
 *            a fixed order for a given (rows, K), so results repeat;
 *   sigma  = the channels sorted by ascending M, equal means in increasing
 *            channel order (sigma[i] is the channel at sorted position i);
 *   T(n)   = 2^b * 2^(n-1) / q_max * max|X| / 254, max over the whole of X:
 *            T(4) with E2M1 (b 1, q_max 6), T(6) with the 6-bit format of
 *            `formats` (E3M2: b 3, q_max 28; E2M3: b 1, q_max 7.5);
 *   n4     = #{j : M_j <= T(4)}, n6 = #{j : T(4) < M_j <= T(6)};
 *   split  = (p4, p6, p8) with p4 = 32 floor(n4 / 32),
 *            p4 + p6 = 32 floor((n4 + n6) / 32), p8 = K - p4 - p6.
 * Since the groups use the same statistic sigma sorts by, G4 = sigma[0, p4),
 * G6 = sigma[p4, p4+p6), G8 = the rest, ready for mm_quantize_act.
 *   x_bf16     device, bf16 [rows, K] row-major, row stride ldx elements
 *              (ldx >= K, ldx % 8 == 0, 16-byte aligned).
 *   formats    fp6 picks T(6)'s constants; fp8 is only validated.
 *   workspace  device, caller-owned, 16-byte aligned, at least
 *              mm_calibrate_workspace_size() bytes; its contents on entry are
 *              ignored and on exit unspecified.  Calls that overlap in time
 *              must not share it.
 *   perm_out   device, int32 [K], 16-byte aligned: sigma.
 *   split_out  device, int32 [3]: (p4, p6, p8); (-1, -1, -1) when X holds an
 *              Inf or NaN, and then perm_out is the identity.
 * Like every call it only enqueues work on `stream` (four launches); read
 * split_out after the stream has reached it.  rows >= 1, K a positive
 * multiple of 32, at most 32768.  Errors: MM_ERR_NULL, MM_ERR_SHAPE,
 * MM_ERR_ALIGN, MM_ERR_FORMAT, MM_ERR_WORKSPACE, MM_ERR_DEVICE.
 */
mm_status mm_calibrate(const void* x_bf16, int64_t rows, int64_t K, int64_t ldx, mm_formats formats,
                       void* workspace, int64_t workspace_bytes, int32_t* perm_out, int32_t* split_out,
                       void* stream);

/*
 * mm_calibrate without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation.  It computes exactly what mm_calibrate
 * computes (same kernels, same results bit for bit), but its workspace is a
 * library-owned static device array of 16 MiB (each GPU the library runs on
 * holds one until the process ends).  The call allocates nothing: the
 * array's device address is looked up once per device, on the first call
 * made with that device current, and cached.
 *   Limit: the plan for (rows, K) must fit the 16 MiB; every rows count fits
 *   for K <= 31488.  Larger plans fail with MM_ERR_WORKSPACE before any work
 *   is enqueued (mm_calibrate with a caller workspace takes them).
 *   Sharing: every call on a GPU uses that GPU's one array.  Calls that
 *   overlap in time on one GPU (other streams, other host threads) race on
 *   it and give undefined results; calls ordered on one stream are safe.
 *   No kernel reads the array before writing it, so what a previous call
 *   left there does not matter.
 * Arguments and errors as mm_calibrate's (no workspace, no workspace_bytes);
 * MM_ERR_DEVICE also when the array's address cannot be looked up.
 */
mm_status mm_calibrate_no_alloc(const void* x_bf16, int64_t rows, int64_t K, int64_t ldx, mm_formats formats,
                                int32_t* perm_out, int32_t* split_out, void* stream);

/* Static English name of a status code. */
const char* mm_status_str(mm_status s);

/* Message of the last error on the calling thread ("" if none). */
const char* mm_last_error(void);

/* MM_ABI_VERSION of the loaded library. */
int mm_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MICROMIX_H */
