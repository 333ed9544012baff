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
 * Three calls implement that path:
 *   mm_quantize_act     online fused reorder-and-quantize of activations
 *                       (Sec. 3.2 "Quantization kernel", Fig. "micromix-design" b)
 *   mm_quantize_weight  the same transform for weights, run once offline
 *                       with the activation's sigma and split (Sec. 3.2)
 *   mm_gemm             mixed-precision block-scaled GEMM, Y = A W^T
 *                       (Sec. 3.2 "GEMM kernel", Fig. "micromix-design" a)
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
 *   q4: row r holds p4/2 bytes at q4 + r*ld4; element 2i in the low nibble
 *       of byte i, element 2i+1 in the high nibble.
 *   q6: row r holds 3*p6/4 bytes at q6 + r*ld6; each block of 32 codes is a
 *       24-byte little-endian bit stream, code i at bits 6i..6i+5.  When
 *       p6/32 is odd, the 8 bytes after the last block (up to the next
 *       multiple of 16) are zero: the quantise calls write them, and
 *       mm_gemm requires them.
 *   q8: row r holds p8 bytes at q8 + r*ld8, one code per byte.
 *   sc: row r holds K/32 E8M0 bytes (2^(byte-127)) at sc + r*ldsc, in
 *       permuted block order (E2M1 blocks first, then E3M2, then E4M3).
 * Element codes are sign | exponent | mantissa with the OCP MX encodings:
 * E2M1 bias 1, E3M2 bias 3, E4M3 bias 7 (S.1111.111 is NaN and never written).
 * Requirements: K > 0 and K % 32 == 0; p4, p6, p8 >= 0, each % 32 == 0,
 * p4 + p6 + p8 == K; every non-empty buffer pointer 16-byte aligned; each
 * ld* a multiple of 16 and >= the row's byte count rounded up to 16.  A
 * buffer of an empty group (p == 0) may be NULL and its ld is ignored.
 *
 * Quantisation rule (bit-exact): for a block with largest magnitude amax the
 * scale exponent is e = floor(log2 amax) - emax, with emax the format's top
 * binade exponent (E2M1 2, E3M2 4, E4M3 8), clamped to [-127, 127], and
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

#define MM_ABI_VERSION 1

typedef enum {
  MM_OK = 0,
  MM_ERR_NULL = 1,   /* a required pointer is NULL                          */
  MM_ERR_SHAPE = 2,  /* rows/K/ld out of range, or a/w disagree in mm_gemm  */
  MM_ERR_SPLIT = 3,  /* p4/p6/p8 not multiples of 32, negative, or sum != K */
  MM_ERR_ALIGN = 4,  /* a pointer or leading dimension is misaligned        */
  MM_ERR_FORMAT = 5, /* reserved for element-format selection               */
  MM_ERR_DEVICE = 6  /* the HIP runtime reported an error at launch         */
} mm_status;

typedef struct {
  int32_t p4, p6, p8; /* channels per group: MXFP4, MXFP6, MXFP8 */
} mm_split;

typedef struct {
  int64_t rows;   /* M for activations, N for weights            */
  int64_t K;      /* channels per row                            */
  mm_split split; /* group sizes, identical for a and w in GEMM  */
  uint8_t* q4;
  int64_t ld4; /* bytes between rows of q4 */
  uint8_t* q6;
  int64_t ld6; /* bytes between rows of q6 */
  uint8_t* q8;
  int64_t ld8; /* bytes between rows of q8 */
  uint8_t* sc;
  int64_t ldsc; /* bytes between rows of sc */
} mm_mx_tensor;

/*
 * Fused reorder-and-quantize of activations (Sec. 3.2 "Quantization kernel";
 * MX rule of Sec. 2.1; groups of Sec. 3.1).
 *   x_bf16  device, bf16 [out->rows, K] row-major, row stride ldx elements
 *           (ldx >= K, ldx % 8 == 0, 16-byte aligned), finite values.
 *   perm    device, int32 [K], a permutation of [0, K) (not checked on the
 *           device: a non-permutation gives unspecified codes but stays in
 *           bounds only if every entry is in [0, K)).
 *   out     host descriptor of device buffers, filled as described above.
 * K may be at most 32768.  Errors: MM_ERR_NULL, MM_ERR_SHAPE, MM_ERR_SPLIT,
 * MM_ERR_ALIGN, MM_ERR_DEVICE.
 */
mm_status mm_quantize_act(const void* x_bf16, int64_t ldx, const int32_t* perm, const mm_mx_tensor* out,
                          void* stream);

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
 * Errors: MM_ERR_NULL, MM_ERR_SHAPE (K or split differ, ld too small),
 * MM_ERR_SPLIT, MM_ERR_ALIGN, MM_ERR_DEVICE.
 */
mm_status mm_gemm(const mm_mx_tensor* a, const mm_mx_tensor* w, void* y_bf16, int64_t ldy, void* stream);

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
