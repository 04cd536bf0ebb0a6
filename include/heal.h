/*
 * heal.h -- C ABI of libheal.so: the bf16x3 algebraically compensated GEMM
 * for AMD Instinct MI355X (gfx950).
 *
 * The method (HEAL, Section 4 "Hybrid Error ALleviation", paragraph on GEMM
 * truncation, and its displayed expansion of GEMM(h, W^T) into 16-bit
 * products summed into an FP32 output) keeps a GEMM on 16-bit matrix units
 * while recovering the significand bits a single 16-bit cast would lose.
 * Here both FP32 operands are split into bfloat16 pairs
 *     hi = RNE_bf16(x),  lo = RNE_bf16(x - hi)
 * and the product is
 *     C = hiA*hiB + hiA*loB + loA*hiB
 * accumulated in FP32 by bf16 MFMA instructions and written as FP32 (the
 * output is never rounded to 16 bits: Appendix "HEAL Implementation", HEAL-Base
 * and HEAL-Full keep GEMM outputs in FP32).
 *
 * Reduction order.  For every output element the sum runs over K in 32-deep
 * chunks, k ascending, each chunk adding its three products into one FP32
 * accumulator in the order hiA*hiB, hiA*loB, loA*hiB; the K tail is padded
 * with zeros.  No entry point splits K across workgroups or uses atomics, and
 * every kernel instance follows this order, so results are bitwise identical
 * run to run, for every M (a row's bits do not depend on the other rows), for
 * every N, and between the plain and batched entry points.
 *
 * Conventions for every entry point:
 *   - matrices are row-major FP32 with leading dimensions in ELEMENTS:
 *     A[i*lda + k], B[k*ldb + j] (or B[j*ldb + k] when transposed), C[i*ldc + j];
 *   - all pointers are DEVICE pointers owned by the caller; the library never
 *     allocates, frees or keeps device memory and holds no state beyond a
 *     per-device architecture check, so calls are thread-safe;
 *   - work is enqueued asynchronously on `stream` (0 = the null stream); the
 *     result is visible after the caller synchronises that stream;
 *   - C is write-only (beta = 0): its previous contents never matter; C must
 *     not overlap A or B (A and B may alias each other);
 *   - any 4-byte-aligned pointer and any leading dimension are accepted; the
 *     widest loads are used when alignment allows, and the result bits never
 *     depend on which load path ran;
 *   - a product whose output holds more than 2^21 blocks of 16 x 16 elements
 *     (over all its batch entries) is enqueued as several kernel launches,
 *     each on a range of batch entries, rows and columns, because a dispatch
 *     counts its work-items in 32 bits; the bits are those of one launch.
 * Errors: arguments are validated before any HIP call, so an invalid call
 * returns HEAL_ERR_INVALID_VALUE without touching the device.  The library
 * never aborts and never prints.
 */
#ifndef HEAL_H
#define HEAL_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum heal_status_t {
    HEAL_OK = 0,
    HEAL_ERR_INVALID_VALUE = 1,      /* bad size, leading dimension, pointer or flag */
    HEAL_ERR_UNSUPPORTED_DEVICE = 2, /* the current device is not gfx950 */
    HEAL_ERR_LAUNCH = 3              /* a HIP call or kernel launch failed */
} heal_status_t;

/* Human-readable name of a status code (a static string; never NULL). */
const char *heal_status_string(heal_status_t status);

/* Library version as 10000*major + 100*minor + patch. */
int heal_version(void);

/* Identity of the sources this library was built from: 16 hex digits of a
 * SHA-256 over the kernel sources, this header and the compiler flags (a
 * static string; "unknown" if the build did not supply it).  A caller can
 * compare it with the same hash of the sources it expects, to refuse a stale
 * binary. */
const char *heal_build_id(void);

/*
 * heal_split_f32 -- the operand decomposition on its own (Section 4, GEMM
 * paragraph: the FP32 input is decomposed into a 16-bit head and residual).
 *   x   : n FP32 values (device, read-only).
 *   hi  : n bf16 bit patterns, hi[i] = RNE_bf16(x[i]) (device, written).
 *   lo  : n bf16 bit patterns, lo[i] = RNE_bf16(x[i] - hi[i]) evaluated in
 *         IEEE arithmetic (device, written).
 *   n   : number of elements, n >= 0 (n == 0 is a no-op).
 * The subtraction x - hi is exact, so |x - hi - lo| <= 2^-17 |x| for every
 * finite x with 2^-117 <= |x| that does not round to infinity; below 2^-117
 * lo can fall into bf16's subnormal range (step 2^-133) and the error is at
 * most 2^-134 in absolute terms.  hi and lo must not overlap x or each
 * other.  Non-finite inputs follow IEEE arithmetic: x = +/-inf gives
 * hi = x and lo = NaN; a finite x that rounds to infinity gives lo = -/+inf;
 * x = NaN gives NaN for both (payloads unspecified).  Any output of the GEMM
 * that such an element reaches is therefore NaN.
 */
heal_status_t heal_split_f32(const float *x, uint16_t *hi, uint16_t *lo, int64_t n,
                             hipStream_t stream);

/*
 * heal_gemm_f32 -- C = A * B with the compensated bf16x3 product (Section 4,
 * displayed GEMM expansion; FP32 accumulation and output).
 *   M, N, K : sizes, each >= 0.  M == 0 or N == 0 is a no-op; K == 0 writes +0.
 *   A       : M x K, row stride lda >= max(K, 1).
 *   B       : K x N, row stride ldb >= max(N, 1).
 *   C       : M x N, row stride ldc >= max(N, 1); written, never read.
 */
heal_status_t heal_gemm_f32(int64_t M, int64_t N, int64_t K,
                            const float *A, const float *B, float *C,
                            int64_t lda, int64_t ldb, int64_t ldc, hipStream_t stream);

/*
 * heal_gemm_f32_strided_batched -- batch independent products
 *     C_b = alpha * (A_b * op(B_b)),  b = 0 .. batch-1,
 * with A_b = A + b*strideA, B_b = B + b*strideB, C_b = C + b*strideC.
 *   trans_b = 0 : op(B) = B, B_b is K x N with row stride ldb >= max(N, 1);
 *   trans_b = 1 : op(B) = B^T, B_b is stored N x K (an nn.Linear weight, or
 *                 the keys of an attention score product) with row stride
 *                 ldb >= max(K, 1).
 *   alpha   : FP32 scale applied once to the FP32 accumulator in the epilogue
 *             (the attention 1/sqrt(d) scale), never folded into the inputs.
 *   strides : in elements, >= 0 (0 reuses the same matrix for every entry).
 *   batch   : >= 0.
 * With alpha == 1, trans_b == 0 and batch == 1 the result is bitwise equal to
 * heal_gemm_f32; with trans_b == 1 it is bitwise equal to trans_b == 0 on the
 * explicitly transposed B.
 */
heal_status_t heal_gemm_f32_strided_batched(int64_t M, int64_t N, int64_t K, float alpha,
                                            const float *A, int64_t lda, int64_t strideA,
                                            const float *B, int64_t ldb, int64_t strideB,
                                            int trans_b,
                                            float *C, int64_t ldc, int64_t strideC,
                                            int64_t batch, hipStream_t stream);

/*
 * Kernel instances.  The instance is normally chosen from (M, N) alone.
 * heal_gemm_f32_instance forces one, for tests of cross-instance bitwise
 * equality and for tuning; every instance computes the same bits.
 *   instance : one of heal_instance_t; HEAL_INSTANCE_AUTO chooses as usual.
 * Other arguments as heal_gemm_f32_strided_batched.
 */
typedef enum heal_instance_t {
    HEAL_INSTANCE_AUTO = 0,
    HEAL_INSTANCE_LARGE = 1,   /* 256 x 256 output tiles (the FP16 and pre-split
                                  products take 256 x 224 where that needs fewer
                                  rounds of workgroups; INT16 scores 128 x 256),
                                  compute-bound shapes */
    HEAL_INSTANCE_MEDIUM = 2,  /* 128 x 128 output tiles.  On this and the large
                                  instance, products with B stored N x K and
                                  K <= 128 (attention scores: bf16x3 with
                                  trans_b = 1, and the INT16 scores) whose rows
                                  are 16-byte aligned run a panel kernel instead:
                                  a 256-row (bf16x3) or 128-row (INT16) panel of
                                  A stays in LDS while the workgroup walks the
                                  columns of C (at least one panel of rows) */
    HEAL_INSTANCE_SKINNY = 3,  /* M <= 64: decode and lm_head shapes, B streamed */
    HEAL_INSTANCE_COUNT = 4
} heal_instance_t;

heal_status_t heal_gemm_f32_instance(int instance, int64_t M, int64_t N, int64_t K, float alpha,
                                     const float *A, int64_t lda, int64_t strideA,
                                     const float *B, int64_t ldb, int64_t strideB,
                                     int trans_b,
                                     float *C, int64_t ldc, int64_t strideC,
                                     int64_t batch, hipStream_t stream);

/* The instance heal_gemm_f32 would choose for an M x N output (no HIP call). */
int heal_gemm_select_instance(int64_t M, int64_t N);

/* ==========================================================================
 * FP16 forms of the method (HEAL-Base and HEAL-Full), the pre-split B
 * operand, and the INT16 Q/K score product (HEAL+).
 *
 * Packed operands.  A weight or B operand used many times is converted once
 * into a packed layout in MFMA fragment order: for each block of 16 columns
 * n (jb = n / 16) and 32-deep chunk of k (kc = k / 32), each plane p holds
 * 512 16-bit values at
 *     packed[((jb * KC + kc) * P + p) * 512 + lane * 8 + t],
 *     lane = (n % 16) + 16 * ((k % 32) / 8),  t = k % 8,  KC = ceil(K / 32),
 * positions beyond K or N holding +0.  heal_packed_size gives the number of
 * uint16 values (ceil(N/16) * KC * P * 512); the buffer must be 16-byte
 * aligned.  K is limited to 2^20 for packed operands.
 * ========================================================================== */

/*
 * heal_split_f16 -- the HEAL-Full activation pair on its own (Section 4, GEMM
 * paragraph: an FP32 activation h becomes h_hi + h_lo / 2^10 in FP16).
 *   hi[i] = RNE_f16(x[i]),  lo[i] = RNE_f16((x[i] - hi[i]) * 2^10),
 * as binary16 bit patterns, x - hi and the 2^10 shift exact in FP32.  For
 * finite |x| < 65520, |x - hi - lo / 2^10| <= 2^-22 |x| + 2^-35.  |x| >= 65520
 * gives hi = +/-inf and lo = -/+inf; x = +/-inf gives lo = NaN; NaN gives NaN.
 * Arguments as heal_split_f32.
 */
heal_status_t heal_split_f16(const float *x, uint16_t *hi, uint16_t *lo, int64_t n,
                             hipStream_t stream);

/* Number of uint16 values of a packed K x N operand with `planes` planes (1 or
 * 2), or -1 for invalid sizes (no HIP call). */
int64_t heal_packed_size(int64_t K, int64_t N, int planes);

/*
 * heal_maxabs_f32 -- max|x| over a rows x cols row-major FP32 matrix (row
 * stride ld >= max(cols, 1)), written as one float to *maxabs (device).  An
 * empty matrix gives +0.  A NaN element makes the result a NaN pattern.
 */
heal_status_t heal_maxabs_f32(const float *x, int64_t rows, int64_t cols, int64_t ld,
                              float *maxabs, hipStream_t stream);

/*
 * heal_f16_weight_exponent -- the per-matrix power-of-two weight scale
 * (Appendix "HEAL Implementation", HEAL-Base: weights are scaled by a power of
 * two before the FP16 GEMM and the output is scaled back).  *e (host) becomes
 * the largest integer with maxabs * 2^e <= 65504, so the scaled weights use
 * the top of the FP16 range and none overflows; maxabs == 0 gives e = 0.
 * maxabs is a host value (for example read back from heal_maxabs_f32); it must
 * be finite and >= 0.  No HIP call.
 */
heal_status_t heal_f16_weight_exponent(float maxabs, int32_t *e);

/*
 * heal_pack_f16_weight -- W16 = packed RNE_f16(W * 2^e), one plane, for the
 * FP16 GEMMs.  W is the FP32 weight of a linear layer, N x K row-major (row
 * stride ldw >= max(K, 1)), so the GEMM computes A * W^T.  |e| <= 300.  W16
 * holds heal_packed_size(K, N, 1) values.
 */
heal_status_t heal_pack_f16_weight(const float *W, int64_t N, int64_t K, int64_t ldw, int32_t e,
                                   uint16_t *W16, hipStream_t stream);

/*
 * heal_gemm_f16w -- FP16 GEMM with FP32 activations and FP32 output:
 *   products == 1 (HEAL-Base):  C = 2^-e * sum_k f16(a) w16
 *   products == 2 (HEAL-Full, Section 4 two-product expansion
 *       GEMM(h_hi, W) + GEMM(h_lo / 2^10, W)):
 *       C = 2^-e * sum_k (h_hi w16 + h_lo f16(w16 2^-10)),
 *       with (h_hi, h_lo) as heal_split_f16.  Both products go into ONE FP32
 *       accumulator, per 32-deep chunk the head product and then the
 *       residual product, and the residual's 2^-10 is applied to the FP16
 *       weight fragment.  w16 2^-10 is exact for |w16| >= 2^-4, that is for
 *       every weight above 2^-20 of the largest (the scaled weights reach
 *       2^15); a smaller weight's w16 2^-10 is rounded to FP16's subnormal
 *       step 2^-24, which moves its residual term by at most
 *       2^-25 |h_lo| <= 2^-26 |h| (before the 2^-e scale).
 *   A   : M x K FP32, row stride lda >= max(K, 1);
 *   W16 : packed FP16 weight from heal_pack_f16_weight (same N, K, e);
 *   C   : M x N FP32, row stride ldc >= max(N, 1); written, never read.
 * Reduction order: K in 32-deep chunks ascending, one FP16 MFMA per chunk and
 * product, so results are bitwise identical run to run and for every M.
 * FP16 overflow of an activation (|a| >= 65520) gives an infinite head and a
 * non-finite output, as the FP16 format implies.
 */
heal_status_t heal_gemm_f16w(int products, int64_t M, int64_t N, int64_t K, const float *A,
                             int64_t lda, const uint16_t *W16, int32_t e, float *C, int64_t ldc,
                             hipStream_t stream);
heal_status_t heal_gemm_f16w_instance(int instance, int products, int64_t M, int64_t N,
                                      int64_t K, const float *A, int64_t lda,
                                      const uint16_t *W16, int32_t e, float *C, int64_t ldc,
                                      hipStream_t stream);

/*
 * heal_presplit_b -- the B operand of heal_gemm_f32 split once (as
 * heal_split_f32) and packed with two planes (hi, lo).  B is K x N with row
 * stride ldb >= max(N, 1) (trans_b = 0), or N x K with ldb >= max(K, 1)
 * (trans_b = 1, a linear layer's weight).  Bp holds heal_packed_size(K, N, 2)
 * values: the same 4 bytes per element as the FP32 operand.
 *
 * heal_gemm_f32_presplit -- C = A * B from the pre-split operand: the same
 * bf16 MFMAs in the same order as heal_gemm_f32, so C is bitwise equal to
 * heal_gemm_f32(A, B) (and to the strided-batched form with trans_b = 1 on the
 * transposed storage); no B element is split on this path.
 */
heal_status_t heal_presplit_b(const float *B, int64_t K, int64_t N, int64_t ldb, int trans_b,
                              uint16_t *Bp, hipStream_t stream);
heal_status_t heal_gemm_f32_presplit(int64_t M, int64_t N, int64_t K, const float *A, int64_t lda,
                                     const uint16_t *Bp, float *C, int64_t ldc,
                                     hipStream_t stream);
heal_status_t heal_gemm_f32_presplit_instance(int instance, int64_t M, int64_t N, int64_t K,
                                              const float *A, int64_t lda, const uint16_t *Bp,
                                              float *C, int64_t ldc, hipStream_t stream);

/*
 * heal_quantize_i16 -- INT16 storage of a tensor (Section 4, Q/K/V
 * paragraph): q[i] = Round(32767 x[i] / m), m = max|x|, where Round takes the
 * real quotient to the nearest integer, ties to even.  The decision is exact
 * for every finite input and every m > 0 however small (it is taken on the
 * correctly rounded FP64 quotient of the exact product 32767 x, which cannot
 * cross a half-integer it does not equal); every code lies in
 * [-32767, 32767] and the extreme element gets +/-32767.  m is written to
 * *maxabs (device) and is the tensor's dequantisation scale
 * (x ~ q * m / 32767).  An all-zero tensor gives m = 0 and zero codes.  x
 * must be finite.  Two kernels are enqueued (the maximum, then the codes);
 * no host synchronisation.
 */
heal_status_t heal_quantize_i16(const float *x, int64_t n, int16_t *q, float *maxabs,
                                hipStream_t stream);

/*
 * heal_scores_i16 -- attention scores from INT16 Q and K with the dual-FP16
 * expansion (Section 4, displayed attention expansion):
 *   S_b = f * (Q_hi + Q_lo/2^10)(K_hi + K_lo/2^10)^T,
 *   f = alpha * (maxQ / 32767) * (maxK / 32767), the dequantisation of both
 *       codes, evaluated in FP64 and rounded once to FP32 (a factor below
 *       2^-126 lands in FP32's subnormal range and loses relative precision),
 * where each code q unpacks exactly into hi = RNE_f16(q) and
 * lo/2^10 = q - hi; all four products are accumulated in FP32 (per 32-deep
 * chunk: hi*hi, hi*lo, lo*hi, lo*lo), so the sum is the integer dot product
 * of the codes up to FP32 accumulation.
 *   Q_b  = Q + b*strideQ : M x K INT16, row stride ldq >= max(K, 1);
 *   K_b  = Kt + b*strideK: N x K INT16 (keys, one row per position), ldk >= max(K, 1);
 *   maxQ, maxK : device floats, the maxima written by heal_quantize_i16;
 *   S_b  = S + b*strideS : M x N FP32, row stride lds >= max(N, 1).
 */
heal_status_t heal_scores_i16(int64_t M, int64_t N, int64_t K, const int16_t *Q, int64_t ldq,
                              int64_t strideQ, const float *maxQ, const int16_t *Kt, int64_t ldk,
                              int64_t strideK, const float *maxK, float alpha, float *S,
                              int64_t lds, int64_t strideS, int64_t batch, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* HEAL_H */
