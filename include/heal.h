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
 *     depend on which load path ran.
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

/*
 * heal_split_f32 -- the operand decomposition on its own (Section 4, GEMM
 * paragraph: the FP32 input is decomposed into a 16-bit head and residual).
 *   x   : n FP32 values (device, read-only).
 *   hi  : n bf16 bit patterns, hi[i] = RNE_bf16(x[i]) (device, written).
 *   lo  : n bf16 bit patterns, lo[i] = RNE_bf16(x[i] - hi[i]) evaluated in
 *         IEEE arithmetic (device, written).
 *   n   : number of elements, n >= 0 (n == 0 is a no-op).
 * The subtraction x - hi is exact, so |x - hi - lo| <= 2^-17 |x| for every
 * finite x that does not round to infinity.  hi and lo must not overlap x or
 * each other.  Non-finite inputs follow IEEE arithmetic: x = +/-inf gives
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
    HEAL_INSTANCE_LARGE = 1,   /* 256 x 256 output tiles, compute-bound shapes */
    HEAL_INSTANCE_MEDIUM = 2,  /* 128 x 128 output tiles */
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

#ifdef __cplusplus
}
#endif

#endif /* HEAL_H */
