// Internal interface between the C-ABI layer (heal_api.cpp) and the kernels.
#pragma once

#include <stdint.h>
#include <hip/hip_runtime.h>

namespace heal {

// One strided-batched product C_b = alpha * A_b * op(B_b); sizes and strides
// in elements, all validated by the caller.
struct GemmArgs {
    int64_t M, N, K;
    const float *A;
    int64_t lda, strideA;
    const float *B;
    int64_t ldb, strideB;
    float *C;
    int64_t ldc, strideC;
    int64_t batch;
    float alpha;
    int vecA;  // A rows can be read with 16-byte loads (A 16B-aligned, lda % 4 == 0)
    int vecB;  // likewise for B
    int vecC;  // C rows can be written with 16-byte stores
};

// Instance ids follow heal_instance_t in heal.h.
hipError_t launch_gemm(int instance, const GemmArgs &args, bool trans_b, bool use_alpha,
                       hipStream_t stream);

// The dedicated large-tile kernel (heal_gemm_large.hip): 256 x 256 tiles,
// 16-byte operand rows.  large_kernel_applies tells whether it can run a call.
bool large_kernel_applies(const GemmArgs &args, bool trans_b);
hipError_t launch_gemm_large(const GemmArgs &args, bool trans_b, bool use_alpha,
                             hipStream_t stream);

// The skinny kernel (heal_gemm_skinny.hip): M <= 64, 16-byte operand rows.
// skinny_strip_width: the column-strip width (16, 32, 64, 128 or 256) that
// an M x N output with M <= 64 takes, shared by every skinny product.
int skinny_strip_width(int64_t N, int64_t M);
bool skinny_kernel_applies(const GemmArgs &args, bool trans_b);
hipError_t launch_gemm_skinny(const GemmArgs &args, bool trans_b, bool use_alpha,
                              hipStream_t stream);

// The short-K panel kernel (heal_gemm_panel.hip): B stored N x K, K <= 128,
// 16-byte rows, at least one panel of rows (256 for bf16x3, 128 for the
// scores); a panel of A stays in LDS while the workgroup walks the columns
// of C (attention scores).  HEAL_PANEL 0
// keeps those products on the tiled kernels.
#ifndef HEAL_PANEL
#define HEAL_PANEL 1
#endif
bool panel_kernel_applies(const GemmArgs &args, bool trans_b);
hipError_t launch_gemm_panel(const GemmArgs &args, bool use_alpha, hipStream_t stream);

hipError_t launch_split(const float *x, uint16_t *hi, uint16_t *lo, int64_t n, hipStream_t stream);

// ---- FP16 / INT16 forms and the pre-split operand (heal_ops.hip, heal_gemm_op.hip) ----

// The products of heal_gemm_op.hip.
enum OpKind : int {
    OP_BASE = 0,      // HEAL-Base: f16(A) * W16, A FP32, W16 packed FP16
    OP_FULL = 1,      // HEAL-Full: (A_hi * W16) + 2^-10 (A_lo * W16)
    OP_SCORES = 2,    // HEAL+ scores: dual-FP16 of INT16 Q and K, four products
    OP_PRESPLIT = 3,  // bf16x3 with B pre-split and packed
};

// One strided-batched product of heal_gemm_op.hip; sizes in elements.
struct OpArgs {
    int64_t M, N, K;
    const void *A;  // FP32 M x K (BASE, FULL, PRESPLIT) or INT16 M x K (SCORES)
    int64_t lda, strideA;
    const void *B;  // packed uint16 (BASE, FULL, PRESPLIT) or INT16 N x K rows (SCORES)
    int64_t ldb, strideB;
    float *C;
    int64_t ldc, strideC;
    int64_t batch;
    int e;                      // BASE, FULL: C is scaled by 2^-e
    const float *maxA, *maxB;   // SCORES: max|Q|, max|K| (device)
    float alpha;                // SCORES
    int vecA, vecB, vecC;       // 16-byte rows (pointer, leading dimension, batch stride)
};

// The INT16 scores on the short-K panel kernel (heal_gemm_panel.hip).
bool scores_panel_applies(const OpArgs &args);
hipError_t launch_scores_panel(const OpArgs &args, hipStream_t stream);

// instance: HEAL_INSTANCE_* (AUTO chooses from M and N).
hipError_t launch_gemm_op(int op, int instance, const OpArgs &args, hipStream_t stream);

hipError_t launch_split_f16(const float *x, uint16_t *hi, uint16_t *lo, int64_t n,
                            hipStream_t stream);
// kind 0: FP16 weight RNE_f16(src * 2^e), one plane; kind 1: bf16 (hi, lo) planes.
hipError_t launch_pack(int kind, const float *src, int64_t K, int64_t N, int64_t ld, bool trans,
                       int e, uint16_t *out, hipStream_t stream);
hipError_t launch_maxabs(const float *x, int64_t rows, int64_t cols, int64_t ld, float *maxabs,
                         hipStream_t stream);
hipError_t launch_quantize(const float *x, int64_t n, int16_t *q, float *maxabs,
                           hipStream_t stream);

}  // namespace heal
