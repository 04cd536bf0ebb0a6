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
bool skinny_kernel_applies(const GemmArgs &args, bool trans_b);
hipError_t launch_gemm_skinny(const GemmArgs &args, bool trans_b, bool use_alpha,
                              hipStream_t stream);

hipError_t launch_split(const float *x, uint16_t *hi, uint16_t *lo, int64_t n, hipStream_t stream);

}  // namespace heal
