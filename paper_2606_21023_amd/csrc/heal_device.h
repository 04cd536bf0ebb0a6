// Device-side building blocks shared by the split and GEMM kernels (gfx950).
#pragma once

#include <stdint.h>
#include <hip/hip_runtime.h>

namespace heal {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Split two FP32 values into packed bf16 pairs (element 0 in the low half):
//   hi = RNE_bf16(x)                       -- one v_cvt_pk_bf16_f32 for both
//   lo = RNE_bf16(x - hi), or +0 when hi is infinite or NaN
// (HEAL Section 4, GEMM paragraph: the FP32 operand becomes a 16-bit head plus
// a 16-bit residual; here both halves are bf16, so no residual scaling).
// x - hi is exact: |x - hi| is at most half a bf16 step of x and lies on x's
// FP32 grid.  Widening a bf16 to FP32 is a 16-bit shift of its pattern.
__device__ __forceinline__ void split2(float x0, float x1, uint32_t &hi, uint32_t &lo)
{
    f32x2 v = {x0, x1};
    hi = __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
    const float h0 = __builtin_bit_cast(float, hi << 16);
    const float h1 = __builtin_bit_cast(float, hi & 0xffff0000u);
    float r0 = x0 - h0;
    float r1 = x1 - h1;
    r0 = (__builtin_fabsf(h0) < __builtin_inff()) ? r0 : 0.0f;
    r1 = (__builtin_fabsf(h1) < __builtin_inff()) ? r1 : 0.0f;
    f32x2 r = {r0, r1};
    lo = __builtin_bit_cast(uint32_t, __builtin_convertvector(r, bf16x2));
}

}  // namespace heal
