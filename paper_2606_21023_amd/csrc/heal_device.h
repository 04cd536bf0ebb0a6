// Device-side building blocks shared by the split and GEMM kernels (gfx950).
#pragma once

#include <stdint.h>
#include <hip/hip_runtime.h>

// Tile rows per rasterisation group of the tiled GEMM kernels: consecutive
// workgroups of one XCD walk GM tile rows before moving to the next tile
// column, so that they share A and B panels in that XCD's L2.
#ifndef HEAL_GROUP_M
#define HEAL_GROUP_M 8
#endif

namespace heal {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

// Split two FP32 values into packed bf16 pairs (element 0 in the low half):
//   hi = RNE_bf16(x)          -- one v_cvt_pk_bf16_f32 for both elements
//   lo = RNE_bf16(x - hi)     -- widen hi (shift / mask), subtract, convert
// (HEAL Section 4, GEMM paragraph: the FP32 operand becomes a 16-bit head plus
// a 16-bit residual; here both halves are bf16, so no residual scaling).
// x - hi is exact for finite hi: |x - hi| is at most half a bf16 step of x and
// lies on x's FP32 grid.  Non-finite inputs follow IEEE arithmetic (an
// infinite x gives lo = NaN).  Six VALU instructions per pair.
__device__ __forceinline__ void split2(float x0, float x1, uint32_t &hi, uint32_t &lo)
{
    f32x2 v = {x0, x1};
    hi = __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
    f32x2 r = {x0 - __builtin_bit_cast(float, hi << 16),
               x1 - __builtin_bit_cast(float, hi & 0xffff0000u)};
    lo = __builtin_bit_cast(uint32_t, __builtin_convertvector(r, bf16x2));
}

// HEAL-Full pair of two FP32 values, packed binary16 (element 0 in the low half):
//   hi = RNE_f16(x)                 -- one v_cvt_pk_f16_f32 for both elements
//   lo = RNE_f16((x - hi) * 2^10)   -- widen hi, subtract, shift, convert
// (HEAL Section 4, GEMM paragraph: the activation becomes an FP16 head plus an
// FP16 residual shifted up by 2^10 so that it keeps FP16's normal range).
// x - hi is exact in FP32 and so is the 2^10 shift (|x - hi| <= 2^4 below the
// overflow threshold); an infinite head gives lo = -/+inf or NaN by IEEE rules.
__device__ __forceinline__ void split2_f16(float x0, float x1, uint32_t &hi, uint32_t &lo)
{
    f32x2 v = {x0, x1};
    f16x2 h = __builtin_convertvector(v, f16x2);
    f32x2 hf = __builtin_convertvector(h, f32x2);
    f32x2 r = {(x0 - hf.x) * 1024.0f, (x1 - hf.y) * 1024.0f};
    hi = __builtin_bit_cast(uint32_t, h);
    lo = __builtin_bit_cast(uint32_t, __builtin_convertvector(r, f16x2));
}

// RNE_f16 of two FP32 values, packed (the single cast of HEAL-Base).
__device__ __forceinline__ uint32_t cvt2_f16(float x0, float x1)
{
    f32x2 v = {x0, x1};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, f16x2));
}

// Dual-FP16 pair of two INT16 codes q (HEAL Section 4, Q/K/V paragraph):
// hi = RNE_f16(q) and the remainder q - hi, an integer with |q - hi| <= 8,
// both exact in FP16, so hi + (q - hi) == q.  The remainder is the paper's
// lower half divided by 2^10; feeding it to the matrix unit instead of the
// shifted half and scaling its products back by 2^-10 gives the same exact
// products.
__device__ __forceinline__ void unpack2_i16(int q0, int q1, uint32_t &hi, uint32_t &lo)
{
    f32x2 v = {(float)q0, (float)q1};
    f16x2 h = __builtin_convertvector(v, f16x2);
    f32x2 hf = __builtin_convertvector(h, f32x2);
    f32x2 r = {v.x - hf.x, v.y - hf.y};
    hi = __builtin_bit_cast(uint32_t, h);
    lo = __builtin_bit_cast(uint32_t, __builtin_convertvector(r, f16x2));
}

// Two 16 x 16 FP32 MFMA results of adjacent 16-column blocks, r0 and r1
// (lane fr + 16 fg holds row fr, columns 4 fg .. 4 fg + 3 of its block),
// rearranged for stores of whole 128-byte lines: lane (fr, fg) of x holds
// row fr & 7, and of y row 8 + (fr & 7), columns 16 (fr >> 3) + 4 fg .. + 3
// of the 32-column pair.  Lanes 8..15 of each 16-lane row trade halves
// with lanes 0..7 (a DPP rotation by 8 within the row), so one store of x
// or y writes 8 rows x 128 bytes instead of 16 rows x 64 bytes.
__device__ __forceinline__ void whole_lines(f32x4 r0, f32x4 r1, int fr, f32x4 &x, f32x4 &y)
{
    const bool low = fr < 8;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        // each element through a scalar first: __builtin_bit_cast of a
        // vector element expression compiles to element 0 for every e
        const float a = r0[e], b = r1[e];
        const float s0 = __builtin_bit_cast(
            float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, a), 0x128, 0xf, 0xf, false));
        const float s1 = __builtin_bit_cast(
            float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, b), 0x128, 0xf, 0xf, false));
        x[e] = low ? a : s1;
        y[e] = low ? s0 : b;
    }
}

}  // namespace heal
