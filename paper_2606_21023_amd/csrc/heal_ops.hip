// Element-wise kernels of the FP16 and INT16 forms of the method:
//   - the HEAL-Full activation pair on its own (split_f16_kernel);
//   - packing a weight into MFMA fragment order, either as FP16 scaled by a
//     power of two (HEAL-Base / HEAL-Full weights) or as a bf16 (hi, lo) pair
//     (pre-split operand of the bf16x3 product);
//   - max|x| of a matrix and the INT16 codes of a tensor (HEAL+).
// All HBM-bound.
#include "heal_device.h"
#include "heal_internal.h"

namespace heal {

namespace {

constexpr int kThreads = 256;
// Streaming kernels take one step per thread up to the grid limit (the loops
// stride only past it): capping the grid at 4096 workgroups that stride over
// the rest cost 10-15% of HBM bandwidth on the standalone splits.  The max|x|
// reduction folds one atomic per workgroup into a single word, so it keeps a
// small grid whose threads stride with four loads in flight (max|x| of 64M
// elements: 512 workgroups 43 us, 1024 49 us, 2048 53 us, 4096 67 us, 8192
// 106 us).
constexpr int64_t kMaxBlocks = 0x40000000LL;
#ifndef HEAL_REDUCE_BLOCKS
#define HEAL_REDUCE_BLOCKS 512
#endif

int64_t blocks_for(int64_t work, int64_t per_block, int64_t cap = kMaxBlocks)
{
    int64_t b = (work + per_block - 1) / per_block;
    if (b > cap) b = cap;
    return b < 1 ? 1 : b;
}

template <bool VEC>
__global__ void __launch_bounds__(kThreads)
split_f16_kernel(const float *__restrict__ x, uint16_t *__restrict__ hi, uint16_t *__restrict__ lo,
                 int64_t n)
{
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    const int64_t t = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    int64_t done = 0;
    if (VEC) {
        const int64_t n8 = n / 8;
        const f32x4 *x4 = reinterpret_cast<const f32x4 *>(x);
        u32x4 *h4 = reinterpret_cast<u32x4 *>(hi);
        u32x4 *l4 = reinterpret_cast<u32x4 *>(lo);
        for (int64_t i = t; i < n8; i += stride) {
            const f32x4 a = __builtin_nontemporal_load(x4 + 2 * i);
            const f32x4 b = __builtin_nontemporal_load(x4 + 2 * i + 1);
            uint32_t h0, h1, h2, h3, l0, l1, l2, l3;
            split2_f16(a.x, a.y, h0, l0);
            split2_f16(a.z, a.w, h1, l1);
            split2_f16(b.x, b.y, h2, l2);
            split2_f16(b.z, b.w, h3, l3);
            const u32x4 h = {h0, h1, h2, h3}, l = {l0, l1, l2, l3};
            __builtin_nontemporal_store(h, h4 + i);
            __builtin_nontemporal_store(l, l4 + i);
        }
        done = n8 * 8;
    }
    for (int64_t i = done + t; i < n; i += stride) {
        uint32_t h, l;
        split2_f16(x[i], 0.0f, h, l);
        hi[i] = (uint16_t)h;
        lo[i] = (uint16_t)l;
    }
}

// Fragment-order packing.  Output unit u = (jb * KC + kc) * 64 + lane holds,
// for each plane p, the 8 values k = 32*kc + 8*(lane >> 4) + t (t = 0..7) of
// column n = 16*jb + (lane & 15), at
//   out[((jb * KC + kc) * P + p) * 512 + lane * 8 + t];
// positions outside K x N hold +0.  Element (k, n) of the operand is
// src[n * ld + k] when the source is stored N x K (TRANS) and src[k * ld + n]
// when it is stored K x N.
// KIND 0: P = 1, RNE_f16(src * 2^e).  KIND 1: P = 2, the bf16 (hi, lo) split.
template <int KIND, bool TRANS>
__global__ void __launch_bounds__(kThreads)
pack_kernel(const float *__restrict__ src, int64_t K, int64_t N, int64_t ld, int e,
            uint16_t *__restrict__ out, int64_t KC, int64_t units)
{
    constexpr int P = KIND == 0 ? 1 : 2;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t u = (int64_t)blockIdx.x * kThreads + threadIdx.x; u < units; u += stride) {
        const int lane = (int)(u & 63);
        const int64_t blk = u >> 6;  // jb * KC + kc
        const int64_t jb = blk / KC, kc = blk - jb * KC;
        const int64_t n = 16 * jb + (lane & 15);
        const int64_t k0 = 32 * kc + 8 * (lane >> 4);
        float v[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int64_t k = k0 + t;
            v[t] = (n < N && k < K) ? (TRANS ? src[n * ld + k] : src[k * ld + n]) : 0.0f;
        }
        uint16_t *dst = out + blk * P * 512 + lane * 8;
        if (KIND == 0) {
            u32x4 h;
#pragma unroll
            for (int t = 0; t < 4; ++t)
                h[t] = cvt2_f16(ldexpf(v[2 * t], e), ldexpf(v[2 * t + 1], e));
            *reinterpret_cast<u32x4 *>(dst) = h;
        } else {
            u32x4 h, l;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                uint32_t hh, ll;
                split2(v[2 * t], v[2 * t + 1], hh, ll);
                h[t] = hh;
                l[t] = ll;
            }
            *reinterpret_cast<u32x4 *>(dst) = h;
            *reinterpret_cast<u32x4 *>(dst + 512) = l;
        }
    }
}

// One thread clears the reduction word (a kernel, not a memset, so that the
// sequence can be captured in a graph).
__global__ void zero_word_kernel(uint32_t *w) { *w = 0u; }

// max|x| of a rows x cols matrix with row stride ld: each workgroup reduces
// its elements and folds the result into *out with one atomic maximum on the
// bit pattern (for non-negative floats the unsigned order of the patterns is
// the numeric order, and a maximum is independent of the order of the folds).
__global__ void __launch_bounds__(kThreads)
maxabs_kernel(const float *__restrict__ x, int64_t rows, int64_t cols, int64_t ld,
              uint32_t *__restrict__ out)
{
    const int64_t n = rows * cols;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    uint32_t m = 0u;
    if (ld == cols && (reinterpret_cast<uintptr_t>(x) & 15u) == 0) {
        const int64_t n4 = n / 4;
        const f32x4 *x4 = reinterpret_cast<const f32x4 *>(x);
        // four 16-byte loads in flight per thread and trip
        for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n4; i += 4 * stride) {
            u32x4 b[4];
#pragma unroll
            for (int u = 0; u < 4; ++u)
                b[u] = i + u * stride < n4
                           ? __builtin_bit_cast(u32x4, __builtin_nontemporal_load(x4 + i + u * stride))
                           : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int t = 0; t < 4; ++t) m = max(m, b[u][t] & 0x7fffffffu);
        }
        for (int64_t i = 4 * n4 + (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride)
            m = max(m, __builtin_bit_cast(uint32_t, x[i]) & 0x7fffffffu);
    } else {
        for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride) {
            const int64_t r = i / cols, c = i - r * cols;
            m = max(m, __builtin_bit_cast(uint32_t, x[r * ld + c]) & 0x7fffffffu);
        }
    }
    // wave, then workgroup reduction
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
    __shared__ uint32_t part[kThreads / 64];
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t b = part[0];
#pragma unroll
        for (int w = 1; w < kThreads / 64; ++w) b = max(b, part[w]);
        atomicMax(out, b);
    }
}

// INT16 code of one element: the real quotient 32767 x / m rounded to the
// nearest integer, ties to even.  32767 x is exact in FP64, and one correctly
// rounded FP64 division cannot carry a quotient across a half-integer it does
// not equal: with x and m on the grid of x's last place 2^a (|m| >= |x|), a
// half-integer other than the quotient is at least 2^a / (2 |m|) away, the
// division's error at most 2^-53 * 32767 |x| / |m| < 2^(a-14) / |m|; a quotient
// that is a half-integer is representable and comes out exactly, so rint
// takes the even side.  The quotient stays within 32767 in magnitude for any
// m > 0, however small.
__device__ __forceinline__ int code_i16(float x, double m)
{
    return (int)__builtin_rint((32767.0 * (double)x) / m);
}

// INT16 codes q = Round(32767 x / m), m = max|X| read from *maxabs (m = 0
// gives all-zero codes).  HBM-bound: the FP64 division per element hides
// behind the 6 bytes each element moves.
__global__ void __launch_bounds__(kThreads)
quantize_kernel(const float *__restrict__ x, int64_t n, int16_t *__restrict__ q,
                const float *__restrict__ maxabs)
{
    const float mf = *maxabs;
    const bool zero = !(mf > 0.0f);
    const double m = zero ? 1.0 : (double)mf;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    const int64_t t0 = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    int64_t done = 0;
    if (((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(q)) & 15u) == 0) {
        const int64_t n8 = n / 8;
        const f32x4 *x4 = reinterpret_cast<const f32x4 *>(x);
        u32x4 *q4 = reinterpret_cast<u32x4 *>(q);
        for (int64_t i = t0; i < n8; i += stride) {
            const f32x4 a = __builtin_nontemporal_load(x4 + 2 * i);
            const f32x4 b = __builtin_nontemporal_load(x4 + 2 * i + 1);
            const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
            u32x4 o;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int c0 = zero ? 0 : code_i16(v[2 * t], m);
                const int c1 = zero ? 0 : code_i16(v[2 * t + 1], m);
                o[t] = ((uint32_t)c0 & 0xffffu) | ((uint32_t)c1 << 16);
            }
            __builtin_nontemporal_store(o, q4 + i);
        }
        done = n8 * 8;
    }
    for (int64_t i = done + t0; i < n; i += stride)
        q[i] = (int16_t)(zero ? 0 : code_i16(x[i], m));
}

}  // namespace

hipError_t launch_split_f16(const float *x, uint16_t *hi, uint16_t *lo, int64_t n,
                            hipStream_t stream)
{
    const bool vec = ((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(hi) |
                       reinterpret_cast<uintptr_t>(lo)) & 15u) == 0;
    const int64_t blocks = blocks_for(n, (int64_t)kThreads * (vec ? 8 : 1));
    if (vec)
        hipLaunchKernelGGL(split_f16_kernel<true>, dim3((unsigned)blocks), dim3(kThreads), 0,
                           stream, x, hi, lo, n);
    else
        hipLaunchKernelGGL(split_f16_kernel<false>, dim3((unsigned)blocks), dim3(kThreads), 0,
                           stream, x, hi, lo, n);
    return hipGetLastError();
}

hipError_t launch_pack(int kind, const float *src, int64_t K, int64_t N, int64_t ld, bool trans,
                       int e, uint16_t *out, hipStream_t stream)
{
    const int64_t KC = (K + 31) / 32;
    const int64_t units = ((N + 15) / 16) * KC * 64;
    const dim3 grid((unsigned)blocks_for(units, kThreads));
    if (kind == 0) {
        if (trans)
            hipLaunchKernelGGL((pack_kernel<0, true>), grid, dim3(kThreads), 0, stream, src, K, N,
                               ld, e, out, KC, units);
        else
            hipLaunchKernelGGL((pack_kernel<0, false>), grid, dim3(kThreads), 0, stream, src, K,
                               N, ld, e, out, KC, units);
    } else {
        if (trans)
            hipLaunchKernelGGL((pack_kernel<1, true>), grid, dim3(kThreads), 0, stream, src, K, N,
                               ld, e, out, KC, units);
        else
            hipLaunchKernelGGL((pack_kernel<1, false>), grid, dim3(kThreads), 0, stream, src, K,
                               N, ld, e, out, KC, units);
    }
    return hipGetLastError();
}

hipError_t launch_maxabs(const float *x, int64_t rows, int64_t cols, int64_t ld, float *maxabs,
                         hipStream_t stream)
{
    uint32_t *w = reinterpret_cast<uint32_t *>(maxabs);
    hipLaunchKernelGGL(zero_word_kernel, dim3(1), dim3(1), 0, stream, w);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    const int64_t n = rows * cols;
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(maxabs_kernel,
                       dim3((unsigned)blocks_for(n, (int64_t)kThreads * 16, HEAL_REDUCE_BLOCKS)),
                       dim3(kThreads), 0, stream, x, rows, cols, ld, w);
    return hipGetLastError();
}

hipError_t launch_quantize(const float *x, int64_t n, int16_t *q, float *maxabs,
                           hipStream_t stream)
{
    hipError_t err = launch_maxabs(x, 1, n, n, maxabs, stream);
    if (err != hipSuccess || n == 0) return err;
    hipLaunchKernelGGL(quantize_kernel, dim3((unsigned)blocks_for(n, (int64_t)kThreads * 8)),
                       dim3(kThreads), 0, stream, x, n, q, maxabs);
    return hipGetLastError();
}

}  // namespace heal
