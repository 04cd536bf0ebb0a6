// GEMM kernels of the FP16 and INT16 forms of the method, and of the bf16x3
// product with a pre-split B operand, for gfx950 (MI355X).
//
//   OP_BASE     HEAL-Base (Appendix "HEAL Implementation"): the FP32 activation
//               is cast once to FP16 and multiplied by the FP16 weight, which
//               was scaled by a per-matrix power of two 2^e;
//               C = 2^-e * sum_k f16(a) w16.
//   OP_FULL     HEAL-Full (Section 4, GEMM paragraph and its two-product
//               expansion): the activation is the pair h_hi = f16(h),
//               h_lo = f16((h - h_hi) 2^10); both products go into one FP32
//               accumulator, the residual's 2^-10 moved onto the weight
//               (GEMM(h_lo / 2^10, W) = GEMM(h_lo, W / 2^10)):
//               C = 2^-e * sum_k (h_hi w16 + h_lo f16(w16 2^-10)).
//               w16 2^-10 is exact for |w16| >= 2^-4, i.e. every weight
//               above 2^-20 of the largest one (the scaled weights reach
//               2^15).
//   OP_SCORES   HEAL+ score product (Section 4, Q/K/V paragraph and its
//               attention expansion): INT16 codes of Q and K are unpacked into
//               dual-FP16 pairs and all four products are accumulated:
//               C = f * sum_k qQ qK, f = alpha (maxQ/32767)(maxK/32767)
//               computed in FP64 and rounded once to FP32.
//   OP_PRESPLIT the bf16x3 compensated product of heal_gemm_f32 with B already
//               split into bf16 (hi, lo) and packed: the same MFMAs in the same
//               order, so the result is bitwise equal to heal_gemm_f32.
//
// Data path of one workgroup (one BM x BN output tile):
//   A (row-major FP32 or INT16) --16-byte loads--> VGPRs --convert / split-->
//   LDS planes (k-contiguous rows, XOR-swizzled);
//   B packed in MFMA fragment order (16 columns x 32 k per 1 KiB block and
//   plane) --16-byte loads--> VGPRs --copy--> LDS (no swizzle: each lane
//   reads its own 16 bytes of a block, consecutive lanes consecutive
//   addresses), or B as INT16 rows converted like A;
//   two LDS stages, one barrier per stage; v_mfma_f32_16x16x32_{f16,bf16}.
// Two kernels share this data path: the generic template gemm_op_kernel (any
// tile configuration; the conversion of the next stage follows the MFMAs)
// and gemm_op8_kernel, the large tiles of the packed-weight products with the
// conversion interleaved between the MFMAs (used wherever its 16-byte loads
// apply).
//
// Reduction order, identical in every instance of one product (so results
// are bitwise equal run to run and for every M): K is walked in 32-deep
// chunks in ascending order; per chunk the products are added in a fixed
// order (listed at each product); the K tail and out-of-range rows and
// columns are zero-filled.  No split-K and no atomics.
//
// MFMA operand roles as in the bf16x3 kernels: the B fragment is the first
// source (16 output columns n), the A fragment the second (16 output rows m),
// so each lane's accumulator is C[m][n..n+3].
#include "heal.h"
#include "heal_device.h"
#include "heal_internal.h"

#include <atomic>

// C stores of whole 128-byte lines (pairs of 16-column result blocks, see
// whole_lines), against 64-byte pieces, same bits: in the hand-scheduled
// large kernel 8192^3 0.8-2.0% and 2048 x 14336 x 4096 3-6% faster for the
// three packed-weight products; in the generic tiles (medium and skinny)
// 2048 x 1792 x 4096 and lm_head 2-6% faster.
#ifndef HEAL_OP8_C_LINES
#define HEAL_OP8_C_LINES 1
#endif
#ifndef HEAL_OP_C_LINES
#define HEAL_OP_C_LINES 1
#endif

namespace heal {

namespace {

template <int OP>
struct OpT;
// AP, BP: LDS planes of A and B;
// A_I16: A holds INT16 codes; B_ROWS: B is INT16 N x K rows (else packed).
template <>
struct OpT<OP_BASE> {
    static constexpr int AP = 1, BP = 1;
    static constexpr bool A_I16 = false, B_ROWS = false;
};
template <>
struct OpT<OP_FULL> {
    static constexpr int AP = 2, BP = 1;
    static constexpr bool A_I16 = false, B_ROWS = false;
};
template <>
struct OpT<OP_SCORES> {
    static constexpr int AP = 2, BP = 2;
    static constexpr bool A_I16 = true, B_ROWS = true;
};
template <>
struct OpT<OP_PRESPLIT> {
    static constexpr int AP = 2, BP = 2;
    static constexpr bool A_I16 = false, B_ROWS = false;
};

template <bool BF16>
__device__ __forceinline__ f32x4 mma(u32x4 b, u32x4 a, f32x4 c)
{
    if constexpr (BF16)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, b),
                                                       __builtin_bit_cast(bf16x8, a), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, b),
                                                      __builtin_bit_cast(f16x8, a), c, 0, 0, 0);
}

constexpr int kRsrcFlags = 0x00020000;  // raw buffer, 32-bit data format
constexpr uint32_t kOOB = 0x80000000u;  // offset beyond num_records: the load returns zeros

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, 0x7fffffff,
                                             kRsrcFlags);
}

__device__ __forceinline__ u32x4 bload(__amdgpu_buffer_rsrc_t r, uint32_t voff)
{
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, 0, 0));
}

// R: register sets of staged operands.  R = 1: the next stage is loaded
// while the current one is multiplied out (one stage of compute to hide the
// load).  R = 2, 4, ...: a ring of R sets, each reloaded R stages ahead, for
// narrow tiles whose compute per stage is too short to hide a load (their
// weight stream is bound by the bytes in flight per CU).
template <int OP, int BM, int BN, int WM, int WN, int NT, int BK, int R, bool VEC>
__global__ void __launch_bounds__(NT)
gemm_op_kernel(OpArgs p)
{
    using O = OpT<OP>;
    constexpr int ROWB = BK * 2;                 // bytes per LDS row of one plane
    constexpr int NCH = BK / 8;                  // 16-byte chunks per row
    constexpr int RPW = BK >= 64 ? 1 : 64 / BK;  // rows sharing one 128-byte window
    constexpr int SWM = (NCH < 8 ? NCH : 8) - 1; // XOR swizzle mask on the chunk index
    constexpr int KS = BK / 32;                  // MFMA chunks per stage
    constexpr int A_PLANE = BM * ROWB;
    constexpr int B_PLANE = BN * ROWB;
    constexpr int STAGE = O::AP * A_PLANE + O::BP * B_PLANE;
    constexpr int WAVES_M = BM / WM;
    constexpr int FM = WM / 16, FN = WN / 16;
    // the first CWAVES waves compute one wave tile each; all NT threads load
    // and convert (extra waves only help move a narrow tile's operands)
    constexpr int CWAVES = WAVES_M * (BN / WN);
    static_assert(BK % 32 == 0 && BK <= 512, "stage depth");
    static_assert(R >= 1 && R <= 8, "register sets");
    static_assert(BM % WM == 0 && BN % WN == 0 && WM % 16 == 0 && WN % 16 == 0, "wave tiling");
    static_assert(CWAVES * 64 <= NT && NT % 64 == 0, "compute waves exceed the workgroup");

    // 16-byte load units of one stage
    constexpr int A_EPU = O::A_I16 ? 8 : 4;      // A elements per unit
    constexpr int A_UPR = BK / A_EPU;            // units per A row
    constexpr int A_UNITS = BM * A_UPR;
    constexpr int A_IT = (A_UNITS + NT - 1) / NT;
    constexpr int B_UPR = BK / 8;                // INT16 B rows: units per row
    constexpr int B_BLK = KS * O::BP * 64;       // packed B: units per 16-column block
    constexpr int B_UNITS = O::B_ROWS ? BN * B_UPR : (BN / 16) * B_BLK;
    constexpr int B_IT = (B_UNITS + NT - 1) / NT;
    constexpr int ESZ_A = O::A_I16 ? 2 : 4;

    static_assert(2 * STAGE <= 160 * 1024, "two LDS stages must fit the 160 KB of a CU");
    __shared__ __attribute__((aligned(16))) char smem0[STAGE];
    __shared__ __attribute__((aligned(16))) char smem1[STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int fr = lane & 15;
    const int fg = lane >> 4;
    const int wm = wave % WAVES_M;
    const int wn = (wave / WAVES_M) % (BN / WN);
    const bool computes = CWAVES * 64 == NT || wave < CWAVES;

    auto swz = [](int row) { return (row / RPW) & SWM; };
    auto chunk_off = [&](int row, int c) { return row * ROWB + ((c ^ swz(row)) << 4); };
    auto quad_off = [&](int row, int kq) {
        return row * ROWB + (((kq >> 1) ^ swz(row)) << 4) + ((kq & 1) << 3);
    };

    // ---- tile coordinates: XCD-aware, grouped along M (as the bf16x3 kernels)
    const int64_t tiles_m = (p.M + BM - 1) / BM;
    const int64_t tiles_n = (p.N + BN - 1) / BN;
    const int64_t nb = (int64_t)gridDim.x;
    int64_t bid = blockIdx.x;
    {
        const int64_t x = bid & 7, i = bid >> 3, q = nb >> 3, r = nb & 7;
        bid = x * q + (x < r ? x : r) + i;
    }
    constexpr int GM = HEAL_GROUP_M;
    const int64_t group = bid / (GM * tiles_n);
    const int64_t first_m = group * GM;
    const int64_t gm = (tiles_m - first_m) < GM ? (tiles_m - first_m) : GM;
    const int64_t in_group = bid - group * GM * tiles_n;
    const int64_t m0 = (first_m + in_group % gm) * BM;
    const int64_t n0 = (in_group / gm) * BN;

    const int64_t M = p.M, N = p.N, K = p.K;
    const int64_t nk = (K + BK - 1) / BK;
    const int64_t KC = (K + 31) / 32;            // packed B: chunks per column block
    const int64_t NB16 = (N + 15) / 16;          // packed B: column blocks

    for (int64_t b = blockIdx.y; b < p.batch; b += gridDim.y) {
        const char *Ab = reinterpret_cast<const char *>(p.A) + b * p.strideA * ESZ_A;
        const char *Bb = reinterpret_cast<const char *>(p.B) + b * p.strideB * 2;
        float *__restrict__ C = p.C + b * p.strideC;

        const __amdgpu_buffer_rsrc_t rsrc_a = make_rsrc(Ab + m0 * p.lda * ESZ_A);
        const __amdgpu_buffer_rsrc_t rsrc_b =
            O::B_ROWS ? make_rsrc(Bb + n0 * p.ldb * 2)
                      : make_rsrc(Bb + (n0 / 16) * KC * O::BP * 1024);

        f32x4 acc[FN][FM];
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int i = 0; i < FM; ++i) acc[j][i] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

        u32x4 ra[R][A_IT], rb[R][B_IT];

        // ---- global -> register set `set` for the stage starting at k0 ---
        auto load_stage = [&](int set, int64_t k0) {
#pragma unroll
            for (int it = 0; it < A_IT; ++it) {
                const int u = it * NT + tid;
                if (A_UNITS % NT != 0 && u >= A_UNITS) continue;
                const int row = u / A_UPR, c = u % A_UPR;
                const int64_t k = k0 + (int64_t)c * A_EPU;
                const bool ok = m0 + row < M && k < K;
                if (VEC) {
                    const uint32_t off =
                        ok ? (uint32_t)(((int64_t)row * p.lda + k) * ESZ_A) : kOOB;
                    ra[set][it] = bload(rsrc_a, off);
                } else {
                    u32x4 v = {0u, 0u, 0u, 0u};
                    if (m0 + row < M) {
                        const char *rp = Ab + ((m0 + row) * p.lda + k) * ESZ_A;
                        if (O::A_I16) {
                            const int16_t *q = reinterpret_cast<const int16_t *>(rp);
#pragma unroll
                            for (int t = 0; t < 8; t += 2) {
                                const uint32_t lo16 = k + t < K ? (uint16_t)q[t] : 0u;
                                const uint32_t hi16 = k + t + 1 < K ? (uint16_t)q[t + 1] : 0u;
                                v[t / 2] = lo16 | (hi16 << 16);
                            }
                        } else {
                            const float *f = reinterpret_cast<const float *>(rp);
#pragma unroll
                            for (int t = 0; t < 4; ++t)
                                v[t] = k + t < K ? __builtin_bit_cast(uint32_t, f[t]) : 0u;
                        }
                    }
                    ra[set][it] = v;
                }
            }
#pragma unroll
            for (int it = 0; it < B_IT; ++it) {
                const int u = it * NT + tid;
                if (B_UNITS % NT != 0 && u >= B_UNITS) continue;
                if (O::B_ROWS) {
                    const int row = u / B_UPR, c = u % B_UPR;
                    const int64_t k = k0 + 8 * (int64_t)c;
                    if (VEC) {
                        const bool ok = n0 + row < N && k < K;
                        const uint32_t off =
                            ok ? (uint32_t)(((int64_t)row * p.ldb + k) * 2) : kOOB;
                        rb[set][it] = bload(rsrc_b, off);
                    } else {
                        u32x4 v = {0u, 0u, 0u, 0u};
                        if (n0 + row < N) {
                            const int16_t *q = reinterpret_cast<const int16_t *>(Bb) +
                                               (n0 + row) * p.ldb + k;
#pragma unroll
                            for (int t = 0; t < 8; t += 2) {
                                const uint32_t lo16 = k + t < K ? (uint16_t)q[t] : 0u;
                                const uint32_t hi16 = k + t + 1 < K ? (uint16_t)q[t + 1] : 0u;
                                v[t / 2] = lo16 | (hi16 << 16);
                            }
                        }
                        rb[set][it] = v;
                    }
                } else {
                    // packed: block j of the tile, unit r = (ks * BP + plane) * 64 + lane
                    const int j = u / B_BLK, r = u % B_BLK;
                    const int64_t kc = k0 / 32 + r / (O::BP * 64);
                    const bool ok = n0 / 16 + j < NB16 && kc < KC;
                    const uint32_t off =
                        ok ? (uint32_t)(((int64_t)j * KC * O::BP * 64 + (k0 / 32) * O::BP * 64 + r) *
                                        16)
                           : kOOB;
                    rb[set][it] = bload(rsrc_b, off);
                }
            }
        };

        // ---- register set -> LDS: convert A (and INT16 B), copy packed B --
        auto store_stage = [&](char *s, int set) {
            char *a0 = s, *a1 = s + A_PLANE;
            char *b0 = s + O::AP * A_PLANE, *b1 = b0 + B_PLANE;
#pragma unroll
            for (int it = 0; it < A_IT; ++it) {
                const int u = it * NT + tid;
                if (A_UNITS % NT != 0 && u >= A_UNITS) continue;
                const int row = u / A_UPR, c = u % A_UPR;
                const u32x4 v = ra[set][it];
                if constexpr (O::A_I16) {
                    u32x4 h, l;
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        uint32_t hh, ll;
                        unpack2_i16((int)(int16_t)(v[t] & 0xffffu), (int)(int16_t)(v[t] >> 16), hh,
                                    ll);
                        h[t] = hh;
                        l[t] = ll;
                    }
                    const int off = chunk_off(row, c);
                    *reinterpret_cast<u32x4 *>(a0 + off) = h;
                    *reinterpret_cast<u32x4 *>(a1 + off) = l;
                } else {
                    // bit-cast the whole vector: this compiler turns a bit-cast of
                    // one vector element into a read of element 0
                    const f32x4 xf = __builtin_bit_cast(f32x4, v);
                    const float x0 = xf.x, x1 = xf.y, x2 = xf.z, x3 = xf.w;
                    const int off = quad_off(row, c);
                    if constexpr (OP == OP_BASE) {
                        const u32x2 h = {cvt2_f16(x0, x1), cvt2_f16(x2, x3)};
                        *reinterpret_cast<u32x2 *>(a0 + off) = h;
                    } else {
                        uint32_t h0, l0, h1, l1;
                        if constexpr (OP == OP_FULL) {
                            split2_f16(x0, x1, h0, l0);
                            split2_f16(x2, x3, h1, l1);
                        } else {
                            split2(x0, x1, h0, l0);
                            split2(x2, x3, h1, l1);
                        }
                        const u32x2 h = {h0, h1}, l = {l0, l1};
                        *reinterpret_cast<u32x2 *>(a0 + off) = h;
                        *reinterpret_cast<u32x2 *>(a1 + off) = l;
                    }
                }
            }
#pragma unroll
            for (int it = 0; it < B_IT; ++it) {
                const int u = it * NT + tid;
                if (B_UNITS % NT != 0 && u >= B_UNITS) continue;
                const u32x4 v = rb[set][it];
                if constexpr (O::B_ROWS) {
                    const int row = u / B_UPR, c = u % B_UPR;
                    u32x4 h, l;
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        uint32_t hh, ll;
                        unpack2_i16((int)(int16_t)(v[t] & 0xffffu), (int)(int16_t)(v[t] >> 16), hh,
                                    ll);
                        h[t] = hh;
                        l[t] = ll;
                    }
                    const int off = chunk_off(row, c);
                    *reinterpret_cast<u32x4 *>(b0 + off) = h;
                    *reinterpret_cast<u32x4 *>(b1 + off) = l;
                } else {
                    *reinterpret_cast<u32x4 *>(b0 + u * 16) = v;
                }
            }
        };

        // ---- LDS -> fragments -> MFMA, one stage -------------------------
        auto compute_stage = [&](const char *s) {
            const char *a0 = s, *a1 = s + A_PLANE;
            const char *b0 = s + O::AP * A_PLANE, *b1 = b0 + B_PLANE;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                u32x4 ah[FM], al[FM];
#pragma unroll
                for (int i = 0; i < FM; ++i) {
                    const int off = chunk_off(wm * WM + i * 16 + fr, ks * 4 + fg);
                    ah[i] = *reinterpret_cast<const u32x4 *>(a0 + off);
                    if (O::AP == 2) al[i] = *reinterpret_cast<const u32x4 *>(a1 + off);
                }
#pragma unroll
                for (int j = 0; j < FN; ++j) {
                    u32x4 bh, bl;
                    if constexpr (O::B_ROWS) {
                        const int off = chunk_off(wn * WN + j * 16 + fr, ks * 4 + fg);
                        bh = *reinterpret_cast<const u32x4 *>(b0 + off);
                        bl = *reinterpret_cast<const u32x4 *>(b1 + off);
                    } else {
                        const int blk = (wn * FN + j) * KS + ks;
                        const int off = blk * O::BP * 1024 + lane * 16;
                        bh = *reinterpret_cast<const u32x4 *>(b0 + off);
                        if (O::BP == 2) bl = *reinterpret_cast<const u32x4 *>(b0 + off + 1024);
                    }
                    // HEAL-Full: the weight fragment scaled by 2^-10 for the
                    // residual product (exact unless it lands below 2^-14)
                    u32x4 bs;
                    if constexpr (OP == OP_FULL)
                        bs = __builtin_bit_cast(
                            u32x4, __builtin_bit_cast(f16x8, bh) * (_Float16)0x1p-10f);
#pragma unroll
                    for (int i = 0; i < FM; ++i) {
                        if constexpr (OP == OP_BASE) {
                            acc[j][i] = mma<false>(bh, ah[i], acc[j][i]);
                        } else if constexpr (OP == OP_FULL) {
                            // head product, then the residual product with the
                            // 2^-10 moved onto the weight: h_lo * (w 2^-10)
                            acc[j][i] = mma<false>(bh, ah[i], acc[j][i]);
                            acc[j][i] = mma<false>(bs, al[i], acc[j][i]);
                        } else if constexpr (OP == OP_SCORES) {
                            // hiQ*hiK, hiQ*loK, loQ*hiK, loQ*loK
                            acc[j][i] = mma<false>(bh, ah[i], acc[j][i]);
                            acc[j][i] = mma<false>(bl, ah[i], acc[j][i]);
                            acc[j][i] = mma<false>(bh, al[i], acc[j][i]);
                            acc[j][i] = mma<false>(bl, al[i], acc[j][i]);
                        } else {
                            // hiA*hiB, hiA*loB, loA*hiB: the order of heal_gemm_f32
                            acc[j][i] = mma<true>(bh, ah[i], acc[j][i]);
                            acc[j][i] = mma<true>(bl, ah[i], acc[j][i]);
                            acc[j][i] = mma<true>(bh, al[i], acc[j][i]);
                        }
                    }
                }
            }
        };

        // ---- main loop: two LDS stages, one barrier per stage -------------
        if constexpr (R == 1) {
            auto step = [&](const char *cur, char *nxt, int64_t kt) {
                if (kt + 1 < nk) load_stage(0, (kt + 1) * BK);
                if (computes) compute_stage(cur);
                if (kt + 1 < nk) store_stage(nxt, 0);
                __syncthreads();
            };
            if (nk > 0) {
                load_stage(0, 0);
                store_stage(smem0, 0);
                __syncthreads();
            }
            for (int64_t kt = 0; kt < nk; kt += 2) {
                step(smem0, smem1, kt);
                if (kt + 1 < nk) step(smem1, smem0, kt + 1);
            }
        } else {
            // stage t lives in register set t % R; at step kt the set of
            // stage kt+1 is stored and then reloaded with stage kt+1+R, so
            // each load has R steps to arrive.  Reloads past the last stage
            // are clamped to it (redundant loads whose data is never used).
            // The loop is unrolled by R (R even) so that the register set of
            // every step, and its LDS buffer, are compile-time constants.
            static_assert(R % 2 == 0, "R >= 2 register sets come in pairs");
            const int64_t last = nk - 1;
            auto clamp = [&](int64_t t) { return (t < last ? t : last) * BK; };
            auto step = [&](const char *cur, char *nxt, int set, int64_t kt) {
                if (computes && kt < nk) compute_stage(cur);
                store_stage(nxt, set);
                load_stage(set, clamp(kt + 1 + R));
                __syncthreads();
            };
            if (nk > 0) {
                load_stage(0, 0);
                store_stage(smem0, 0);
                // the sets are issued in ring order (scheduling barriers keep
                // the compiler from interleaving them), the order the loop
                // keeps, so that every wait before a store is exact
#pragma unroll
                for (int t = 1; t < R; ++t) {
                    __builtin_amdgcn_sched_barrier(0);
                    load_stage(t, clamp(t));
                }
                __builtin_amdgcn_sched_barrier(0);
                load_stage(0, clamp(R));
                __builtin_amdgcn_sched_barrier(0);
                __syncthreads();
            }
            // Every group of R steps runs whole, loads and stores included;
            // only the multiply of a step past the last stage is skipped (at
            // most R - 1 steps that load and store clamped copies).  With a
            // step under a branch the compiler has to assume a path around
            // it and waits for every outstanding load before each store
            // (vmcnt(0)), which empties the ring.
            for (int64_t kt0 = 0; kt0 < nk; kt0 += R) {
#pragma unroll
                for (int u = 0; u < R; ++u) {
                    if (u & 1)
                        step(smem1, smem0, (u + 1) % R, kt0 + u);
                    else
                        step(smem0, smem1, (u + 1) % R, kt0 + u);
                }
            }
        }

        // ---- epilogue: FP32 accumulators -> FP32 C, no downcast -----------
        float factor = 1.0f;
        if constexpr (OP == OP_SCORES) {
            // alpha (maxQ / 32767)(maxK / 32767) evaluated in FP64, rounded once
            factor = (float)((double)p.alpha * (double)*p.maxA * (double)*p.maxB /
                             (32767.0 * 32767.0));
        }
        auto result = [&](int j, int i) {
            f32x4 v;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                if constexpr (OP == OP_BASE || OP == OP_FULL)
                    v[t] = ldexpf(acc[j][i][t], -p.e);
                else if constexpr (OP == OP_SCORES)
                    v[t] = acc[j][i][t] * factor;
                else
                    v[t] = acc[j][i][t];
            }
            return v;
        };
        auto store_c = [&](int64_t m, int64_t n, f32x4 v) {
            if (m < M && n < N) {
                float *cp = C + m * p.ldc + n;
                if (p.vecC && n + 4 <= N) {
                    // streaming store: C is not read again here (INT16
                    // scores 1.07x, lm_head 1.01-1.035x, others unchanged)
                    __builtin_nontemporal_store(v, reinterpret_cast<f32x4 *>(cp));
                } else {
                    cp[0] = v.x;
                    if (n + 1 < N) cp[1] = v.y;
                    if (n + 2 < N) cp[2] = v.z;
                    if (n + 3 < N) cp[3] = v.w;
                }
            }
        };
        if (computes) {
            // pairs of 16-column blocks as whole 128-byte lines (not in the
            // 256-row tiles, which would spill more registers for it)
            constexpr int FL = HEAL_OP_C_LINES && BM < 256 ? FN / 2 * 2 : 0;
#pragma unroll
            for (int j = 0; j < FL; j += 2) {
#pragma unroll
                for (int i = 0; i < FM; ++i) {
                    f32x4 x, y;
                    whole_lines(result(j, i), result(j + 1, i), fr, x, y);
                    const int64_t mx = m0 + wm * WM + i * 16 + (fr & 7);
                    const int64_t n = n0 + wn * WN + j * 16 + 16 * (fr >> 3) + 4 * fg;
                    store_c(mx, n, x);
                    store_c(mx + 8, n, y);
                }
            }
#pragma unroll
            for (int j = FL; j < FN; ++j) {
#pragma unroll
                for (int i = 0; i < FM; ++i)
                    store_c(m0 + wm * WM + i * 16 + fr, n0 + wn * WN + j * 16 + 4 * fg, result(j, i));
            }
        }
        if (b + gridDim.y < p.batch) __syncthreads();  // LDS reuse by the next batch entry
    }
}

// The packed-weight products (HEAL-Base, HEAL-Full, pre-split) at 256 x BN
// tiles (BN = 256, or 224 where that needs fewer rounds of workgroups) with
// the schedule of the large bf16x3 kernel: eight waves of 64 x BN/2, two LDS
// stages, one barrier per stage of KS 32-deep chunks (KS = 2 for HEAL-Base,
// whose single product per chunk is short against the barrier; 1 otherwise).
// While stage s is multiplied out, each staged register group of stage s+1
// is converted into the other LDS buffer between the MFMAs of one column
// block and at once reloaded with stage s+2.  Per stage and thread: 4 KS
// 16-byte quads of A (quad q = tid + 512u: row q / (8 KS), k-quad
// q % (8 KS)), converted in the generic kernel's LDS layout (HEAL-Full: the
// FP16 pair; HEAL-Base: one FP16 plane; pre-split: the bf16 pair), and the
// tile's packed B as 16-byte units r = tid + 512v in packed order (column
// block, chunk, plane, lane), copied to LDS unchanged.  Same products in the
// same order as the generic kernel, so the bits are the same.
#ifndef HEAL_OP_LARGE8
#define HEAL_OP_LARGE8 1
#endif
#ifndef HEAL_OP_N224
#define HEAL_OP_N224 1
#endif
#ifndef HEAL_OP8_N224
#define HEAL_OP8_N224 1
#endif
#ifndef HEAL_OP8_BASE_KS
#define HEAL_OP8_BASE_KS 2
#endif

template <int OP, int BN, bool TAIL>
__global__ void __launch_bounds__(512, 1)
gemm_op8_kernel(OpArgs p)
{
    using O = OpT<OP>;
    static_assert(!O::A_I16 && !O::B_ROWS, "packed-weight products only");
    constexpr bool BF16 = OP == OP_PRESPLIT;
    constexpr int KS = OP == OP_BASE ? HEAL_OP8_BASE_KS : 1;   // 32-deep chunks per stage
    constexpr int NT = 512, BM = 256, BK = 32 * KS, ROWB = 2 * BK;
    static_assert(BN == 256 || BN == 224, "tile width");
    constexpr int WB = BN / 32;                  // column blocks per wave (two waves across)
    constexpr int TB = BN / 16;                  // column blocks per tile
    constexpr int KQ = BK / 4;                   // k-quads per A row and stage
    constexpr int RPW = BK >= 64 ? 1 : 64 / BK;  // rows sharing one 128-byte window
    constexpr int SWM = (BK / 8 < 8 ? BK / 8 : 8) - 1;
    constexpr int A_PLANE = BM * ROWB;           // one 16-bit plane of A
    constexpr int B_BYTES = TB * KS * O::BP * 1024;  // the tile's column blocks, fragment order
    constexpr int B_UNITS = TB * KS * O::BP * 64;   // 16-byte B units per stage
    constexpr int STAGE = O::AP * A_PLANE + B_BYTES;
    constexpr int NAU = BM * KQ / NT;            // A quads per thread and stage
    constexpr int NBU = (B_UNITS + NT - 1) / NT; // B units per thread and stage
    constexpr int NU = NAU + NBU;                // conversion units per thread and stage
    constexpr int MF = 4 * (OP == OP_BASE ? 1 : OP == OP_FULL ? 2 : 3);  // MFMAs per column block
    static_assert(NAU * NT == BM * KQ, "whole A quads per thread");
    constexpr int NSLOT = WB * KS;               // column blocks x chunks of one stage
    static_assert(NU <= 2 * NSLOT, "at most two units per column block and chunk");
    // instruction pattern per column block: NV x (MFMA, VPM VALU), then the
    // rest (measured at 8192^3: 8 x 2 for the pre-split product, 1.1% faster
    // than 10 x 3; 6 x 2 for HEAL-Full, within 0.5% of 6 x 3; HEAL-Base flat)
#ifdef HEAL_OP8_NV
    constexpr int NV = HEAL_OP8_NV < MF ? HEAL_OP8_NV : MF - 1;
#else
    constexpr int NV = MF == 12 ? 8 : MF - 2;
#endif
#ifdef HEAL_OP8_VPM
    constexpr int VPM = HEAL_OP8_VPM;
#else
    constexpr int VPM = MF == 4 ? 4 : 2;
#endif
    static_assert(2 * STAGE <= 160 * 1024, "two LDS stages must fit the 160 KB of a CU");
    __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave & 3, wn = wave >> 2;
    const int fr = lane & 15, fg = lane >> 4;
    auto swz = [](int row) { return (row / RPW) & SWM; };
    auto chunk_off = [&](int row, int c) { return row * ROWB + ((c ^ swz(row)) << 4); };
    auto quad_off = [&](int row, int kq) {
        return row * ROWB + (((kq >> 1) ^ swz(row)) << 4) + ((kq & 1) << 3);
    };

    // tile coordinates: XCD-aware, grouped along M (as the generic kernel)
    const int64_t tiles_m = (p.M + BM - 1) / BM;
    const int64_t tiles_n = (p.N + BN - 1) / BN;
    const int64_t nb = (int64_t)gridDim.x;
    int64_t bid = blockIdx.x;
    {
        const int64_t x = bid & 7, i = bid >> 3, q = nb >> 3, r = nb & 7;
        bid = x * q + (x < r ? x : r) + i;
    }
    constexpr int GM = HEAL_GROUP_M;
    const int64_t group = bid / (GM * tiles_n);
    const int64_t first_m = group * GM;
    const int64_t gm = (tiles_m - first_m) < GM ? (tiles_m - first_m) : GM;
    const int64_t in_group = bid - group * GM * tiles_n;
    const int64_t m0 = (first_m + in_group % gm) * BM;
    const int64_t n0 = (in_group / gm) * BN;

    const int64_t M = p.M, N = p.N, K = p.K;
    const int ns = (int)((K + BK - 1) / BK);     // stages
    const int64_t KC = (K + 31) / 32;            // packed chunks per column block
    const int64_t NB16 = (N + 15) / 16;
    const int rows_a = (int)((M - m0) < BM ? (M - m0) : BM);
    const int blocks_b = (int)((NB16 - n0 / 16) < TB ? (NB16 - n0 / 16) : TB);

    // A quad u of this thread: q = tid + 512u -> row q / KQ, k-quad q % KQ
    const int a_kq = tid % KQ;
    int st_a[NAU], a_rw[NAU];
#pragma unroll
    for (int u = 0; u < NAU; ++u) {
        a_rw[u] = (tid + NT * u) / KQ;
        st_a[u] = quad_off(a_rw[u], a_kq);
    }
    // B unit v: r = tid + 512v -> column block r / (64 KS BP), then chunk,
    // plane and lane (the packed order within a block)
    int b_kc[NBU];
#pragma unroll
    for (int v = 0; v < NBU; ++v) b_kc[v] = ((tid + NT * v) % (64 * KS * O::BP)) / (64 * O::BP);

    for (int64_t b = blockIdx.y; b < p.batch; b += gridDim.y) {
        const float *A = reinterpret_cast<const float *>(p.A) + b * p.strideA + m0 * p.lda;
        const char *Bp = reinterpret_cast<const char *>(p.B) + b * p.strideB * 2 +
                         (n0 / 16) * KC * O::BP * 1024;
        float *__restrict__ C = p.C + b * p.strideC;
        // ranges checked on the host to stay below 2^31 bytes
        const __amdgpu_buffer_rsrc_t ra_src = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<float *>(A), (short)0, (int)(((int64_t)(rows_a - 1) * p.lda + K) * 4),
            kRsrcFlags);
        const __amdgpu_buffer_rsrc_t rb_src = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<char *>(Bp), (short)0, (int)(blocks_b * KC * O::BP * 1024), kRsrcFlags);
        uint32_t va[NAU], vb[NBU];
#pragma unroll
        for (int u = 0; u < NAU; ++u)
            va[u] = a_rw[u] < rows_a ? (uint32_t)((a_rw[u] * p.lda + 4 * a_kq) * 4) : kOOB;
#pragma unroll
        for (int v = 0; v < NBU; ++v) {
            const int r = tid + NT * v, j = r / (64 * KS * O::BP);
            vb[v] = j < blocks_b && (B_UNITS % NT == 0 || r < B_UNITS)
                        ? (uint32_t)(j * KC * O::BP * 1024 + (r % (64 * KS * O::BP)) * 16)
                        : kOOB;
        }

        f32x4 ra[NAU];
        u32x4 rb[NBU];
        auto load_a = [&](int u, int s) {
            uint32_t v = va[u];
            if (TAIL && s * BK + 4 * a_kq >= K) v = kOOB;
            ra[u] = __builtin_bit_cast(
                f32x4, __builtin_amdgcn_raw_buffer_load_b128(ra_src, (int)v, s * BK * 4, 0));
        };
        auto load_b = [&](int v, int s) {
            uint32_t o = vb[v];
            // a stage reaching past the last packed chunk (K tail, KS > 1)
            if (TAIL && KS > 1 && s * KS + b_kc[v] >= KC) o = kOOB;
            rb[v] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                  rb_src, (int)o, s * KS * O::BP * 1024, 0));
        };
        // units 0..NAU-1: the A quads, converted; then packed B units, copied
        auto split_unit = [&](char *st, int u) {
            if (u < NAU) {
                const float x0 = ra[u].x, x1 = ra[u].y, x2 = ra[u].z, x3 = ra[u].w;
                const int off = st_a[u];
                if constexpr (OP == OP_BASE) {
                    const u32x2 h = {cvt2_f16(x0, x1), cvt2_f16(x2, x3)};
                    *reinterpret_cast<u32x2 *>(st + off) = h;
                } else {
                    uint32_t h0, l0, h1, l1;
                    if constexpr (OP == OP_FULL) {
                        split2_f16(x0, x1, h0, l0);
                        split2_f16(x2, x3, h1, l1);
                    } else {
                        split2(x0, x1, h0, l0);
                        split2(x2, x3, h1, l1);
                    }
                    const u32x2 h = {h0, h1}, l = {l0, l1};
                    *reinterpret_cast<u32x2 *>(st + off) = h;
                    *reinterpret_cast<u32x2 *>(st + A_PLANE + off) = l;
                }
            } else {
                const int v = u - NAU;
                if (B_UNITS % NT != 0 && tid + NT * v >= B_UNITS) return;
                *reinterpret_cast<u32x4 *>(st + O::AP * A_PLANE + (tid + NT * v) * 16) = rb[v];
            }
        };
        auto reload_unit = [&](int u, int s) {
            if (u < NAU) load_a(u, s);
            else load_b(u - NAU, s);
        };

        f32x4 acc[WB][4];
#pragma unroll
        for (int j = 0; j < WB; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[j][i] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

        if (ns > 0) {
#pragma unroll
            for (int u = 0; u < NU; ++u) reload_unit(u, 0);
#pragma unroll
            for (int u = 0; u < NU; ++u) split_unit(smem, u);
            const int s1 = ns > 1 ? 1 : 0;
#pragma unroll
            for (int u = 0; u < NU; ++u) reload_unit(u, s1);
            __syncthreads();
        }

        for (int s = 0; s < ns; ++s) {
            const char *cur = smem + (s & 1) * STAGE;
            char *nxt = smem + ((s + 1) & 1) * STAGE;
            const int s_reload = s + 2 < ns ? s + 2 : ns - 1;
            const char *a_hi = cur, *a_lo = cur + A_PLANE, *bw = cur + O::AP * A_PLANE;
#pragma unroll
            for (int kc = 0; kc < KS; ++kc) {
                // column block j of chunk kc: (wn*8 + j) KS BP KiB + kc BP KiB
                const int rd_b = ((wn * WB) * KS + kc) * O::BP * 1024 + lane * 16;
                const int rd_a = chunk_off(wm * 64 + fr, kc * 4 + fg);
                u32x4 ah[4], al[4], bh[2], bl[2];
                bh[0] = *reinterpret_cast<const u32x4 *>(bw + rd_b);
                if (O::BP == 2) bl[0] = *reinterpret_cast<const u32x4 *>(bw + rd_b + 1024);
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    ah[i] = *reinterpret_cast<const u32x4 *>(a_hi + rd_a + i * 16 * ROWB);
                if (O::AP == 2) {
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        al[i] = *reinterpret_cast<const u32x4 *>(a_lo + rd_a + i * 16 * ROWB);
                }
#pragma unroll
                for (int j = 0; j < WB; ++j) {
                    const int c = j & 1, slot = kc * WB + j;
                    if (j + 1 < WB) {
                        const int off = rd_b + (j + 1) * KS * O::BP * 1024;
                        bh[c ^ 1] = *reinterpret_cast<const u32x4 *>(bw + off);
                        if (O::BP == 2) bl[c ^ 1] = *reinterpret_cast<const u32x4 *>(bw + off + 1024);
                    }
#pragma unroll
                    for (int i = 0; i < 4; ++i) acc[j][i] = mma<BF16>(bh[c], ah[i], acc[j][i]);
                    // unit u goes to slot u, or (more units than slots) to
                    // slot u * NSLOT / NU
#pragma unroll
                    for (int u = 0; u < NU; ++u) {
                        if ((NU <= NSLOT ? u : u * NSLOT / NU) == slot) {
                            split_unit(nxt, u);
                            reload_unit(u, s_reload);
                        }
                    }
                    if constexpr (OP == OP_FULL) {
                        // the weight fragment scaled by 2^-10 for the residual product
                        const u32x4 bs = __builtin_bit_cast(
                            u32x4, __builtin_bit_cast(f16x8, bh[c]) * (_Float16)0x1p-10f);
#pragma unroll
                        for (int i = 0; i < 4; ++i) acc[j][i] = mma<false>(bs, al[i], acc[j][i]);
                    } else if constexpr (OP == OP_PRESPLIT) {
                        // hiA*hiB, hiA*loB, loA*hiB: the order of heal_gemm_f32
#pragma unroll
                        for (int i = 0; i < 4; ++i) acc[j][i] = mma<true>(bl[c], ah[i], acc[j][i]);
#pragma unroll
                        for (int i = 0; i < 4; ++i) acc[j][i] = mma<true>(bh[c], al[i], acc[j][i]);
                    }
                    // one column block: fragment reads, then MFMAs interleaved with
                    // the conversion's VALU work, LDS writes and the reloads
                    __builtin_amdgcn_sched_group_barrier(0x100, O::BP, 0);
#pragma unroll
                    for (int t = 0; t < NV; ++t) {
                        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                        __builtin_amdgcn_sched_group_barrier(0x002, VPM, 0);
                    }
                    __builtin_amdgcn_sched_group_barrier(0x200, 2, 0);
                    __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x008, MF - NV, 0);
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
            __syncthreads();
        }

        // epilogue: FP32 C (2^-e acc for the FP16 forms), streaming stores
        auto result = [&](int j, int i) {
            f32x4 v;
#pragma unroll
            for (int t = 0; t < 4; ++t)
                v[t] = OP == OP_PRESPLIT ? acc[j][i][t] : ldexpf(acc[j][i][t], -p.e);
            return v;
        };
        auto store_c = [&](int64_t m, int64_t n, f32x4 v) {
            if (m < M && n < N) {
                float *cp = C + m * p.ldc + n;
                if (p.vecC && n + 4 <= N) {
                    __builtin_nontemporal_store(v, reinterpret_cast<f32x4 *>(cp));
                } else {
                    cp[0] = v.x;
                    if (n + 1 < N) cp[1] = v.y;
                    if (n + 2 < N) cp[2] = v.z;
                    if (n + 3 < N) cp[3] = v.w;
                }
            }
        };
        constexpr int WL = HEAL_OP8_C_LINES ? WB / 2 * 2 : 0;   // blocks stored in whole lines
#pragma unroll
        for (int j = 0; j < WL; j += 2) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                f32x4 x, y;
                whole_lines(result(j, i), result(j + 1, i), fr, x, y);
                const int64_t mx = m0 + wm * 64 + i * 16 + (fr & 7);
                const int64_t n = n0 + wn * (BN / 2) + j * 16 + 16 * (fr >> 3) + 4 * fg;
                store_c(mx, n, x);
                store_c(mx + 8, n, y);
            }
        }
#pragma unroll
        for (int j = WL; j < WB; ++j) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                store_c(m0 + wm * 64 + i * 16 + fr, n0 + wn * (BN / 2) + j * 16 + 4 * fg, result(j, i));
        }
        if (b + gridDim.y < p.batch) __syncthreads();  // LDS reuse by the next batch entry
    }
}

// Whether the hand-scheduled kernel can run the call: 16-byte A rows, whole
// quads along K, and every buffer range below 2^31 bytes.
template <int OP>
bool op8_applies(const OpArgs &a)
{
    const int64_t lim = 0x7fffffffLL;
    if (!a.vecA || a.K % 4 != 0) return false;
    if (((int64_t)255 * a.lda + a.K) * 4 >= lim) return false;
    const int64_t KC = (a.K + 31) / 32;
    if (16 * KC * OpT<OP>::BP * 1024 >= lim) return false;
    return (a.M + 255) / 256 * ((a.N + 223) / 224) <= lim;
}

template <int OP, int BN>
hipError_t launch_op8(const OpArgs &a, hipStream_t stream)
{
    const int64_t tiles = ((a.M + 255) / 256) * ((a.N + BN - 1) / BN);
    const unsigned gy = (unsigned)(a.batch < 65535 ? a.batch : 65535);
    const dim3 grid((unsigned)tiles, gy);
    const int bk = OP == OP_BASE ? 32 * HEAL_OP8_BASE_KS : 32;
    if (a.K % bk)
        hipLaunchKernelGGL((gemm_op8_kernel<OP, BN, true>), grid, dim3(512), 0, stream, a);
    else
        hipLaunchKernelGGL((gemm_op8_kernel<OP, BN, false>), grid, dim3(512), 0, stream, a);
    return hipGetLastError();
}

// Whether the 16-byte buffer-load path can run the call: rows aligned, whole
// 16-byte units along K, and every byte offset inside a tile below 2^31.
// (Packed B is always read with buffer loads; the caller bounds K so that a
// tile's packed offsets stay below 2^31.)
// ---------------------------------------------------------------------------
// Streamed narrow tiles of the packed-B products (M <= 64, one 16-column
// block of the packed operand per workgroup).
//
// A K-sum of an output element stays in one wave (the fixed order), so a
// narrow tile is one chain of dependent MFMAs per 16-row block, K/32 x
// products long.  With one workgroup barrier per stage, every stage of that
// chain also waits for the fragment reads of its first chunk and for the
// barrier.  Here the roles are split: LW loader waves move A (converting it)
// and the packed B block into a ring of D LDS stages, one compute wave walks
// the ring chunk by chunk, reading the next chunk's fragments while the
// current chunk's MFMAs run, and the two sides hand stages over through LDS
// counters instead of barriers:
//   ready[s]  the loader waves that have stored the stage now in ring slot s
//             (a stage t in slot t % D is complete when ready reaches
//             (t / D + 1) * LW);
//   consumed  the stages the compute wave has finished reading (a loader
//             stores stage t only once consumed >= t - D + 1).
// A loader makes its LDS stores complete (s_waitcnt lgkmcnt(0)) before it
// adds to ready, and a wave's LDS requests are served in order, so a
// consumer that has seen the count reads the stored data.  Every wait on a
// counter polls at most HEAL_STREAM_SPIN_LIMIT times (seconds, far beyond any
// real wait): a defect that stalled a counter would give a wrong result
// instead of a kernel that never ends.
// Same conversions, MFMAs, chunk order and product order as gemm_op_kernel,
// so the bits are those of every other instance.
#ifndef HEAL_STREAM_SPIN_LIMIT
#define HEAL_STREAM_SPIN_LIMIT (1 << 20)
#endif

__device__ __forceinline__ uint32_t lds_load_relaxed(const uint32_t *p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ void spin_until_at_least(const uint32_t *p, uint32_t target)
{
    for (int i = 0; i < HEAL_STREAM_SPIN_LIMIT; ++i) {
        if (lds_load_relaxed(p) >= target) return;
        __builtin_amdgcn_s_sleep(1);
    }
}

template <int OP, int BM, int BK, int D, int LW, int PF, int R>
__global__ void __launch_bounds__((LW + 1) * 64)
gemm_op_stream_kernel(OpArgs p)
{
    using O = OpT<OP>;
    static_assert(!O::A_I16 && !O::B_ROWS, "packed-B products of an FP32 A");
    constexpr int ROWB = BK * 2;                 // bytes per LDS row of one A plane
    constexpr int NCH = BK / 8;
    constexpr int RPW = BK >= 64 ? 1 : 64 / BK;
    constexpr int SWM = (NCH < 8 ? NCH : 8) - 1;
    constexpr int KS = BK / 32;                  // MFMA chunks per stage
    constexpr int FM = BM / 16;
    constexpr int A_PLANE = BM * ROWB;
    constexpr int B_PLANE = KS * 1024;           // one packed 16-column block, one plane
    constexpr int STAGE = O::AP * A_PLANE + O::BP * B_PLANE;
    constexpr int NL = LW * 64;                  // loader threads
    constexpr int A_UPR = BK / 4;                // 16-byte units per A row
    constexpr int A_UNITS = BM * A_UPR;
    constexpr int A_IT = (A_UNITS + NL - 1) / NL;
    constexpr int B_UNITS = KS * O::BP * 64;
    constexpr int B_IT = (B_UNITS + NL - 1) / NL;
    static_assert(BK % 32 == 0 && BK <= 512 && BM % 16 == 0 && BM <= 64, "tile");
    static_assert(D >= 2 && D * STAGE <= 159 * 1024, "the LDS ring must fit one CU");

    __shared__ __attribute__((aligned(16))) char ring[D * STAGE];
    __shared__ uint32_t ready[D];
    __shared__ uint32_t consumed;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int fr = lane & 15;
    const int fg = lane >> 4;

    auto swz = [](int row) { return (row / RPW) & SWM; };
    auto chunk_off = [&](int row, int c) { return row * ROWB + ((c ^ swz(row)) << 4); };
    auto quad_off = [&](int row, int kq) {
        return row * ROWB + (((kq >> 1) ^ swz(row)) << 4) + ((kq & 1) << 3);
    };

    // one 16-column block per workgroup, XCD-aware numbering
    const int64_t nb = (int64_t)gridDim.x;
    int64_t bid = blockIdx.x;
    {
        const int64_t x = bid & 7, i = bid >> 3, q = nb >> 3, r = nb & 7;
        bid = x * q + (x < r ? x : r) + i;
    }
    const int64_t n0 = bid * 16;
    const int64_t M = p.M, N = p.N, K = p.K;
    const int64_t nk = (K + BK - 1) / BK;
    const int64_t KC = (K + 31) / 32;

    if (tid < D) ready[tid] = 0u;
    if (tid == 0) consumed = 0u;
    __syncthreads();
    if (nk == 0) return;

    const char *Ab = reinterpret_cast<const char *>(p.A);
    const char *Bb = reinterpret_cast<const char *>(p.B);
    const __amdgpu_buffer_rsrc_t rsrc_a = make_rsrc(Ab);
    const __amdgpu_buffer_rsrc_t rsrc_b = make_rsrc(Bb + (n0 / 16) * KC * O::BP * 1024);

    if (wave < LW) {
        // ---------------- loader waves ----------------
        u32x4 ra[R][A_IT], rb[R][B_IT];
        const int64_t last = nk - 1;
        auto load_stage = [&](int set, int64_t t) {
            const int64_t k0 = (t < last ? t : last) * BK;
#pragma unroll
            for (int it = 0; it < A_IT; ++it) {
                const int u = it * NL + tid;
                if (A_UNITS % NL != 0 && u >= A_UNITS) continue;
                const int row = u / A_UPR, c = u % A_UPR;
                const int64_t k = k0 + (int64_t)c * 4;
                const bool ok = row < M && k < K;
                ra[set][it] = bload(rsrc_a, ok ? (uint32_t)(((int64_t)row * p.lda + k) * 4) : kOOB);
            }
#pragma unroll
            for (int it = 0; it < B_IT; ++it) {
                const int u = it * NL + tid;
                if (B_UNITS % NL != 0 && u >= B_UNITS) continue;
                const int64_t kc = k0 / 32 + u / (O::BP * 64);
                const bool ok = kc < KC;
                rb[set][it] =
                    bload(rsrc_b, ok ? (uint32_t)(((k0 / 32) * O::BP * 64 + u) * 16) : kOOB);
            }
        };
        auto store_stage = [&](char *s, int set) {
            char *a0 = s, *a1 = s + A_PLANE, *b0 = s + O::AP * A_PLANE;
#pragma unroll
            for (int it = 0; it < A_IT; ++it) {
                const int u = it * NL + tid;
                if (A_UNITS % NL != 0 && u >= A_UNITS) continue;
                const int row = u / A_UPR, c = u % A_UPR;
                const f32x4 xf = __builtin_bit_cast(f32x4, ra[set][it]);
                const int off = quad_off(row, c);
                if constexpr (OP == OP_BASE) {
                    const u32x2 h = {cvt2_f16(xf.x, xf.y), cvt2_f16(xf.z, xf.w)};
                    *reinterpret_cast<u32x2 *>(a0 + off) = h;
                } else {
                    uint32_t h0, l0, h1, l1;
                    if constexpr (OP == OP_FULL) {
                        split2_f16(xf.x, xf.y, h0, l0);
                        split2_f16(xf.z, xf.w, h1, l1);
                    } else {
                        split2(xf.x, xf.y, h0, l0);
                        split2(xf.z, xf.w, h1, l1);
                    }
                    const u32x2 h = {h0, h1}, l = {l0, l1};
                    *reinterpret_cast<u32x2 *>(a0 + off) = h;
                    *reinterpret_cast<u32x2 *>(a1 + off) = l;
                }
            }
#pragma unroll
            for (int it = 0; it < B_IT; ++it) {
                const int u = it * NL + tid;
                if (B_UNITS % NL != 0 && u >= B_UNITS) continue;
                *reinterpret_cast<u32x4 *>(b0 + u * 16) = rb[set][it];
            }
        };
        // stage t sits in register set t % R and is reloaded with stage t + R
        // once stored (R stages of loads in flight per loader); every group
        // of R steps runs whole (loads included), so that each wait before a
        // store is for that set's loads alone
        auto step = [&](int set, int64_t t) {
            if (t < nk) {
                if (t >= D) spin_until_at_least(&consumed, (uint32_t)(t - D + 1));
                store_stage(ring + (t % D) * STAGE, set);
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
                if (lane == 0)
                    __hip_atomic_fetch_add(&ready[t % D], 1u, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_WORKGROUP);
            }
            load_stage(set, t + R);
        };
#pragma unroll
        for (int r = 0; r < R; ++r) {
            load_stage(r, r);
            __builtin_amdgcn_sched_barrier(0);
        }
        for (int64_t t = 0; t < nk; t += R) {
#pragma unroll
            for (int r = 0; r < R; ++r) step(r, t + r);
        }
        return;
    }

    // ---------------- the compute wave ----------------
    f32x4 acc[FM];
#pragma unroll
    for (int i = 0; i < FM; ++i) acc[i] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    // fragments of PF + 1 chunks: chunk k sits in buffer k % (PF + 1)
    constexpr int NBUF = PF + 1;
    static_assert(KS % NBUF == 0, "a stage holds whole turns of the fragment ring");
    u32x4 fa[NBUF][FM], fl[NBUF][FM], fb[NBUF], fbl[NBUF];
    auto read_chunk = [&](int buf, int64_t t, int ks) {
        const char *s = ring + (t % D) * STAGE;
        const char *a0 = s, *a1 = s + A_PLANE, *b0 = s + O::AP * A_PLANE;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const int off = chunk_off(i * 16 + fr, ks * 4 + fg);
            fa[buf][i] = *reinterpret_cast<const u32x4 *>(a0 + off);
            if (O::AP == 2) fl[buf][i] = *reinterpret_cast<const u32x4 *>(a1 + off);
        }
        const int off = ks * O::BP * 1024 + lane * 16;
        fb[buf] = *reinterpret_cast<const u32x4 *>(b0 + off);
        if (O::BP == 2) fbl[buf] = *reinterpret_cast<const u32x4 *>(b0 + off + 1024);
    };
    auto mma_chunk = [&](int buf) {
        const u32x4 bh = fb[buf];
        u32x4 bs;
        if constexpr (OP == OP_FULL)
            bs = __builtin_bit_cast(u32x4, __builtin_bit_cast(f16x8, bh) * (_Float16)0x1p-10f);
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            if constexpr (OP == OP_BASE) {
                acc[i] = mma<false>(bh, fa[buf][i], acc[i]);
            } else if constexpr (OP == OP_FULL) {
                acc[i] = mma<false>(bh, fa[buf][i], acc[i]);
                acc[i] = mma<false>(bs, fl[buf][i], acc[i]);
            } else {
                acc[i] = mma<true>(bh, fa[buf][i], acc[i]);
                acc[i] = mma<true>(fbl[buf], fa[buf][i], acc[i]);
                acc[i] = mma<true>(bh, fl[buf][i], acc[i]);
            }
        }
    };
    // Chunk k + PF is read while chunk k is multiplied out (a stage's
    // MFMAs are too short to cover an LDS read one chunk ahead); the first
    // read from stage t + 1 waits for that stage.  For the last stage the
    // reads ahead go to its own chunks again, complete and still in their
    // slot, so that no read sits under a branch and the wait before each
    // chunk's MFMAs is for that chunk's reads alone.  The stage goes back to
    // the loaders once the MFMAs of its last chunk have their operands;
    // every lane writes the same count.
    spin_until_at_least(&ready[0], (uint32_t)LW);
#pragma unroll
    for (int k = 0; k < PF; ++k) read_chunk(k, 0, k);
    for (int64_t t = 0; t < nk; ++t) {
        const int64_t tn = t + 1 < nk ? t + 1 : t;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int kk = ks + PF;
            if (kk < KS) {
                read_chunk(kk % NBUF, t, kk);
            } else {
                if (kk == KS)
                    spin_until_at_least(&ready[tn % D], (uint32_t)((tn / D + 1) * LW));
                read_chunk(kk % NBUF, tn, kk - KS);
            }
            mma_chunk(ks % NBUF);
        }
        __hip_atomic_store(&consumed, (uint32_t)(t + 1), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_WORKGROUP);
    }

    float *__restrict__ C = p.C;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int64_t m = i * 16 + fr;
        const int64_t n = n0 + 4 * fg;
        f32x4 v;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            if constexpr (OP == OP_BASE || OP == OP_FULL)
                v[t] = ldexpf(acc[i][t], -p.e);
            else
                v[t] = acc[i][t];
        }
        if (m < M && n < N) {
            float *cp = C + m * p.ldc + n;
            if (p.vecC && n + 4 <= N) {
                __builtin_nontemporal_store(v, reinterpret_cast<f32x4 *>(cp));
            } else {
                cp[0] = v.x;
                if (n + 1 < N) cp[1] = v.y;
                if (n + 2 < N) cp[2] = v.z;
                if (n + 3 < N) cp[3] = v.w;
            }
        }
    }
}

template <int OP, int BM, int BN, int BK>
bool vec_path_applies(const OpArgs &a)
{
    using O = OpT<OP>;
    const int64_t lim = 0x7fffffffLL;
    const int esz_a = O::A_I16 ? 2 : 4;
    const int upk = O::A_I16 ? 8 : 4;
    if (!a.vecA || a.K % upk != 0) return false;
    if (((int64_t)(BM - 1) * a.lda + a.K + BK) * esz_a >= lim) return false;
    if (O::B_ROWS) {
        if (!a.vecB || a.K % 8 != 0) return false;
        if (((int64_t)(BN - 1) * a.ldb + a.K + BK) * 2 >= lim) return false;
    }
    return true;
}

// The streamed narrow tiles: LDS ring depth, and per tile height the loader
// waves and their register sets (stages of loads in flight per loader).
#ifndef HEAL_OP_STREAM
#define HEAL_OP_STREAM 1
#endif
#ifndef HEAL_STREAM_D
#define HEAL_STREAM_D 4
#endif
#ifndef HEAL_STREAM16_LW
#define HEAL_STREAM16_LW 4
#endif
#ifndef HEAL_STREAM16_R
#define HEAL_STREAM16_R 2
#endif
#ifndef HEAL_STREAM32_LW
#define HEAL_STREAM32_LW 8
#endif
#ifndef HEAL_STREAM32_R
#define HEAL_STREAM32_R 4
#endif
#ifndef HEAL_STREAM64_LW
#define HEAL_STREAM64_LW 8
#endif
#ifndef HEAL_STREAM64_R
#define HEAL_STREAM64_R 4
#endif
#ifndef HEAL_STREAM16_BK
#define HEAL_STREAM16_BK 256
#endif
#ifndef HEAL_STREAM32_BK
#define HEAL_STREAM32_BK 128
#endif
#ifndef HEAL_STREAM64_BK
#define HEAL_STREAM64_BK 64
#endif
// chunks read ahead by the compute wave
#ifndef HEAL_STREAM16_PF
#define HEAL_STREAM16_PF 3
#endif
#ifndef HEAL_STREAM32_PF
#define HEAL_STREAM32_PF 3
#endif
#ifndef HEAL_STREAM64_PF
#define HEAL_STREAM64_PF 1
#endif

template <int OP, int BM, int BK, int PF, int LW, int R>
hipError_t launch_stream(const OpArgs &a, hipStream_t stream)
{
    const int64_t blocks = (a.N + 15) / 16;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL((gemm_op_stream_kernel<OP, BM, BK, HEAL_STREAM_D, LW, PF, R>),
                       dim3((unsigned)blocks), dim3((LW + 1) * 64), 0, stream, a);
    return hipGetLastError();
}

template <int OP, int BM, int BN, int WM, int WN, int NT, int BK, int R = 1>
hipError_t launch_cfg(const OpArgs &a, hipStream_t stream)
{
    const int64_t tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
    if (tiles > 0x7fffffffLL) return hipErrorInvalidValue;
    const unsigned gy = (unsigned)(a.batch < 65535 ? a.batch : 65535);
    const dim3 grid((unsigned)tiles, gy);
    if (vec_path_applies<OP, BM, BN, BK>(a))
        hipLaunchKernelGGL((gemm_op_kernel<OP, BM, BN, WM, WN, NT, BK, R, true>), grid, dim3(NT),
                           0, stream, a);
    else
        hipLaunchKernelGGL((gemm_op_kernel<OP, BM, BN, WM, WN, NT, BK, R, false>), grid, dim3(NT),
                           0, stream, a);
    return hipGetLastError();
}

// Instance configurations: BM, BN, WM, WN, threads, BK[, register sets].
// Threads beyond the (BM/WM)(BN/WN) compute waves only load and convert.
#ifndef HEAL_OP_LARGE_CFG
#define HEAL_OP_LARGE_CFG 128, 256, 64, 64, 512, 32
#endif
// 256 x 256 tiles, eight waves of 64 x 128 (128 accumulator VGPRs at two
// waves per SIMD).  HEAL-Full keeps two register sets (1.03x faster at
// 8192^3, 1.06x at 2048 x 14336 x 4096, despite 8 spilled VGPRs); Base and
// the pre-split product were no faster or slower with two.
#ifndef HEAL_OP_LARGE_FULL_CFG
#define HEAL_OP_LARGE_FULL_CFG 256, 256, 64, 128, 512, 32, 2
#endif
#ifndef HEAL_OP_LARGE_BASE_CFG
#define HEAL_OP_LARGE_BASE_CFG 256, 256, 64, 128, 512, 64
#endif
#ifndef HEAL_OP_LARGE_PRESPLIT_CFG
#define HEAL_OP_LARGE_PRESPLIT_CFG 256, 256, 64, 128, 512, 32
#endif
// Medium tiles keep two register sets: each stage's loads have a whole
// stage to arrive (at 4096 deep on 2048 x 1792, 1024 x 1024, 2048 x 2048
// and 512 x 4096 outputs: HEAL-Full 1.16-1.55x, HEAL-Base 1.7-1.9x, the
// pre-split product 1.23-1.33x faster than one set; 64-deep stages with
// two sets were within 10% either way).
#ifndef HEAL_OP_MEDIUM_CFG
#define HEAL_OP_MEDIUM_CFG 128, 128, 32, 64, 512, 32, 2
#endif
// M <= 64, wide N: 256-column tiles, four compute waves of 16..64 x 64
#ifndef HEAL_OP_SKINNY16_CFG
#define HEAL_OP_SKINNY16_CFG 16, 256, 16, 64, 256, 64
#endif
#ifndef HEAL_OP_SKINNY32_CFG
#define HEAL_OP_SKINNY32_CFG 32, 256, 32, 64, 256, 64
#endif
#ifndef HEAL_OP_SKINNY64_CFG
#define HEAL_OP_SKINNY64_CFG 64, 256, 64, 64, 256, 32
#endif
// M <= 64, narrow N (too few 256-column tiles to fill the chip): 16-column
// tiles, one compute wave and 7 or 15 more waves that load and convert, and
// two register sets (the stage's few MFMAs cannot hide a load: 1.1-1.4x
// faster than one set on 16..64 x 4096 x 4096).  Measured on those shapes,
// 512 threads beat 256 by 1.09-1.13x at 16 and 32 rows (HEAL-Full and the
// pre-split product), 1024 threads beat 256 by 1.09-1.15x at 64 rows.
#ifndef HEAL_OP_NARROW16_CFG
#define HEAL_OP_NARROW16_CFG 16, 16, 16, 16, 512, 256, 2
#endif
#ifndef HEAL_OP_NARROW32_CFG
#define HEAL_OP_NARROW32_CFG 32, 16, 32, 16, 512, 128, 2
#endif
#ifndef HEAL_OP_NARROW64_CFG
#define HEAL_OP_NARROW64_CFG 64, 16, 64, 16, 1024, 64, 2
#endif
// M <= 64, outputs between: 32-, 64- and 128-column tiles of 16-column
// compute waves (32-column ones for 128) and as many waves again that load
// and convert.  The tile width follows the bf16x3 skinny kernel's strips
// (the widest that still gives about one tile per CU at 64 rows, two at 16
// or 32 rows).  On 64 x 16032 x 4096 (one eighth of lm_head's columns)
// 64-column tiles of 512 threads ran HEAL-Full in 44.6 us, HEAL-Base in
// 34.8 us and the pre-split product in 54.5 us, against 116.8, 92.9 and
// 132.1 us for the streamed 16-column tiles (1002 of them, each
// converting all of A), 48.7 / 36.3 / 61.4 us with 256 threads and
// 64.4 / 44.8 / 90.4 us for 128-column tiles.
#ifndef HEAL_OP_MID32_16
#define HEAL_OP_MID32_16 16, 32, 16, 16, 256, 128, 2
#endif
#ifndef HEAL_OP_MID64_16
#define HEAL_OP_MID64_16 16, 64, 16, 16, 512, 128, 2
#endif
#ifndef HEAL_OP_MID128_16
#define HEAL_OP_MID128_16 16, 128, 16, 32, 512, 64, 2
#endif
#ifndef HEAL_OP_MID32_32
#define HEAL_OP_MID32_32 32, 32, 32, 16, 256, 128, 2
#endif
#ifndef HEAL_OP_MID64_32
#define HEAL_OP_MID64_32 32, 64, 32, 16, 512, 128, 2
#endif
#ifndef HEAL_OP_MID128_32
#define HEAL_OP_MID128_32 32, 128, 32, 32, 512, 64, 2
#endif
#ifndef HEAL_OP_MID32_64
#define HEAL_OP_MID32_64 64, 32, 64, 16, 256, 64, 2
#endif
#ifndef HEAL_OP_MID64_64
#define HEAL_OP_MID64_64 64, 64, 64, 16, 512, 64, 2
#endif
#ifndef HEAL_OP_MID128_64
#define HEAL_OP_MID128_64 64, 128, 64, 32, 512, 64, 2
#endif

// The same with 224-column tiles (eight waves of 64 x 112), for shapes whose
// 256-column tiles leave the last round of workgroups part-empty.
#ifndef HEAL_OP_LARGE_FULL_N224_CFG
#define HEAL_OP_LARGE_FULL_N224_CFG 256, 224, 64, 112, 512, 32, 2
#endif
#ifndef HEAL_OP_LARGE_BASE_N224_CFG
#define HEAL_OP_LARGE_BASE_N224_CFG 256, 224, 64, 112, 512, 64
#endif
#ifndef HEAL_OP_LARGE_PRESPLIT_N224_CFG
#define HEAL_OP_LARGE_PRESPLIT_N224_CFG 256, 224, 64, 112, 512, 32
#endif

// Compute units of the current device, queried once per device.
int device_cus()
{
    constexpr int kMaxDev = 64;
    static std::atomic<int> cache[kMaxDev];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDev) return 256;
    int n = cache[dev].load(std::memory_order_relaxed);
    if (n > 0) return n;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n <= 0)
        n = 256;
    cache[dev].store(n, std::memory_order_relaxed);
    return n;
}

// Relative time of a grid of 256 x bn tiles: the 256 x 256 instances hold
// one workgroup per CU (LDS), so the grid runs in ceil(workgroups / CUs)
// rounds, each as long as one tile, which grows with bn at fixed K.
int64_t large_cost(const OpArgs &a, int bn, int cus)
{
    const int64_t wgs = ((a.M + 255) / 256) * ((a.N + bn - 1) / bn) * a.batch;
    return (wgs + cus - 1) / cus * bn;
}

template <int OP>
hipError_t launch_large(const OpArgs &a, hipStream_t stream)
{
    if constexpr (OP == OP_SCORES) {
        return launch_cfg<OP, HEAL_OP_LARGE_CFG>(a, stream);
    } else {
        // the hand-scheduled kernel wherever it applies (it beats the generic
        // 224-column tiles also where those need fewer rounds)
        const int cus = device_cus();
        const bool n224 = HEAL_OP_N224 && large_cost(a, 224, cus) < large_cost(a, 256, cus);
        // 224-column tiles where they need fewer rounds (prefill_up: HEAL-Full
        // 1.01x, pre-split 1.02x; HEAL-Base 0.99x, so it keeps 256)
        if (HEAL_OP_LARGE8 && op8_applies<OP>(a))
            return n224 && HEAL_OP8_N224 && OP != OP_BASE ? launch_op8<OP, 224>(a, stream)
                                                          : launch_op8<OP, 256>(a, stream);
        if constexpr (OP == OP_FULL)
            return n224 ? launch_cfg<OP, HEAL_OP_LARGE_FULL_N224_CFG>(a, stream)
                        : launch_cfg<OP, HEAL_OP_LARGE_FULL_CFG>(a, stream);
        else if constexpr (OP == OP_BASE)
            return n224 ? launch_cfg<OP, HEAL_OP_LARGE_BASE_N224_CFG>(a, stream)
                        : launch_cfg<OP, HEAL_OP_LARGE_BASE_CFG>(a, stream);
        else
            return n224 ? launch_cfg<OP, HEAL_OP_LARGE_PRESPLIT_N224_CFG>(a, stream)
                        : launch_cfg<OP, HEAL_OP_LARGE_PRESPLIT_CFG>(a, stream);
    }
}

// HEAL-Full at M <= 64, wide N: eight waves of 64 x 32 (measured faster than
// four of 64 x 64: the A split is shared by twice the threads)
#ifndef HEAL_OP_SKINNY64_FULL_CFG
#define HEAL_OP_SKINNY64_FULL_CFG 64, 256, 64, 32, 512, 32
#endif

template <int OP>
hipError_t launch_op(int instance, const OpArgs &a, hipStream_t stream)
{
    if constexpr (OP == OP_SCORES) {
        if (HEAL_PANEL && instance != HEAL_INSTANCE_SKINNY && scores_panel_applies(a))
            return launch_scores_panel(a, stream);
    }
    switch (instance) {
    case HEAL_INSTANCE_LARGE: return launch_large<OP>(a, stream);
    case HEAL_INSTANCE_MEDIUM: return launch_cfg<OP, HEAL_OP_MEDIUM_CFG>(a, stream);
    case HEAL_INSTANCE_SKINNY: {
        const int w = skinny_strip_width(a.N, a.M);
        const bool wide = w == 256;
        if (w == 32 || w == 64 || w == 128) {
            if (a.M <= 16)
                return w == 32   ? launch_cfg<OP, HEAL_OP_MID32_16>(a, stream)
                       : w == 64 ? launch_cfg<OP, HEAL_OP_MID64_16>(a, stream)
                                 : launch_cfg<OP, HEAL_OP_MID128_16>(a, stream);
            if (a.M <= 32)
                return w == 32   ? launch_cfg<OP, HEAL_OP_MID32_32>(a, stream)
                       : w == 64 ? launch_cfg<OP, HEAL_OP_MID64_32>(a, stream)
                                 : launch_cfg<OP, HEAL_OP_MID128_32>(a, stream);
            return w == 32   ? launch_cfg<OP, HEAL_OP_MID32_64>(a, stream)
                   : w == 64 ? launch_cfg<OP, HEAL_OP_MID64_64>(a, stream)
                             : launch_cfg<OP, HEAL_OP_MID128_64>(a, stream);
        }
        if constexpr (OP != OP_SCORES) {
            if (!wide && HEAL_OP_STREAM) {
                if (a.M <= 16 && vec_path_applies<OP, 16, 16, HEAL_STREAM16_BK>(a))
                    return launch_stream<OP, 16, HEAL_STREAM16_BK, HEAL_STREAM16_PF, HEAL_STREAM16_LW,
                                         HEAL_STREAM16_R>(a, stream);
                if (a.M > 16 && a.M <= 32 && vec_path_applies<OP, 32, 16, HEAL_STREAM32_BK>(a))
                    return launch_stream<OP, 32, HEAL_STREAM32_BK, HEAL_STREAM32_PF, HEAL_STREAM32_LW,
                                         HEAL_STREAM32_R>(a, stream);
                if (a.M > 32 && a.M <= 64 && vec_path_applies<OP, 64, 16, HEAL_STREAM64_BK>(a))
                    return launch_stream<OP, 64, HEAL_STREAM64_BK, HEAL_STREAM64_PF, HEAL_STREAM64_LW,
                                         HEAL_STREAM64_R>(a, stream);
            }
        }
        if (a.M <= 16)
            return wide ? launch_cfg<OP, HEAL_OP_SKINNY16_CFG>(a, stream)
                        : launch_cfg<OP, HEAL_OP_NARROW16_CFG>(a, stream);
        if (a.M <= 32)
            return wide ? launch_cfg<OP, HEAL_OP_SKINNY32_CFG>(a, stream)
                        : launch_cfg<OP, HEAL_OP_NARROW32_CFG>(a, stream);
        if (!wide) return launch_cfg<OP, HEAL_OP_NARROW64_CFG>(a, stream);
        if constexpr (OP == OP_FULL) return launch_cfg<OP, HEAL_OP_SKINNY64_FULL_CFG>(a, stream);
        return launch_cfg<OP, HEAL_OP_SKINNY64_CFG>(a, stream);
    }
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_gemm_op(int op, int instance, const OpArgs &a, hipStream_t stream)
{
    if (instance == HEAL_INSTANCE_AUTO)
        instance = a.M <= 64 ? HEAL_INSTANCE_SKINNY
                   : a.M * a.N <= (int64_t)2048 * 2048 ? HEAL_INSTANCE_MEDIUM
                                                       : HEAL_INSTANCE_LARGE;
    switch (op) {
    case OP_BASE: return launch_op<OP_BASE>(instance, a, stream);
    case OP_FULL: return launch_op<OP_FULL>(instance, a, stream);
    case OP_SCORES: return launch_op<OP_SCORES>(instance, a, stream);
    case OP_PRESPLIT: return launch_op<OP_PRESPLIT>(instance, a, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace heal
