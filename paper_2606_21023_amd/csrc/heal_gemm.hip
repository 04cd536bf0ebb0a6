// The compensated bf16x3 GEMM kernels for gfx950 (MI355X).
//
// HEAL Section 4 (GEMM paragraph and its displayed expansion) recovers the
// bits a 16-bit cast drops by adding residual products on the 16-bit matrix
// units, accumulating in FP32.  Here both FP32 operands are split into bf16
// (hi, lo) and C = hiA*hiB + hiA*loB + loA*hiB.
//
// Data path of one workgroup (one BM x BN output tile, batch entry b):
//   HBM --16-byte loads--> VGPRs --split (v_cvt_pk_bf16_f32)--> LDS planes
//   {A_hi, A_lo, B_hi, B_lo}, k-contiguous, XOR-swizzled, double-buffered
//   --ds_read_b128--> MFMA fragments --3x v_mfma_f32_16x16x32_bf16--> FP32
//   accumulators --> FP32 C (16-byte stores).
// Each FP32 element is split once per workgroup that stages it.
//
// Reduction order (identical in every instance, so results are bitwise equal
// across runs, instances and M): for each output element, K is walked in
// 32-deep chunks in ascending order; each chunk adds hiA*hiB, then hiA*loB,
// then loA*hiB into a single FP32 accumulator; the K tail and out-of-range
// rows/columns are zero-filled.  No split-K, no atomics.
//
// MFMA operand roles: the B fragment is the MFMA's first source (16 rows =
// 16 output columns n) and the A fragment the second (16 columns = output
// rows m), so each lane's four accumulators are C[m][n..n+3], four
// consecutive FP32 of one output row, written with one 16-byte store.
#include <type_traits>

#include "heal.h"
#include "heal_device.h"
#include "heal_internal.h"

namespace heal {

// Batch entries per workgroup of a strided-batched launch (the attention
// score product: 32 heads of 2048 x 2048 x 128 ran 1.09x faster with two
// than with one; four or more were slower again).
#ifndef HEAL_TILE_BATCH_PER_WG
#define HEAL_TILE_BATCH_PER_WG 2
#endif

namespace {

constexpr int kChunk = 32;  // K depth of one bf16 MFMA: the unit of the reduction order

// Steady-state interleave: the split of the next stage starts after
// SPLIT_AT/8 of the current stage's MFMA chunks, giving its global loads that
// long to arrive.
#ifndef HEAL_SCHED_SPLIT_AT
#define HEAL_SCHED_SPLIT_AT 4
#endif
// The same with the register ring (loads two stages ahead), and the fewest
// full stages for which the ring runs: on 4096-deep medium tiles the ring
// with the split from 2/8 of the stage was 1.17-1.32x faster than one set
// (4/8: 1.10-1.27x); on 256-deep ones (4 stages) it was 4-7% slower.
#ifndef HEAL_SCHED_SPLIT_AT_RING
#define HEAL_SCHED_SPLIT_AT_RING 2
#endif
#ifndef HEAL_RING_MIN_STAGES
#define HEAL_RING_MIN_STAGES 8
#endif
// Epilogue: pairs of 16-column blocks of a wave stored as whole 128-byte
// lines, non-temporal.  Off: in the medium tile it costs two spilled VGPRs
// (1024 x 1024 x 4096 4% slower; 2048 x 2048 x 256 10% faster, 2048 x 1792
// x 4096 unchanged).
#ifndef HEAL_TILE_C_LINES
#define HEAL_TILE_C_LINES 0
#endif
// Instance configurations: BM, BN, BK, WM, WN, threads[, register sets].
// The medium tile stages 64-deep: two MFMA chunks per barrier and per round
// of loads (at 4096 deep 1.30-1.34x faster than 32-deep stages on 2048 x
// 1792, 2048 x 2048, 1024 x 1024 and 512 x 4096 outputs; 1.02-1.05x at 256
// deep).
#ifndef HEAL_MEDIUM_CFG
#define HEAL_MEDIUM_CFG 128, 128, 64, 32, 64, 512, 2
#endif
#ifndef HEAL_SKINNY16_CFG
#define HEAL_SKINNY16_CFG 16, 64, 64, 16, 16, 256
#endif
#ifndef HEAL_SKINNY32_CFG
#define HEAL_SKINNY32_CFG 32, 64, 64, 32, 16, 256
#endif
#ifndef HEAL_SKINNY64_CFG
#define HEAL_SKINNY64_CFG 64, 64, 64, 64, 16, 256
#endif
#ifndef HEAL_LARGE_CFG
#define HEAL_LARGE_CFG 256, 256, 32, 64, 128, 512
#endif

template <int BM, int BN, int BK, int WM, int WN, int NT>
struct Tile {
    static_assert(BK % kChunk == 0, "stage depth must be whole MFMA chunks");
    static_assert(BM % WM == 0 && BN % WN == 0 && WM % 16 == 0 && WN % 16 == 0, "wave tiling");
    static constexpr int WAVES_M = BM / WM;
    static constexpr int CWAVES = WAVES_M * (BN / WN);  // waves that compute
    static_assert(CWAVES * 64 <= NT && NT % 64 == 0, "compute waves exceed the workgroup");
    static constexpr int ROWB = BK * 2;                  // bytes per LDS row of one plane
    static constexpr int NCH = BK / 8;                   // 16-byte chunks per row
    static constexpr int RPW = BK >= 64 ? 1 : 64 / BK;   // rows sharing one 128-byte window
    static constexpr int SWM = (NCH < 8 ? NCH : 8) - 1;  // XOR swizzle mask on the chunk index
    static constexpr int A_PLANE = BM * ROWB;
    static constexpr int B_PLANE = BN * ROWB;
    static constexpr int STAGE = 2 * A_PLANE + 2 * B_PLANE;
    static constexpr int KQ = BK / 4;                    // 4-element quads per row per stage
    static constexpr int QA = BM * KQ;                   // A quads per stage
    static constexpr int QBT = BN * KQ;                  // B quads per stage, B stored N x K
    static constexpr int BB = KQ * (BN / 4);             // 4x4 blocks per stage, B stored K x N
    static constexpr int ITA = (QA + NT - 1) / NT;
    static constexpr int ITBT = (QBT + NT - 1) / NT;
    static constexpr int ITB = (BB + NT - 1) / NT;

    static constexpr int LKQ = KQ == 8 ? 3 : KQ == 16 ? 4 : KQ == 32 ? 5 : -1;
    static_assert(LKQ > 0, "stage depth must be 32, 64 or 128");
    // LDS row of B column n.  With 64-byte rows the two halves of each
    // 8-row group trade their odd/even rows when bit 2 of n is set, so the
    // register-transposed B writes of one instruction (all lanes writing the
    // same column offset nn) still land on both row parities, i.e. on all
    // 32 banks.  A read pass covers whole 8-row groups, so reads are
    // unaffected.
    static __device__ __forceinline__ int brow(int n)
    {
        return ROWB == 64 ? n ^ ((n >> 2) & 1) : n;
    }
    // byte offset of 4 consecutive k (k = 4*kq) of row `row` in a plane
    static __device__ __forceinline__ int quad_off(int row, int kq)
    {
        return row * ROWB + ((((kq >> 1) ^ ((row / RPW) & SWM))) << 4) + ((kq & 1) << 3);
    }
    // byte offset of the 16-byte chunk `c` (8 consecutive k) of row `row`
    static __device__ __forceinline__ int chunk_off(int row, int c)
    {
        return row * ROWB + ((c ^ ((row / RPW) & SWM)) << 4);
    }
};

// Elements (r, c .. c+3) of a row-major matrix with nr x nc valid entries,
// zero outside (edge tiles and the K tail).  VEC: the row is 16-byte aligned
// and nc % 4 == 0, so a quad is either wholly inside or wholly outside.
template <bool VEC>
__device__ __forceinline__ f32x4 load_quad_checked(const float *__restrict__ row_ptr, bool row_ok,
                                                   int64_t c, int64_t nc)
{
    f32x4 v = {0.0f, 0.0f, 0.0f, 0.0f};
    if (VEC) {
        if (row_ok && c < nc) v = *reinterpret_cast<const f32x4 *>(row_ptr);
    } else if (row_ok) {
        if (c < nc) v.x = row_ptr[0];
        if (c + 1 < nc) v.y = row_ptr[1];
        if (c + 2 < nc) v.z = row_ptr[2];
        if (c + 3 < nc) v.w = row_ptr[3];
    }
    return v;
}

__device__ __forceinline__ void store_pair(char *plane, int off, uint32_t a, uint32_t b)
{
    u32x2 v = {a, b};
    *reinterpret_cast<u32x2 *>(plane + off) = v;
}

// RS: register sets of staged operands.  With two (tiles whose waves all
// multiply), each stage's loads are issued two stages before their split;
// with one, half a stage before.
template <int BM, int BN, int BK, int WM, int WN, int NT, int RS, bool TRANS_B, bool ALPHA, bool VEC>
__global__ void __launch_bounds__(NT)
gemm_bf16x3_kernel(GemmArgs p)
{
    using T = Tile<BM, BN, BK, WM, WN, NT>;
    static_assert(RS == 1 || RS == 2, "register sets");
    constexpr bool RING = RS == 2 && T::CWAVES * 64 == NT;
    // Work distribution of the loads (see the load lambdas below).
    constexpr int A_ROWS_PER_PASS = NT / T::KQ;          // A rows covered by one pass of NT threads
    constexpr int BT_ROWS_PER_PASS = NT / T::KQ;         // same for B stored N x K
    // B stored K x N: each thread loads a 4 (k) x 4 (n) block, which it
    // transposes in registers.  Lane bits 1..LKQ pick the k-quad, lane bit 0
    // and the remaining lane and wave bits the 4-column group, so that one
    // write instruction's 16-lane passes cover all 16 eight-byte bank slots
    // and one load instruction reads whole 128-byte row segments.
    constexpr int B_NQ_PER_PASS = NT / T::KQ;            // 4-column groups per pass
    static_assert(NT % T::KQ == 0 && T::KQ <= 32, "load distribution");
    static_assert((A_ROWS_PER_PASS / T::RPW) % (T::SWM + 1) == 0 || T::ITA == 1,
                  "swizzle must repeat across A passes");
    static_assert((BT_ROWS_PER_PASS / T::RPW) % (T::SWM + 1) == 0 || T::ITBT == 1,
                  "swizzle must repeat across B passes");
    static_assert((16 / T::RPW) % (T::SWM + 1) == 0, "swizzle must repeat every 16 rows");

    // Two LDS stage buffers as distinct objects, so the compiler can tell the
    // split's writes into one from the fragment reads of the other and
    // interleave them.
    static_assert(2 * T::STAGE <= 160 * 1024, "two LDS stages must fit the 160 KB of a CU");
    __shared__ __attribute__((aligned(16))) char smem0[T::STAGE];
    __shared__ __attribute__((aligned(16))) char smem1[T::STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;

    // ---- tile coordinates: XCD-aware, grouped along M --------------------
    // Workgroups are dealt to the 8 XCDs round-robin; renumber so each XCD
    // owns a contiguous range of tiles, then walk tiles in groups of GM
    // tile-rows so that concurrently running tiles share A and B panels in
    // that XCD's L2.
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
    // interior: whole tile in range, 16-byte aligned rows, and every byte
    // offset of a tile (A, B stored N x K) or of a stage (B stored K x N)
    // below 2^31, so the fast path can use buffer loads with 32-bit offsets.
    const bool interior = VEC && m0 + BM <= M && n0 + BN <= N &&
                          (int64_t)BM * p.lda * 4 < 0x7fffffffLL &&
                          (int64_t)(TRANS_B ? BN : BK) * p.ldb * 4 < 0x7fffffffLL;

    const int wm = wave % T::WAVES_M;
    const int wn = wave / T::WAVES_M;
    const bool computes = T::CWAVES * 64 == NT || wave < T::CWAVES;
    const int fr = lane & 15;   // fragment row (n for B, m for A) within a 16-block
    const int fg = lane >> 4;   // fragment k-group: k = 8*fg .. 8*fg+7 of the chunk

    // per-thread load coordinates (fixed for the whole tile)
    const int a_row = tid / T::KQ;                 // + pass * A_ROWS_PER_PASS
    const int a_kq = tid % T::KQ;
    const int b_kq = (lane >> 1) & (T::KQ - 1);   // B stored K x N
    const int b_nq = (lane & 1) | ((lane >> (1 + T::LKQ)) << 1) | (wave << (6 - T::LKQ));
                                                   // + pass * B_NQ_PER_PASS
    const int a_st = T::quad_off(a_row, a_kq);     // LDS store offsets
    const int bt_st = a_st;                        // B stored N x K uses the A pattern

    for (int64_t b = blockIdx.y; b < p.batch; b += gridDim.y) {
        const float *__restrict__ A = p.A + b * p.strideA;
        const float *__restrict__ B = p.B + b * p.strideB;
        float *__restrict__ C = p.C + b * p.strideC;
        const float *__restrict__ pa = A + (m0 + a_row) * p.lda + 4 * a_kq;
        const float *__restrict__ pb = TRANS_B ? B + (n0 + a_row) * p.ldb + 4 * a_kq
                                               : B + (int64_t)(4 * b_kq) * p.ldb + n0 + 4 * b_nq;

        f32x4 acc[WN / 16][WM / 16];
#pragma unroll
        for (int j = 0; j < WN / 16; ++j)
#pragma unroll
            for (int i = 0; i < WM / 16; ++i) acc[j][i] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

        f32x4 ra[RS][T::ITA];
        f32x4 rb[RS][TRANS_B ? T::ITBT : T::ITB][TRANS_B ? 1 : 4];

        // Full stage of an interior tile: buffer loads, one 32-bit VGPR offset
        // per operand and thread; stage and pass offsets are scalar.
        constexpr int kRsrcFlags = 0x00020000;   // raw buffer, 32-bit data format
        const __amdgpu_buffer_rsrc_t rsrc_a = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<float *>(A + m0 * p.lda), (short)0, 0x7fffffff, kRsrcFlags);
        const int voff_a = (a_row * (int)p.lda + 4 * a_kq) * 4;
        const int voff_b = TRANS_B ? (a_row * (int)p.ldb + 4 * a_kq) * 4
                                   : (4 * b_kq * (int)p.ldb + 4 * b_nq) * 4;
        // One pass `it` of A, or of B, of a full stage into register set `set`.
        auto load_a_fast = [&](int set, int it, int64_t k0) {
            if (T::QA % NT == 0 || it * NT + tid < T::QA)
                ra[set][it] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                    rsrc_a, voff_a, (int)(k0 * 4) + it * A_ROWS_PER_PASS * (int)p.lda * 4, 0));
        };
        auto load_b_fast = [&](int set, int it, int64_t k0) {
            if (TRANS_B) {
                const __amdgpu_buffer_rsrc_t rsrc_b = __builtin_amdgcn_make_buffer_rsrc(
                    const_cast<float *>(B + n0 * p.ldb), (short)0, 0x7fffffff, kRsrcFlags);
                if (T::QBT % NT == 0 || it * NT + tid < T::QBT)
                    rb[set][it][0] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                        rsrc_b, voff_b, (int)(k0 * 4) + it * BT_ROWS_PER_PASS * (int)p.ldb * 4, 0));
            } else {
                const __amdgpu_buffer_rsrc_t rsrc_b = __builtin_amdgcn_make_buffer_rsrc(
                    const_cast<float *>(B + k0 * p.ldb + n0), (short)0, 0x7fffffff, kRsrcFlags);
                if ((BN / 4) % B_NQ_PER_PASS == 0 || b_nq + it * B_NQ_PER_PASS < BN / 4)
#pragma unroll
                    for (int kk = 0; kk < 4; ++kk)
                        rb[set][it][kk] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                            rsrc_b, voff_b, kk * (int)p.ldb * 4 + it * B_NQ_PER_PASS * 16, 0));
            }
        };
        auto load_stage_fast = [&](int64_t k0, int set) {
#pragma unroll
            for (int it = 0; it < T::ITA; ++it) load_a_fast(set, it, k0);
#pragma unroll
            for (int it = 0; it < (TRANS_B ? T::ITBT : T::ITB); ++it) load_b_fast(set, it, k0);
        };

        // Any stage: element-wise bounds checks, zero fill outside.
        auto load_stage_checked = [&](int64_t k0) {
#pragma unroll
            for (int it = 0; it < T::ITA; ++it)
                if (T::QA % NT == 0 || it * NT + tid < T::QA) {
                    const int64_t r = it * A_ROWS_PER_PASS;
                    ra[0][it] = load_quad_checked<VEC>(pa + r * p.lda + k0, m0 + a_row + r < M,
                                                  k0 + 4 * a_kq, K);
                }
            if (TRANS_B) {
#pragma unroll
                for (int it = 0; it < T::ITBT; ++it)
                    if (T::QBT % NT == 0 || it * NT + tid < T::QBT) {
                        const int64_t r = it * BT_ROWS_PER_PASS;
                        rb[0][it][0] = load_quad_checked<VEC>(pb + r * p.ldb + k0, n0 + a_row + r < N,
                                                         k0 + 4 * a_kq, K);
                    }
            } else {
#pragma unroll
                for (int it = 0; it < T::ITB; ++it)
                    if ((BN / 4) % B_NQ_PER_PASS == 0 || b_nq + it * B_NQ_PER_PASS < BN / 4)
#pragma unroll
                        for (int kk = 0; kk < 4; ++kk) {
                            const int64_t kr = k0 + 4 * b_kq + kk;
                            rb[0][it][kk] = load_quad_checked<VEC>(
                                pb + (k0 + kk) * p.ldb + 4 * it * B_NQ_PER_PASS, kr < K,
                                n0 + 4 * (b_nq + it * B_NQ_PER_PASS), N);
                        }
            }
        };

        // Split units: one 4-element quad (two split2 calls, two 8-byte LDS
        // writes per plane pair) of this thread's staged data.
        constexpr int NU = T::ITA + (TRANS_B ? T::ITBT : 4 * T::ITB);
        auto store_unit = [&](char *s, const int u, const int set) {
            char *a_hi = s, *a_lo = s + T::A_PLANE;
            char *b_hi = s + 2 * T::A_PLANE, *b_lo = b_hi + T::B_PLANE;
            uint32_t h0, l0, h1, l1;
            if (u < T::ITA) {
                const int it = u;
                if (T::QA % NT == 0 || it * NT + tid < T::QA) {
                    split2(ra[set][it].x, ra[set][it].y, h0, l0);
                    split2(ra[set][it].z, ra[set][it].w, h1, l1);
                    const int off = a_st + it * A_ROWS_PER_PASS * T::ROWB;
                    store_pair(a_hi, off, h0, h1);
                    store_pair(a_lo, off, l0, l1);
                }
            } else if (TRANS_B) {
                const int it = u - T::ITA;
                if (T::QBT % NT == 0 || it * NT + tid < T::QBT) {
                    split2(rb[set][it][0].x, rb[set][it][0].y, h0, l0);
                    split2(rb[set][it][0].z, rb[set][it][0].w, h1, l1);
                    const int off = bt_st + it * BT_ROWS_PER_PASS * T::ROWB;
                    store_pair(b_hi, off, h0, h1);
                    store_pair(b_lo, off, l0, l1);
                }
            } else {
                // register transpose: column nn of the 4x4 block is 4 consecutive k
                const int it = (u - T::ITA) / 4, nn = (u - T::ITA) % 4;
                if ((BN / 4) % B_NQ_PER_PASS == 0 || b_nq + it * B_NQ_PER_PASS < BN / 4) {
                    split2(rb[set][it][0][nn], rb[set][it][1][nn], h0, l0);
                    split2(rb[set][it][2][nn], rb[set][it][3][nn], h1, l1);
                    const int off = T::quad_off(T::brow(4 * (b_nq + it * B_NQ_PER_PASS) + nn), b_kq);
                    store_pair(b_hi, off, h0, h1);
                    store_pair(b_lo, off, l0, l1);
                }
            }
        };

        auto store_stage = [&](char *s, int set) {
#pragma unroll
            for (int u = 0; u < NU; ++u) store_unit(s, u, set);
        };
        // Ring: reload the registers of unit u of `set` with the stage at
        // k0 once the unit is split (B stored K x N: a 4x4 block's four rows
        // after its last column).
        auto reload_unit = [&](int u, int set, int64_t k0) {
            if (u < T::ITA) {
                load_a_fast(set, u, k0);
            } else if (TRANS_B) {
                load_b_fast(set, u - T::ITA, k0);
            } else if ((u - T::ITA) % 4 == 3) {
                load_b_fast(set, (u - T::ITA) / 4, k0);
            }
        };

        // One steady-state stage of an interior tile, software-interleaved:
        // the stage's MFMAs are cut into chunks (one 16-column block of B and
        // one 32-deep k step each), and the split of the next stage's data is
        // spread over the later chunks, so that VALU work issues while the
        // matrix cores run.  Scheduling barriers keep the chunks apart.
        // k_next: with one register set, the stage loaded now and split into
        // `nxt` later in this stage; with the ring, the stage that reloads
        // `set` after its split (set holds the stage split into `nxt`).
        auto stage_fast = [&](const char *cur, char *nxt, int set, int64_t k_next, auto ring_tag) {
            constexpr bool R2 = decltype(ring_tag)::value;
            if (!R2) load_stage_fast(k_next, 0);
            const char *a_hi = cur, *a_lo = cur + T::A_PLANE;
            const char *b_hi = cur + 2 * T::A_PLANE, *b_lo = b_hi + T::B_PLANE;
            constexpr int NJ = WN / 16, KS = BK / kChunk, NC = NJ * KS;
            constexpr int C0s = NC * (R2 ? HEAL_SCHED_SPLIT_AT_RING : HEAL_SCHED_SPLIT_AT) / 8;
            constexpr int C0 = C0s < NC ? C0s : NC - 1;  // first chunk that splits
            bf16x8 ah[WM / 16], al[WM / 16], bh[2], bl[2];
            auto read_b = [&](int c, int slot) {
                const int off = T::chunk_off(TRANS_B ? wn * WN + fr : T::brow(wn * WN + fr),
                                             (c / NJ) * 4 + fg) + (c % NJ) * 16 * T::ROWB;
                bh[slot] = *reinterpret_cast<const bf16x8 *>(b_hi + off);
                bl[slot] = *reinterpret_cast<const bf16x8 *>(b_lo + off);
            };
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                const int ks = c / NJ, j = c % NJ;
                if (j == 0) {
                    const int a_off = T::chunk_off(wm * WM + fr, ks * 4 + fg);
#pragma unroll
                    for (int i = 0; i < WM / 16; ++i) {
                        ah[i] = *reinterpret_cast<const bf16x8 *>(a_hi + a_off + i * 16 * T::ROWB);
                        al[i] = *reinterpret_cast<const bf16x8 *>(a_lo + a_off + i * 16 * T::ROWB);
                    }
                }
                if (c == 0) read_b(0, 0);
                if (c + 1 < NC) read_b(c + 1, (c + 1) & 1);
                const int sl = c & 1;
#pragma unroll
                for (int i = 0; i < WM / 16; ++i)
                    acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bh[sl], ah[i], acc[j][i], 0, 0, 0);
#pragma unroll
                for (int i = 0; i < WM / 16; ++i)
                    acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bl[sl], ah[i], acc[j][i], 0, 0, 0);
#pragma unroll
                for (int i = 0; i < WM / 16; ++i)
                    acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bh[sl], al[i], acc[j][i], 0, 0, 0);
#pragma unroll
                for (int u = 0; u < NU; ++u)
                    if (C0 + (u * (NC - C0)) / NU == c) {
                        store_unit(nxt, u, R2 ? set : 0);
                        if (R2) reload_unit(u, set, k_next);
                    }
                __builtin_amdgcn_sched_barrier(0);
            }
        };

        auto compute_stage = [&](const char *s) {
            const char *a_hi = s, *a_lo = s + T::A_PLANE;
            const char *b_hi = s + 2 * T::A_PLANE, *b_lo = b_hi + T::B_PLANE;
#pragma unroll
            for (int ks = 0; ks < BK / kChunk; ++ks) {
                const int c = ks * 4 + fg;
                const int a_off = T::chunk_off(wm * WM + fr, c);
                const int b_off = T::chunk_off(TRANS_B ? wn * WN + fr : T::brow(wn * WN + fr), c);
                bf16x8 ah[WM / 16], al[WM / 16];
#pragma unroll
                for (int i = 0; i < WM / 16; ++i) {
                    ah[i] = *reinterpret_cast<const bf16x8 *>(a_hi + a_off + i * 16 * T::ROWB);
                    al[i] = *reinterpret_cast<const bf16x8 *>(a_lo + a_off + i * 16 * T::ROWB);
                }
#pragma unroll
                for (int j = 0; j < WN / 16; ++j) {
                    const bf16x8 bh = *reinterpret_cast<const bf16x8 *>(b_hi + b_off + j * 16 * T::ROWB);
                    const bf16x8 bl = *reinterpret_cast<const bf16x8 *>(b_lo + b_off + j * 16 * T::ROWB);
#pragma unroll
                    for (int i = 0; i < WM / 16; ++i)
                        acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bh, ah[i], acc[j][i], 0, 0, 0);
#pragma unroll
                    for (int i = 0; i < WM / 16; ++i)
                        acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bl, ah[i], acc[j][i], 0, 0, 0);
#pragma unroll
                    for (int i = 0; i < WM / 16; ++i)
                        acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bh, al[i], acc[j][i], 0, 0, 0);
                }
            }
        };

        // Main loop, one barrier per stage: while the MFMAs consume stage kt
        // from one LDS buffer, stage kt+1 is split into the other.  Its loads
        // were issued at the start of stage kt (one register set), or during
        // stage kt-2 (the ring: set 1 holds stage kt+1 and set 0 stage kt+2
        // at the top of each trip; each set is reloaded three stages ahead,
        // clamped to the last full stage, as soon as it is split).
        const int64_t nk_full = K / BK;  // stages without a K tail
        const bool ring = RING && VEC && interior && nk_full >= HEAL_RING_MIN_STAGES;
        using one_set = std::integral_constant<bool, false>;
        using two_sets = std::integral_constant<bool, RING>;
        int64_t kt = 0;
        if (nk > 0) {
            if (VEC && interior && BK <= K) {
                load_stage_fast(0, 0);
                if (ring) load_stage_fast(BK, RS - 1);
            } else {
                load_stage_checked(0);
            }
            store_stage(smem0, 0);
            if (ring) load_stage_fast(2 * BK, 0);
            __syncthreads();
        }
        if (VEC && interior) {
            // two stages per trip so that each buffer is a compile-time choice
            const int64_t last = (nk_full - 1) * BK;
            for (; kt + 2 < nk_full; kt += 2) {
                if (RING && ring) {
                    const int64_t k3 = (kt + 3) * BK, k4 = (kt + 4) * BK;
                    stage_fast(smem0, smem1, RS - 1, k3 < last ? k3 : last, two_sets{});
                    __syncthreads();
                    stage_fast(smem1, smem0, 0, k4 < last ? k4 : last, two_sets{});
                    __syncthreads();
                    continue;
                }
                if (T::CWAVES * 64 == NT) {
                    stage_fast(smem0, smem1, 0, (kt + 1) * BK, one_set{});
                } else {
                    load_stage_fast((kt + 1) * BK, 0);
                    if (computes) compute_stage(smem0);
                    store_stage(smem1, 0);
                }
                __syncthreads();
                if (T::CWAVES * 64 == NT) {
                    stage_fast(smem1, smem0, 0, (kt + 2) * BK, one_set{});
                } else {
                    load_stage_fast((kt + 2) * BK, 0);
                    if (computes) compute_stage(smem1);
                    store_stage(smem0, 0);
                }
                __syncthreads();
            }
        }
        for (; kt < nk; ++kt) {
            char *cur = (kt & 1) ? smem1 : smem0;
            char *nxt = (kt & 1) ? smem0 : smem1;
            if (kt + 1 < nk) load_stage_checked((kt + 1) * BK);
            if (computes) compute_stage(cur);
            if (kt + 1 < nk) store_stage(nxt, 0);
            __syncthreads();
        }

        // ---- epilogue: FP32 accumulators -> FP32 C, no downcast ----------
        auto result = [&](int j, int i) {
            f32x4 v = acc[j][i];
            if (ALPHA) v = v * p.alpha;
            return v;
        };
        auto store_c = [&](int64_t m, int64_t n, f32x4 v, bool nt) {
            if (m < M && n < N) {
                float *cp = C + m * p.ldc + n;
                if (VEC && p.vecC && n + 4 <= N) {
                    if (nt)
                        __builtin_nontemporal_store(v, reinterpret_cast<f32x4 *>(cp));
                    else
                        *reinterpret_cast<f32x4 *>(cp) = v;
                } else {
                    cp[0] = v.x;
                    if (n + 1 < N) cp[1] = v.y;
                    if (n + 2 < N) cp[2] = v.z;
                    if (n + 3 < N) cp[3] = v.w;
                }
            }
        };
        if (computes) {
            // pairs of 16-column blocks as whole 128-byte lines, streamed
            constexpr int NL = HEAL_TILE_C_LINES && VEC ? (WN / 16) / 2 * 2 : 0;
#pragma unroll
            for (int j = 0; j < NL; j += 2) {
#pragma unroll
                for (int i = 0; i < WM / 16; ++i) {
                    f32x4 x, y;
                    whole_lines(result(j, i), result(j + 1, i), fr, x, y);
                    const int64_t mx = m0 + wm * WM + i * 16 + (fr & 7);
                    const int64_t n = n0 + wn * WN + j * 16 + 16 * (fr >> 3) + 4 * fg;
                    store_c(mx, n, x, true);
                    store_c(mx + 8, n, y, true);
                }
            }
#pragma unroll
            for (int j = NL; j < WN / 16; ++j) {
#pragma unroll
                for (int i = 0; i < WM / 16; ++i)
                    store_c(m0 + wm * WM + i * 16 + fr, n0 + wn * WN + j * 16 + 4 * fg, result(j, i),
                            false);
            }
        }
        if (b + gridDim.y < p.batch) __syncthreads();  // LDS reuse by the next batch entry
    }
}

template <int BM, int BN, int BK, int WM, int WN, int NT, int RS, bool TRANS_B, bool ALPHA>
hipError_t launch_tile3(const GemmArgs &a, dim3 grid, hipStream_t stream)
{
    // The 16-byte path needs every A row and every op(B) row 16-byte aligned
    // and whole quads along K (A, B stored N x K) or N (B stored K x N).
    const bool vec = a.vecA && a.vecB && a.K % 4 == 0 && (TRANS_B || a.N % 4 == 0);
    if (vec)
        hipLaunchKernelGGL((gemm_bf16x3_kernel<BM, BN, BK, WM, WN, NT, RS, TRANS_B, ALPHA, true>), grid,
                           dim3(NT), 0, stream, a);
    else
        hipLaunchKernelGGL((gemm_bf16x3_kernel<BM, BN, BK, WM, WN, NT, RS, TRANS_B, ALPHA, false>), grid,
                           dim3(NT), 0, stream, a);
    return hipGetLastError();
}

template <int BM, int BN, int BK, int WM, int WN, int NT, int RS = 1>
hipError_t launch_tile(const GemmArgs &a, bool trans_b, bool use_alpha, hipStream_t stream)
{
    const int64_t tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
    if (tiles > 0x7fffffffLL) return hipErrorInvalidValue;
    // grid y: each workgroup walks batch entries y, y + gy, ...; two
    // entries per workgroup halve the number of short workgroups
    const int64_t gy64 = (a.batch + HEAL_TILE_BATCH_PER_WG - 1) / HEAL_TILE_BATCH_PER_WG;
    const unsigned gy = (unsigned)(gy64 < 65535 ? gy64 : 65535);
    const dim3 grid((unsigned)tiles, gy);
    if (trans_b)
        return use_alpha ? launch_tile3<BM, BN, BK, WM, WN, NT, RS, true, true>(a, grid, stream)
                         : launch_tile3<BM, BN, BK, WM, WN, NT, RS, true, false>(a, grid, stream);
    return use_alpha ? launch_tile3<BM, BN, BK, WM, WN, NT, RS, false, true>(a, grid, stream)
                     : launch_tile3<BM, BN, BK, WM, WN, NT, RS, false, false>(a, grid, stream);
}

}  // namespace

hipError_t launch_gemm(int instance, const GemmArgs &a, bool trans_b, bool use_alpha,
                       hipStream_t stream)
{
    switch (instance) {
    case HEAL_INSTANCE_LARGE:
        if (HEAL_PANEL && panel_kernel_applies(a, trans_b)) return launch_gemm_panel(a, use_alpha, stream);
        if (large_kernel_applies(a, trans_b)) return launch_gemm_large(a, trans_b, use_alpha, stream);
        return launch_tile<HEAL_LARGE_CFG>(a, trans_b, use_alpha, stream);
    case HEAL_INSTANCE_MEDIUM:
        if (HEAL_PANEL && panel_kernel_applies(a, trans_b)) return launch_gemm_panel(a, use_alpha, stream);
        return launch_tile<HEAL_MEDIUM_CFG>(a, trans_b, use_alpha, stream);
    case HEAL_INSTANCE_SKINNY:
        if (skinny_kernel_applies(a, trans_b)) return launch_gemm_skinny(a, trans_b, use_alpha, stream);
        if (a.M <= 16) return launch_tile<HEAL_SKINNY16_CFG>(a, trans_b, use_alpha, stream);
        if (a.M <= 32) return launch_tile<HEAL_SKINNY32_CFG>(a, trans_b, use_alpha, stream);
        return launch_tile<HEAL_SKINNY64_CFG>(a, trans_b, use_alpha, stream);
    default:
        return hipErrorInvalidValue;
    }
}

}  // namespace heal
