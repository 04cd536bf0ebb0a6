// The skinny compensated bf16x3 GEMM for gfx950 (MI355X): M <= 64 rows,
// the decode and lm_head shapes, where the product is bound by streaming B
// from HBM.
//
// HEAL Section 4 (GEMM paragraph and its displayed expansion): both FP32
// operands are split into bf16 (hi, lo) and C = hiA*hiB + hiA*loB + loA*hiB,
// summed in FP32 and written as FP32.
//
// Work split.  A workgroup owns a strip of BN = 16*CB columns of C and all
// of its (at most 64) rows, or one group of its rows, and walks K in stages
// of BK.  Each element of B is loaded and split by the one workgroup of its
// strip (by each row group's); A (at most 64 x K, resident in L2) is
// re-read by every workgroup.  Strips are as wide as the output allows
// while every CU still gets one (256 columns for a 128256-wide lm_head; 32
// columns with the rows in two groups for a 4096-wide decode): HBM
// bandwidth needs all CUs with loads in flight, and wider strips read
// longer row pieces of B and fewer copies of A.
//
// Pipeline.  A and B are staged in a ring of R register sets: while stage s
// is multiplied out of LDS, stage s+1 is split into the other LDS buffer and
// its register set is reloaded with stage s+1+R, so each load (HBM for B,
// mostly L2 for A) has R stages to arrive.  Split, LDS layout and fragment
// reads follow the large kernel: 16-byte buffer loads, 4x4 register
// transposes of B stored K x N, hi and lo planes with k-contiguous rows,
// 16x16x32 bf16 MFMA fragments.  Lanes outside the matrix read zeros through
// out-of-range buffer offsets; with K % BK != 0 the last stage is masked
// along K the same way.
//
// Reduction order: identical to every other instance (K in 32-deep chunks
// ascending, hiA*hiB, hiA*loB, loA*hiB into one FP32 accumulator, K tail
// zero-filled, the B fragment as the MFMA's first source), so results are
// bitwise equal to them.
#include "heal.h"
#include "heal_device.h"
#include "heal_internal.h"

namespace heal {

namespace {

constexpr uint32_t kOOB = 0x80000000u;  // buffer offset beyond every range: reads 0

__device__ __forceinline__ f32x4 bload(__amdgpu_buffer_rsrc_t r, uint32_t voff, int soff)
{
    return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, soff, 0));
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const float *base, int64_t bytes)
{
    // raw buffer, 32-bit elements; `bytes` < 2^31 is checked on the host
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(base), (short)0, (int)bytes,
                                             0x00020000);
}

// LDS geometry of one stage for a given depth BK (bytes per plane row RP =
// 2*BK).  The LDS has 64 four-byte banks (256-byte bank lines).
//  * chunk swizzle: the 16-byte chunk c of row r is stored at c ^ swz(r),
//    so the 16 lanes of a fragment read (16 rows, one chunk) hit 16
//    different 16-byte bank slots; with rows of 256 bytes or more, odd
//    16-row groups also flip bit 1 (for the row-contiguous B map of
//    32-column strips, below).  The hardware counters still read some
//    conflict cycles with rows of 256 bytes or more (0.56 M per 16 x 4096 x
//    4096 dispatch, 1.08 M at 8192 columns); a swizzle that removes them
//    for 16-column strips left the time unchanged (22.3 vs 22.4 us): these
//    strips are bound by their B stream, not by the LDS;
//  * brow: the LDS row of B column n (B stored K x N), chosen so that one
//    transposed 8-byte store instruction (32 lanes per cycle) covers all
//    banks; it permutes rows within aligned groups of 16, which fragment
//    reads cover whole.
//  With 64-byte rows (32-deep stages) the layout is the large kernel's:
//  chunk swizzle (row >> 1) & 3, odd and even rows of each 8-row group
//  swapped when bit 2 of n is set.  An earlier (row >> 2) & 3 swizzle with
//  a 2-bit row swap read 16.4 M LDS bank-conflict cycles per lm_head
//  dispatch (64 rows, 256-column strips) against 0 for this one, same bits.
template <int BK>
struct Lds {
    static constexpr int RP = 2 * BK;
    static_assert(BK == 32 || BK == 64 || BK >= 128, "stage depth");
    static __device__ __forceinline__ int swz(int row)
    {
        return RP >= 256 ? ((row & 15) ^ ((row >> 3) & 2)) : RP == 128 ? ((row >> 1) & 7)
                                                                         : ((row >> 1) & 3);
    }
    static __device__ __forceinline__ int brow(int n)
    {
        return RP >= 256 ? n : (n ^ ((n >> 2) & 1));
    }
    static __device__ __forceinline__ int chunk_off(int row, int c)
    {
        return row * RP + ((c ^ swz(row)) << 4);
    }
    static __device__ __forceinline__ int quad_off(int row, int kq)
    {
        return row * RP + (((kq >> 1) ^ swz(row)) << 4) + ((kq & 1) << 3);
    }
};

__device__ __forceinline__ void lds_store2(char *base, int off, uint32_t a, uint32_t b)
{
    u32x2 v = {a, b};
    *reinterpret_cast<u32x2 *>(base + off) = v;
}

__device__ __forceinline__ bf16x8 lds_frag(const char *base, int off)
{
    return *reinterpret_cast<const bf16x8 *>(base + off);
}

// Workgroups per CU the LDS of one configuration allows (two when a
// workgroup's two stage buffers fit in half of the 160 KB).
constexpr int skinny_occupancy(int MB, int CB, int BK)
{
    return 2 * 2 * (16 * MB + 16 * CB) * (2 * BK) <= 80 * 1024 ? 2 : 1;
}

// MB: 16-row blocks of the tile (M <= 16*MB); CB: 16-column blocks per
// workgroup; BK: stage depth; R: depth of the A and B register ring (stages in
// flight), even; NT: threads (all load and split; the first
// min(CB, 4) waves also multiply).
template <int MB, int CB, int BK, int R, int NT, bool TRANS_B, bool ALPHA, bool TAIL>
__global__ void __launch_bounds__(NT, skinny_occupancy(MB, CB, BK))
gemm_skinny_kernel(GemmArgs p)
{
    static_assert(R >= 2 && R % 2 == 0, "ring depth");
    static_assert(BK <= 512, "stage depth (offset bounds of skinny_kernel_applies)");
    using L = Lds<BK>;
    constexpr int BM = 16 * MB, BN = 16 * CB, KQ = BK / 4, RP = L::RP;
    constexpr int A_PLANE = BM * RP, B_PLANE = BN * RP;
    constexpr int STAGE = 2 * A_PLANE + 2 * B_PLANE;
    static_assert(2 * STAGE <= 160 * 1024, "two LDS stages must fit the 160 KB of a CU");
    // per thread and stage: NA quads of A; NB quads of B (N x K) or NB/4
    // 4x4 blocks of B (K x N)
    constexpr int NA = BM * KQ / NT;
    constexpr int NB = BN * KQ / NT;
    static_assert(NT % 64 == 0 && NT <= 1024, "whole waves");
    static_assert(NA >= 1 && NA * NT == BM * KQ, "A quads per thread");
    static_assert(NB >= 1 && NB * NT == BN * KQ, "B quads per thread");
    static_assert(TRANS_B || NB % 4 == 0 || NB == 2, "whole or half 4x4 B blocks per thread");
    constexpr int CW = CB < 4 ? CB : 4;         // waves that multiply
    constexpr int JW = CB / CW;                 // column blocks per computing wave
    static_assert(CB % CW == 0, "column blocks per wave");

    __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int fr = lane & 15, fg = lane >> 4;

    // Strips are dealt to XCDs so that each XCD owns a contiguous run of
    // them: workgroups are dispatched to the 8 XCDs round-robin, and without
    // the renumbering two neighbouring 16-column strips, which read the two
    // 64-byte halves of the same 128-byte lines of B, would each miss in a
    // different XCD's L2 and fetch the line from HBM twice.
    int64_t strip = blockIdx.x;
    {
        const int64_t nb = gridDim.x, x = strip & 7, i = strip >> 3, q = nb >> 3, r = nb & 7;
        strip = x * q + (x < r ? x : r) + i;
    }
    const int64_t n0 = strip * BN;
    const int64_t M = p.M, N = p.N, K = p.K;
    const int cols = (int)((N - n0) < BN ? (N - n0) : BN);
    const int ns = (int)((K + BK - 1) / BK);
    const int k_end = (int)K;

    // A quads: q = tid + 256u -> row q / KQ, k-quad q % KQ
    int a_row[NA], a_kq[NA], st_a[NA];
#pragma unroll
    for (int u = 0; u < NA; ++u) {
        const int q = tid + NT * u;
        a_row[u] = q / KQ;
        a_kq[u] = q % KQ;
        st_a[u] = L::quad_off(a_row[u], a_kq[u]);
    }
    // B: N x K quads (like A), or K x N 4x4 blocks b = tid + 256u.  Strips
    // of 16 or 32 columns (64- or 128-byte row pieces) take the row map:
    // column group b % (4 CB), k-quad b / (4 CB), so the lanes of one load
    // instruction read whole row pieces (16 pieces per instruction rather
    // than 64 quarter pieces: 1.4x faster on a 16 x 4096 x 4096 decode).
    // Wider strips take column group b / KQ, k-quad b % KQ, which already
    // reads whole 128-byte lines and has no store conflicts in their LDS
    // geometry.
    // With two units per thread (HALF: twice as many threads as 4x4
    // blocks), a thread loads two rows of a block: column group t % (4 CB),
    // row pair (t / (4 CB)) % 2, k-quad t / (8 CB); one load instruction
    // still reads 16 whole row pieces, and its transposed 4-byte stores
    // (k pairs) fill all 64 banks.
    constexpr bool ROWMAP = CB <= 2 && RP >= 256;
    constexpr bool HALF = !TRANS_B && NB == 2;
    static_assert(!HALF || ROWMAP, "half blocks use the row map");
    int b_kq[NB], b_n[NB], st_b[NB], b_r0[NB];
    int st_h[4] = {0, 0, 0, 0};                  // HALF: LDS offset of column 4c + nn
#pragma unroll
    for (int u = 0; u < NB; ++u) {
        if (TRANS_B) {
            const int q = tid + NT * u;
            b_n[u] = q / KQ;
            b_kq[u] = q % KQ;
            st_b[u] = L::quad_off(b_n[u], b_kq[u]);
            b_r0[u] = 0;
        } else if (HALF) {
            const int c = tid % (4 * CB), half = (tid / (4 * CB)) & 1;
            b_kq[u] = tid / (8 * CB);
            b_n[u] = 4 * c;
            b_r0[u] = 4 * b_kq[u] + 2 * half;    // first of the thread's two rows
            st_b[u] = 0;
#pragma unroll
            for (int nn = 0; nn < 4; ++nn)
                st_h[nn] = L::quad_off(L::brow(4 * c + nn), b_kq[u]) + 4 * half;
        } else {
            const int bl = tid + NT * (u >> 2), nn = u & 3;
            if (ROWMAP) {
                b_kq[u] = bl / (4 * CB);
                b_n[u] = 4 * (bl % (4 * CB)) + nn;
            } else {
                b_kq[u] = bl % KQ;
                b_n[u] = 4 * (bl / KQ) + nn;          // column of unit u
            }
            st_b[u] = L::quad_off(L::brow(b_n[u]), b_kq[u]);
            b_r0[u] = 4 * b_kq[u];
        }
    }
    const int wj0 = wave;                        // first column block of this wave

    for (int64_t b = blockIdx.y; b < p.batch; b += gridDim.y) {
        const float *__restrict__ A = p.A + b * p.strideA;
        const float *__restrict__ B = p.B + b * p.strideB + (TRANS_B ? n0 * p.ldb : n0);
        float *__restrict__ C = p.C + b * p.strideC;

        const __amdgpu_buffer_rsrc_t ra_src = make_rsrc(A, ((M - 1) * p.lda + K) * 4);
        const __amdgpu_buffer_rsrc_t rb_src =
            TRANS_B ? make_rsrc(B, ((int64_t)(cols - 1) * p.ldb + K) * 4)
                    : make_rsrc(B, ((K - 1) * p.ldb + cols) * 4);
        uint32_t va[NA], vb[NB];
#pragma unroll
        for (int u = 0; u < NA; ++u)
            va[u] = a_row[u] < M ? (uint32_t)((a_row[u] * p.lda + 4 * a_kq[u]) * 4) : kOOB;
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            if (TRANS_B)
                vb[u] = b_n[u] < cols ? (uint32_t)((b_n[u] * p.ldb + 4 * b_kq[u]) * 4) : kOOB;
            else {
                const int nq4 = b_n[u] & ~3;         // first column of the block
                vb[u] = nq4 < cols ? (uint32_t)((b_r0[u] * p.ldb + nq4) * 4) : kOOB;
            }
        }
        const int ldb4 = (int)(p.ldb * 4);

        f32x4 xa[R][NA];     // staged A and B: R stages, set = stage % R
        f32x4 xb[R][NB];

        auto load_a = [&](int set, int s) {
#pragma unroll
            for (int u = 0; u < NA; ++u) {
                uint32_t v = va[u];
                if (TAIL && s * BK + 4 * a_kq[u] >= k_end) v = kOOB;
                xa[set][u] = bload(ra_src, v, s * BK * 4);
            }
        };
        auto load_b = [&](int set, int s) {
#pragma unroll
            for (int u = 0; u < NB; ++u) {
                uint32_t v = vb[u];
                if (TRANS_B) {
                    if (TAIL && s * BK + 4 * b_kq[u] >= k_end) v = kOOB;
                    xb[set][u] = bload(rb_src, v, s * BK * 4);
                } else {
                    // row kk = u & 3 of block u >> 2 (HALF: row u of the pair)
                    const int kk = HALF ? u : (u & 3);
                    if (TAIL && s * BK + b_r0[u] + kk >= k_end) v = kOOB;
                    xb[set][u] = bload(rb_src, v, (s * BK + kk) * ldb4);
                }
            }
        };
        auto split_a = [&](char *st, int set) {
#pragma unroll
            for (int u = 0; u < NA; ++u) {
                uint32_t h0, l0, h1, l1;
                split2(xa[set][u].x, xa[set][u].y, h0, l0);
                split2(xa[set][u].z, xa[set][u].w, h1, l1);
                lds_store2(st, st_a[u], h0, h1);
                lds_store2(st + A_PLANE, st_a[u], l0, l1);
            }
        };
        auto split_b = [&](char *st, int set) {
            char *bh = st + 2 * A_PLANE, *bl = bh + B_PLANE;
            if constexpr (HALF) {
                // column nn of the block: element nn of the thread's two rows
#pragma unroll
                for (int nn = 0; nn < 4; ++nn) {
                    uint32_t h, l;
                    split2(xb[set][0][nn], xb[set][1][nn], h, l);
                    *reinterpret_cast<uint32_t *>(bh + st_h[nn]) = h;
                    *reinterpret_cast<uint32_t *>(bl + st_h[nn]) = l;
                }
            } else {
#pragma unroll
                for (int u = 0; u < NB; ++u) {
                    uint32_t h0, l0, h1, l1;
                    if (TRANS_B) {
                        split2(xb[set][u].x, xb[set][u].y, h0, l0);
                        split2(xb[set][u].z, xb[set][u].w, h1, l1);
                    } else {
                        // column nn of the block: element nn of its four rows
                        const int blk = u >> 2, nn = u & 3;
                        split2(xb[set][4 * blk + 0][nn], xb[set][4 * blk + 1][nn], h0, l0);
                        split2(xb[set][4 * blk + 2][nn], xb[set][4 * blk + 3][nn], h1, l1);
                    }
                    lds_store2(bh, st_b[u], h0, h1);
                    lds_store2(bl, st_b[u], l0, l1);
                }
            }
        };

        f32x4 acc[MB][JW];
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
            for (int j = 0; j < JW; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

        // Multiply one stage out of the LDS buffer at `st`.  All fragment
        // reads of the stage are issued first, in the order the MFMAs use
        // them, so their latencies overlap instead of adding up per chunk.
        auto compute = [&](const char *st) {
            if (wave >= CW) return;
            const char *ah = st, *al = st + A_PLANE;
            const char *bh = st + 2 * A_PLANE, *bl = bh + B_PLANE;
            constexpr int KC = BK / 32;
            bf16x8 fah[KC][MB], fal[KC][MB], fbh[KC][JW], fbl[KC][JW];
#pragma unroll
            for (int kc = 0; kc < KC; ++kc) {
#pragma unroll
                for (int j = 0; j < JW; ++j) {
                    const int col = (wj0 + CW * j) * 16 + fr;
                    const int off = L::chunk_off(TRANS_B ? col : L::brow(col), 4 * kc + fg);
                    fbh[kc][j] = lds_frag(bh, off);
                    fbl[kc][j] = lds_frag(bl, off);
                }
#pragma unroll
                for (int i = 0; i < MB; ++i) {
                    const int off = L::chunk_off(i * 16 + fr, 4 * kc + fg);
                    fah[kc][i] = lds_frag(ah, off);
                    fal[kc][i] = lds_frag(al, off);
                }
            }
#pragma unroll
            for (int kc = 0; kc < KC; ++kc) {
#pragma unroll
                for (int j = 0; j < JW; ++j) {
#pragma unroll
                    for (int i = 0; i < MB; ++i)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fbh[kc][j], fah[kc][i], acc[i][j], 0, 0, 0);
#pragma unroll
                    for (int i = 0; i < MB; ++i)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fbl[kc][j], fah[kc][i], acc[i][j], 0, 0, 0);
#pragma unroll
                    for (int i = 0; i < MB; ++i)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fbh[kc][j], fal[kc][i], acc[i][j], 0, 0, 0);
                }
            }
        };

        // Stage t lives in register set t % R.  At step s stage s is
        // multiplied out of LDS buffer s & 1 while the set of stage s+1 is
        // split into the other buffer and then reloaded with stage s+1+R, so
        // each HBM load has R steps to arrive.  Reloads past the last stage
        // are clamped to it (redundant loads whose data is never used).  The
        // loop is unrolled by R (R even), so that register sets and LDS
        // buffers are compile-time choices, and every group of R steps runs
        // whole: only the multiply of a step past the last stage is skipped.
        // With a step under a branch the compiler has to assume a path
        // around it and waits for every outstanding load before the split
        // (vmcnt(0)), which halves the depth of the ring.
        static_assert(R % 2 == 0, "register sets come in pairs");
        const int last = ns - 1;
        auto clamp = [&](int t) { return t < last ? t : last; };
        auto load_set = [&](int set, int s) {
            load_a(set, s);
            load_b(set, s);
        };
        if (ns > 0) {
            load_set(0, 0);
            split_a(smem, 0);
            split_b(smem, 0);
            // the sets are issued in ring order (scheduling barriers keep the
            // compiler from interleaving them), the order the loop keeps, so
            // that every wait before a split is exact
#pragma unroll
            for (int t = 1; t < R; ++t) {
                __builtin_amdgcn_sched_barrier(0);
                load_set(t, clamp(t));
            }
            __builtin_amdgcn_sched_barrier(0);
            load_set(0, clamp(R));
            __builtin_amdgcn_sched_barrier(0);
            __syncthreads();
        }
        for (int s0 = 0; s0 < ns; s0 += R) {
#pragma unroll
            for (int t = 0; t < R; ++t) {
                const int s = s0 + t;
                char *cur = smem + (t & 1) * STAGE;
                char *nxt = smem + ((t + 1) & 1) * STAGE;
                if (s < ns) compute(cur);
                split_a(nxt, (t + 1) % R);
                split_b(nxt, (t + 1) % R);
                load_set((t + 1) % R, clamp(s + 1 + R));
                __syncthreads();
            }
        }

        // ---- epilogue: FP32 accumulators -> FP32 C, no downcast ----------
        if (wave < CW) {
#pragma unroll
            for (int i = 0; i < MB; ++i) {
                const int64_t m = i * 16 + fr;
#pragma unroll
                for (int j = 0; j < JW; ++j) {
                    const int64_t n = n0 + (wj0 + CW * j) * 16 + 4 * fg;
                    f32x4 v = acc[i][j];
                    if (ALPHA) v = v * p.alpha;
                    if (m < M && n < N) *reinterpret_cast<f32x4 *>(C + m * p.ldc + n) = v;
                }
            }
        }
    }
}

template <int MB, int CB, int BK, int R, int NT, bool TRANS_B, bool ALPHA>
hipError_t launch(const GemmArgs &a, hipStream_t stream)
{
    const int64_t tiles = (a.N + 16 * CB - 1) / (16 * CB);
    const unsigned gy = (unsigned)(a.batch < 65535 ? a.batch : 65535);
    if (a.K % BK)
        hipLaunchKernelGGL((gemm_skinny_kernel<MB, CB, BK, R, NT, TRANS_B, ALPHA, true>),
                           dim3((unsigned)tiles, gy), dim3(NT), 0, stream, a);
    else
        hipLaunchKernelGGL((gemm_skinny_kernel<MB, CB, BK, R, NT, TRANS_B, ALPHA, false>),
                           dim3((unsigned)tiles, gy), dim3(NT), 0, stream, a);
    return hipGetLastError();
}

template <int MB, int CB, int BK, int R, int NT>
hipError_t launch_mb(const GemmArgs &a, bool trans_b, bool use_alpha, hipStream_t stream)
{
    if (trans_b)
        return use_alpha ? launch<MB, CB, BK, R, NT, true, true>(a, stream)
                         : launch<MB, CB, BK, R, NT, true, false>(a, stream);
    return use_alpha ? launch<MB, CB, BK, R, NT, false, true>(a, stream)
                     : launch<MB, CB, BK, R, NT, false, false>(a, stream);
}

// Strip width, stage depth and B ring depth by shape.  Measured on the
// MI355X with read-only kernels of the same access pattern (4096-deep B):
// 16-column strips read 64-byte pieces of rows that lie a full row pitch
// apart and stream at ~3.4-3.7 TB/s when each load instruction covers whole
// pieces (~2.5 TB/s with quarter pieces), 32-column strips at ~5.5 TB/s,
// 128- and 256-column strips at ~6.8 TB/s when there are enough of them.
// Every strip re-reads all of A (from L2), and the K order keeps each
// output element in one workgroup, so an output takes the widest strips of
// which it still has enough: about one per CU at 64 rows (at least
// HEAL_SKINNY_MIN_STRIPS), about two at 16 or 32 rows, whose A is cheaper
// to re-read (HEAL_SKINNY_MIN_STRIPS_SMALL), and 32-column strips rather
// than 16 from HEAL_SKINNY_MIN_STRIPS_32 of them (5120 to 7168 columns at
// 16 / 64 rows, 4096 deep: HEAL-Base 17.4-19.7 / 37.5-38.5 us with 16-column
// strips, 16.6-18.2 / 26.5-26.9 with 32; HEAL-Full 21.4-22.2 / 53.9-54.4
// against 18.3-18.6 / 42.5-42.8; pre-split 25.0-27.6 / 59.1-59.8 against
// 20.9-23.5 / 46.9-47.1; bf16x3 41.1-41.8 / 64.0-64.5 against 25.7-26.5 /
// 37.8-38.5; at 4096 columns, 128 strips of 32, the 16-column strips stay
// faster for the packed products).  4096 deep, 64 rows: 4096
// columns 35.4 us with 256 16-column strips (35.9 with 128 of 32 columns);
// 8192 columns 38.7 us with 256 of 32 columns (68.0 with 512 of 16, 61.7
// with 128 of 64); 16032 columns 66.0 us with 251 of 64 columns (127.9 with
// 1002 of 16, 72.3 with 501 of 32, 93.1 with 126 of 128); 32064 columns
// 110 us with 251 of 128 (131 with 501 of 64).  16 rows: 8192 columns 28.9
// us with 256 of 32 (41.6 with 512 of 16); 16032 columns 46.8 us with 501
// of 32 (53.9 with 251 of 64); 65536 columns 212 us with 512 of 128 (241
// with 256 of 256).  The stage depth
// is the smallest that gives every thread whole 16-byte units of A and B at
// the tile's row count.  16-column strips of 64 rows run 512 threads (half
// blocks of B; 33.6 vs 37.6 us with 256), of 17 to 32 rows 256 threads
// (25.7 vs 26.5 us with 512), of 16 rows either (22.6 us; a read-only
// kernel of the same B pattern takes 17.5 us, 20.5 us when it also reads A
// from L2 as every workgroup here does).  256-column strips (lm_head, 64 x
// 128256 x 4096, with 16, 32 or 64 rows): 512 threads where every thread
// still gets whole A quads: 0.43 / 0.40 / 0.37 ms against 0.55 / 0.45 /
// 0.39 ms for 128-column strips at 16 and 32 rows and 256 threads.
// Configurations: CB (16-column blocks per strip), BK, R, NT; the suffix is
// the strip width, _1 / _2 / _4 the row count (16 / 32 / 64 rows).
#ifndef HEAL_SKINNY_N1
#define HEAL_SKINNY_N1 1, 256, 2, 512
#endif
#ifndef HEAL_SKINNY_N2
#define HEAL_SKINNY_N2 1, 128, 2, 256
#endif
#ifndef HEAL_SKINNY_N4
#define HEAL_SKINNY_N4 1, 256, 2, 512      // 160 KB of LDS: one workgroup per CU
#endif
#ifndef HEAL_SKINNY_S32
#define HEAL_SKINNY_S32 2, 128, 2, 512     // half blocks of B, every row count
#endif
#ifndef HEAL_SKINNY_S64_1
#define HEAL_SKINNY_S64_1 4, 64, 2, 256
#endif
#ifndef HEAL_SKINNY_S64_2
#define HEAL_SKINNY_S64_2 4, 64, 2, 256
#endif
#ifndef HEAL_SKINNY_S64_4
#define HEAL_SKINNY_S64_4 4, 64, 2, 256
#endif
#ifndef HEAL_SKINNY_S128_1
#define HEAL_SKINNY_S128_1 8, 64, 2, 256
#endif
#ifndef HEAL_SKINNY_S128_2
#define HEAL_SKINNY_S128_2 8, 64, 2, 512
#endif
#ifndef HEAL_SKINNY_S128_4
#define HEAL_SKINNY_S128_4 8, 64, 2, 512
#endif
#ifndef HEAL_SKINNY_W1
#define HEAL_SKINNY_W1 16, 64, 2, 256
#endif
#ifndef HEAL_SKINNY_W2
#define HEAL_SKINNY_W2 16, 64, 2, 512
#endif
#ifndef HEAL_SKINNY_W4
#define HEAL_SKINNY_W4 16, 32, 2, 512
#endif
#ifndef HEAL_SKINNY_MIN_STRIPS
#define HEAL_SKINNY_MIN_STRIPS 240
#endif
#ifndef HEAL_SKINNY_MIN_STRIPS_SMALL
#define HEAL_SKINNY_MIN_STRIPS_SMALL 480
#endif
#ifndef HEAL_SKINNY_MIN_STRIPS_32
#define HEAL_SKINNY_MIN_STRIPS_32 160
#endif

// Row groups.  Where the width rule leaves an output with 16-column strips
// (fewer than HEAL_SKINNY_MIN_STRIPS_32 of 32 columns), a product with one
// batch entry runs on 32-column strips instead, its rows split into G
// groups (1, 2 or 4, dividing M) that run as separate workgroups, as many
// as gives at most HEAL_SKINNY_GROUP_WGS workgroups and at least
// HEAL_SKINNY_GROUP_MIN_WGS.  With B stored K x N each workgroup then
// requests every 128-byte line of its strip whole (a 16-column strip reads
// half lines) and re-reads only its group's rows of A.  A row's bits do not
// depend on the other rows, so the result is that of one group.  Measured
// on 4096-deep products (us; 16-column strips, then the groups): 2048
// columns at 16 / 64 rows 21.3 / 33.1 -> 19.2 / 21.4 (four groups); 3072
// columns 22.7 / 33.9 -> 21.8 / 27.2 (two); 4096 columns 22.6 / 33.7 ->
// 20.9 / 26.2 (two).  More groups than that (more than 256 workgroups)
// were slower again.  With B stored N x K a 16-column strip already reads
// whole lines, and only A's re-reads favour groups: there they apply with
// more than 32 rows and at least HEAL_SKINNY_GROUP_MIN_WGS_NK workgroups
// (2048 / 4096 columns at 64 rows 31.1 / 33.1 -> 17.4 / 23.2; at 16 rows
// they were slower, 14.3 / 16.7 -> 16.5 / 17.7; one group of 32-column
// strips at 4096 columns, 128 workgroups, 16.7 -> 18.2).
#ifndef HEAL_SKINNY_ROW_GROUPS
#define HEAL_SKINNY_ROW_GROUPS 1
#endif
#ifndef HEAL_SKINNY_GROUP_WGS
#define HEAL_SKINNY_GROUP_WGS 256
#endif
#ifndef HEAL_SKINNY_GROUP_MIN_WGS
#define HEAL_SKINNY_GROUP_MIN_WGS 128
#endif
#ifndef HEAL_SKINNY_GROUP_MIN_WGS_NK
#define HEAL_SKINNY_GROUP_MIN_WGS_NK 160
#endif

template <int MB>
hipError_t launch_width(const GemmArgs &a, int w, bool trans_b, bool use_alpha, hipStream_t stream)
{
    if (w == 32) return launch_mb<MB, HEAL_SKINNY_S32>(a, trans_b, use_alpha, stream);
    if constexpr (MB == 1) {
        if (w == 256) return launch_mb<1, HEAL_SKINNY_W1>(a, trans_b, use_alpha, stream);
        if (w == 128) return launch_mb<1, HEAL_SKINNY_S128_1>(a, trans_b, use_alpha, stream);
        if (w == 64) return launch_mb<1, HEAL_SKINNY_S64_1>(a, trans_b, use_alpha, stream);
        return launch_mb<1, HEAL_SKINNY_N1>(a, trans_b, use_alpha, stream);
    } else if constexpr (MB == 2) {
        if (w == 256) return launch_mb<2, HEAL_SKINNY_W2>(a, trans_b, use_alpha, stream);
        if (w == 128) return launch_mb<2, HEAL_SKINNY_S128_2>(a, trans_b, use_alpha, stream);
        if (w == 64) return launch_mb<2, HEAL_SKINNY_S64_2>(a, trans_b, use_alpha, stream);
        return launch_mb<2, HEAL_SKINNY_N2>(a, trans_b, use_alpha, stream);
    } else {
        if (w == 256) return launch_mb<4, HEAL_SKINNY_W4>(a, trans_b, use_alpha, stream);
        if (w == 128) return launch_mb<4, HEAL_SKINNY_S128_4>(a, trans_b, use_alpha, stream);
        if (w == 64) return launch_mb<4, HEAL_SKINNY_S64_4>(a, trans_b, use_alpha, stream);
        return launch_mb<4, HEAL_SKINNY_N4>(a, trans_b, use_alpha, stream);
    }
}

}  // namespace

// Strip width in columns for an output of N columns and M <= 64 rows: the
// widest of 256, 128, 64 and 32 with at least HEAL_SKINNY_MIN_STRIPS_SMALL
// strips at up to 32 rows (HEAL_SKINNY_MIN_STRIPS above), else 32 if that
// still gives HEAL_SKINNY_MIN_STRIPS_32, else 16.
int skinny_strip_width(int64_t N, int64_t M)
{
    const int64_t least = M <= 32 ? HEAL_SKINNY_MIN_STRIPS_SMALL : HEAL_SKINNY_MIN_STRIPS;
    for (int w = 256; w >= 32; w /= 2)
        if ((N + w - 1) / w >= least) return w;
    return (N + 31) / 32 >= HEAL_SKINNY_MIN_STRIPS_32 ? 32 : 16;
}

bool skinny_kernel_applies(const GemmArgs &a, bool trans_b)
{
    // At most 64 rows, 16-byte rows, whole quads along K (and N).  Buffer
    // offsets are 32-bit: the largest is that of the last element a lane may
    // address, (M-1)*lda + K (+ one stage, at most 512 deep, for a clamped
    // reload) for A, the same with the 256-row strip for B stored N x K, and
    // (K+3)*ldb + 256 for B stored K x N (row k + kk of a 4-row block).
    if (a.M > 64 || !(a.vecA && a.vecB && a.vecC) || a.K % 4 != 0 || a.N % 4 != 0) return false;
    const int64_t lim = 0x7fffffffLL;
    if (((a.M - 1) * a.lda + a.K + 512) * 4 >= lim) return false;
    if (trans_b ? ((int64_t)255 * a.ldb + a.K + 512) * 4 >= lim : ((a.K + 3) * a.ldb + 256) * 4 >= lim)
        return false;
    return (a.N + 15) / 16 <= 0x7fffffffLL;
}

// Row groups of an output (0: none apply; see HEAL_SKINNY_ROW_GROUPS).
static int skinny_row_groups(int64_t N, int64_t M, bool trans_b, int64_t batch)
{
    if (!HEAL_SKINNY_ROW_GROUPS || batch != 1 || M < 1 || skinny_strip_width(N, M) != 16)
        return 0;
    const int64_t strips = (N + 31) / 32;
    const int gmax = trans_b && M <= 32 ? 1 : 4;
    int g = 1;
    while (g < gmax && strips * 2 * g <= HEAL_SKINNY_GROUP_WGS && M % (2 * g) == 0) g *= 2;
    const int64_t least = trans_b ? HEAL_SKINNY_GROUP_MIN_WGS_NK : HEAL_SKINNY_GROUP_MIN_WGS;
    return strips * g >= least ? g : 0;
}

hipError_t launch_gemm_skinny(const GemmArgs &a, bool trans_b, bool use_alpha, hipStream_t stream)
{
    GemmArgs r = a;
    int w = skinny_strip_width(a.N, a.M);
    if (const int g = skinny_row_groups(a.N, a.M, trans_b, a.batch)) {
        // the groups as batch entries: rows M/g each, B shared
        w = 32;
        r.M = a.M / g;
        r.batch = g;
        r.strideA = r.M * a.lda;
        r.strideB = 0;
        r.strideC = r.M * a.ldc;
    }
    if (r.M <= 16) return launch_width<1>(r, w, trans_b, use_alpha, stream);
    if (r.M <= 32) return launch_width<2>(r, w, trans_b, use_alpha, stream);
    return launch_width<4>(r, w, trans_b, use_alpha, stream);
}

}  // namespace heal
