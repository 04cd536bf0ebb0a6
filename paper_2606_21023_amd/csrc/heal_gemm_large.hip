// The large-tile compensated bf16x3 GEMM for gfx950 (MI355X): 256 x 256
// output tiles.  Two forms share the data path below: eight waves of
// 64 x 128 (two waves per SIMD, the default) and four waves of 128 x 128
// (one wave per SIMD).
//
// HEAL Section 4 (GEMM paragraph and its displayed expansion) keeps a GEMM
// on the 16-bit matrix units and recovers the bits a single 16-bit cast
// drops by adding residual products, summed in FP32.  Both FP32 operands are
// split into bf16 (hi, lo) and C = hiA*hiB + hiA*loB + loA*hiB.
//
// Why these shapes.  Per 32-deep stage the workgroup moves 64 KB of FP32
// from L2, splits it (six VALU instructions per element pair), stores 64 KB
// of bf16 planes into LDS and reads the MFMA fragments back, against 768
// bf16 MFMAs.  On gfx950 one wave cannot issue 16x16x32 bf16 MFMAs back to
// back: a register-only loop sustains about two thirds of the matrix core's
// rate with one wave per SIMD and nearly all of it with two.  The eight-wave
// form therefore keeps two waves per SIMD (128 accumulators each, 64 x 128
// wave tiles, 192 KB of fragment reads per stage); the four-wave form reads
// a third less LDS (128 x 128 wave tiles, 256 accumulators per lane in
// AGPRs) but is capped by the single-wave issue rate.  On 8192^3 the
// eight-wave form is about 4% faster, on 2048 x 14336 x 4096 about 11%.
// In both, the split and the LDS traffic are interleaved with the MFMAs.
//
// Pipeline.  Two LDS stage buffers.  While stage s is multiplied out of one
// buffer, the FP32 data of stage s+1 (already in VGPRs) is split into the
// other, and each staged register group is reloaded with stage s+2 as soon
// as its split is done, so every global load has one full stage to arrive.
// One barrier per stage.
//
// Edges.  Loads are buffer loads: a lane whose row or column lies outside
// the matrix gets an offset beyond the buffer's range and reads zeros, so
// edge tiles run the same code.  The K tail (K % 32 != 0) is one extra stage
// with the same masking applied along K.  Stores are masked per row.
//
// Reduction order: for every output element, K in 32-deep chunks ascending,
// each chunk adding hiA*hiB, hiA*loB, loA*hiB into one FP32 accumulator, K
// tail zero-filled; MFMA operand roles as in every other instance (the B
// fragment is the first source).  Results are therefore bitwise equal to the
// other instances.
#include "heal.h"
#include "heal_device.h"
#include "heal_internal.h"

namespace heal {

namespace {

constexpr int kBM = 256, kBN = 256, kBK = 32, kNT = 256;
constexpr int kWT = 128;                // wave tile edge
constexpr int kRowB = kBK * 2;          // bytes per LDS row of one plane (32 bf16)
constexpr int kPlane = 256 * kRowB;     // 16 KB
constexpr int kStage = 4 * kPlane;      // A_hi, A_lo, B_hi, B_lo
constexpr uint32_t kOOB = 0x80000000u;  // buffer offset beyond every range: reads 0

// Tuning knobs.  Waves per workgroup: 8, or 4 for the one-wave-per-SIMD form.
#ifndef HEAL_LARGE_WAVES
#define HEAL_LARGE_WAVES 8
#endif
// Instruction pattern of one 12-MFMA column block of the 8-wave form:
// 1: fragment reads, 6 x (MFMA, 2 VALU), LDS writes, reloads, 6 MFMAs;
// 2: 12 x (MFMA, VALU); 3: 10 x (MFMA, 3 VALU), then the rest;
// 4 (default): fragment reads, HEAL_L8_NV x (MFMA, HEAL_L8_VPM VALU), the
// reloads, the LDS writes, the remaining MFMAs (8 x 2: 1.1-1.3% faster than
// 1 at 8192^3 on two boards; 7, 9, 10 pairs or 1 or 3 VALU per MFMA were
// not; reloads before the LDS writes another 0.9-1.3% on two boards).
#ifndef HEAL_L8_PATTERN
#define HEAL_L8_PATTERN 4
#endif
#ifndef HEAL_L8_NV
#define HEAL_L8_NV 8
#endif
#ifndef HEAL_L8_VPM
#define HEAL_L8_VPM 2
#endif
#ifndef HEAL_L8_VMEM_FIRST
#define HEAL_L8_VMEM_FIRST 1
#endif
// Epilogue of the 8-wave form: whole-line non-temporal C stores (8192^3
// 1.0% faster in six interleaved rounds, 2048 x 14336 x 4096 unchanged;
// same bits).
#ifndef HEAL_LARGE_C_LINES
#define HEAL_LARGE_C_LINES 1
#endif
// 4-wave form: VALU slots of one 24-MFMA group, and VALU per slot.
#ifndef HEAL_LARGE_VALU_SLOTS
#define HEAL_LARGE_VALU_SLOTS 12
#endif
#ifndef HEAL_LARGE_VALU_PER_MFMA
#define HEAL_LARGE_VALU_PER_MFMA 2
#endif

// LDS layout of one plane: row r (m for A, n for B) holds its 32 k values,
// 64 bytes, as four 16-byte chunks of 8 k; the chunk index is XORed with
// bits 1..2 of the row so that 16 lanes reading one chunk column of 16 rows,
// and 16 lanes writing 8-byte quads, hit distinct banks.
__device__ __forceinline__ int chunk_off(int row, int c)
{
    return row * kRowB + ((c ^ ((row >> 1) & 3)) << 4);
}
// 4 consecutive k (k = 4*kq) of row `row`
__device__ __forceinline__ int quad_off(int row, int kq)
{
    return row * kRowB + ((((kq >> 1) ^ ((row >> 1) & 3))) << 4) + ((kq & 1) << 3);
}
// LDS row of B column n (B stored K x N): the halves of each 8-row group swap
// odd and even rows when bit 2 of n is set, so that the transposed writes of
// one instruction (all lanes at the same column offset within their 4x4
// block) cover every bank.  Reads cover whole 8-row groups and are unaffected.
__device__ __forceinline__ int brow(int n) { return n ^ ((n >> 2) & 1); }

__device__ __forceinline__ void lds_store2(char *base, int off, uint32_t a, uint32_t b)
{
    u32x2 v = {a, b};
    *reinterpret_cast<u32x2 *>(base + off) = v;
}

__device__ __forceinline__ bf16x8 lds_frag(const char *base, int off)
{
    return *reinterpret_cast<const bf16x8 *>(base + off);
}

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

template <bool TRANS_B, bool ALPHA, bool TAIL>
__global__ void __launch_bounds__(kNT, 1)
gemm_large_kernel(GemmArgs p)
{
    // Thread -> data maps (per stage, 16 loads of 16 bytes per thread):
    //   A, and B stored N x K: quad u (0..7) is row tid/8 + 32u, k-quad tid%8.
    //   B stored K x N: block u (0..1) is the 4 (k) x 4 (n) block with
    //     k-quad (lane>>1)&7 and column group (lane&1) | (lane>>4)<<1 |
    //     wave<<3, + 32u; its four rows are loaded and transposed in registers.
    // TAIL: K % 32 != 0, the last stage is masked along K.
    __shared__ __attribute__((aligned(16))) char smem[2 * kStage];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    const int fr = lane & 15, fg = lane >> 4;

    // ---- tile coordinates: XCD-aware renumbering, grouped along M --------
    const int64_t tiles_m = (p.M + kBM - 1) / kBM;
    const int64_t tiles_n = (p.N + kBN - 1) / kBN;
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
    const int64_t m0 = (first_m + in_group % gm) * kBM;
    const int64_t n0 = (in_group / gm) * kBN;

    const int64_t M = p.M, N = p.N, K = p.K;
    const int rows_a = (int)((M - m0) < kBM ? (M - m0) : kBM);    // valid rows of the tile
    const int cols_b = (int)((N - n0) < kBN ? (N - n0) : kBN);    // valid columns
    const int ns = (int)((K + kBK - 1) / kBK);                    // stages, the tail included

    const int a_row = tid >> 3, a_kq = tid & 7;
    const int b_kq = (lane >> 1) & 7;
    const int b_nq = (lane & 1) | ((lane >> 4) << 1) | (wave << 3);

    // LDS store offsets: quad u of A is 32u rows below quad 0, which leaves
    // the swizzle bits unchanged; B stored K x N has one offset per column
    // nn of the 4x4 block, and block 1 is 128 rows below block 0.
    const int st_a = quad_off(a_row, a_kq);
    int st_b[4];
#pragma unroll
    for (int nn = 0; nn < 4; ++nn) st_b[nn] = TRANS_B ? st_a : quad_off(brow(4 * b_nq + nn), b_kq);
    // fragment read offsets
    const int rd_a = chunk_off(wm * kWT + fr, fg);
    const int rd_b = chunk_off(TRANS_B ? wn * kWT + fr : brow(wn * kWT + fr), fg);

    for (int64_t b = blockIdx.y; b < p.batch; b += gridDim.y) {
        const float *__restrict__ A = p.A + b * p.strideA + m0 * p.lda;
        const float *__restrict__ B = p.B + b * p.strideB + (TRANS_B ? n0 * p.ldb : n0);
        float *__restrict__ C = p.C + b * p.strideC;

        // buffer ranges: the tile's rows (A, and B stored N x K) or the
        // tile's columns over all K (B stored K x N); every valid element of
        // the tile lies inside, and masked lanes use kOOB.
        const __amdgpu_buffer_rsrc_t ra_src = make_rsrc(A, ((int64_t)(rows_a - 1) * p.lda + K) * 4);
        const __amdgpu_buffer_rsrc_t rb_src =
            TRANS_B ? make_rsrc(B, ((int64_t)(cols_b - 1) * p.ldb + K) * 4)
                    : make_rsrc(B, ((K - 1) * p.ldb + cols_b) * 4);
        uint32_t va[8], vb[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            va[u] = a_row + 32 * u < rows_a ? (uint32_t)(((a_row + 32 * u) * p.lda + 4 * a_kq) * 4) : kOOB;
        if (TRANS_B) {
#pragma unroll
            for (int u = 0; u < 8; ++u)
                vb[u] = a_row + 32 * u < cols_b ? (uint32_t)(((a_row + 32 * u) * p.ldb + 4 * a_kq) * 4) : kOOB;
        } else {
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int n = 4 * (b_nq + 32 * u);
                vb[u] = n < cols_b ? (uint32_t)((4 * b_kq * p.ldb + n) * 4) : kOOB;
            }
        }
        const int ldb4 = (int)(p.ldb * 4);
        const int k_end = (int)K;

        // staged FP32 data of one stage
        f32x4 ra[8], rb[8];

        // Load quad / row u of stage s.  With TAIL, k >= K reads zeros (the
        // test is always true on full stages).
        auto load_a = [&](int u, int s) {
            uint32_t v = va[u];
            if (TAIL && s * kBK + 4 * a_kq >= k_end) v = kOOB;
            ra[u] = bload(ra_src, v, s * kBK * 4);
        };
        auto load_b = [&](int u, int s) {
            if (TRANS_B) {
                uint32_t v = vb[u];
                if (TAIL && s * kBK + 4 * a_kq >= k_end) v = kOOB;
                rb[u] = bload(rb_src, v, s * kBK * 4);
            } else {
                // block u>>2, row kk = u&3
                const int kk = u & 3;
                uint32_t v = vb[u >> 2];
                if (TAIL && s * kBK + 4 * b_kq + kk >= k_end) v = kOOB;
                rb[u] = bload(rb_src, v, (s * kBK + kk) * ldb4);
            }
        };
        // Split unit u (0..15) of the staged data into the stage buffer at `s`.
        auto split_unit = [&](char *s, int u) {
            uint32_t h0, l0, h1, l1;
            if (u < 8) {
                split2(ra[u].x, ra[u].y, h0, l0);
                split2(ra[u].z, ra[u].w, h1, l1);
                lds_store2(s, st_a + u * 32 * kRowB, h0, h1);
                lds_store2(s + kPlane, st_a + u * 32 * kRowB, l0, l1);
            } else if (TRANS_B) {
                const int v = u - 8;
                split2(rb[v].x, rb[v].y, h0, l0);
                split2(rb[v].z, rb[v].w, h1, l1);
                lds_store2(s + 2 * kPlane, st_a + v * 32 * kRowB, h0, h1);
                lds_store2(s + 3 * kPlane, st_a + v * 32 * kRowB, l0, l1);
            } else {
                // column nn of block blk: the four rows' element nn
                const int v = u - 8, blk = v >> 2, nn = v & 3;
                split2(rb[4 * blk + 0][nn], rb[4 * blk + 1][nn], h0, l0);
                split2(rb[4 * blk + 2][nn], rb[4 * blk + 3][nn], h1, l1);
                lds_store2(s + 2 * kPlane, st_b[nn] + blk * 128 * kRowB, h0, h1);
                lds_store2(s + 3 * kPlane, st_b[nn] + blk * 128 * kRowB, l0, l1);
            }
        };
        // After unit u is split, reload its registers with stage s.
        auto reload_unit = [&](int u, int s) {
            if (u < 8) {
                load_a(u, s);
            } else if (TRANS_B) {
                load_b(u - 8, s);
            } else if ((u & 3) == 3) {
                const int blk = (u - 8) >> 2;
#pragma unroll
                for (int kk = 0; kk < 4; ++kk) load_b(4 * blk + kk, s);
            }
        };

        f32x4 acc[8][8];
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

        // ---- prologue: stage 0 into buffer 0, stage 1 into registers -----
        if (ns > 0) {
#pragma unroll
            for (int u = 0; u < 8; ++u) load_a(u, 0);
#pragma unroll
            for (int u = 0; u < 8; ++u) load_b(u, 0);
#pragma unroll
            for (int u = 0; u < 16; ++u) split_unit(smem, u);
            const int s1 = ns > 1 ? 1 : 0;
#pragma unroll
            for (int u = 0; u < 8; ++u) load_a(u, s1);
#pragma unroll
            for (int u = 0; u < 8; ++u) load_b(u, s1);
            __syncthreads();
        }

        // ---- main loop: one stage per trip, one barrier ------------------
        // Stage s is multiplied out of buffer s&1 (192 MFMAs per wave);
        // meanwhile the staged data of stage s+1 is split into the other
        // buffer, unit by unit, each unit's registers being reloaded with
        // stage s+2 (clamped to the last stage: the last trips split and
        // load redundant copies that are never read).
        for (int s = 0; s < ns; ++s) {
            const char *cur = smem + (s & 1) * kStage;
            char *nxt = smem + ((s + 1) & 1) * kStage;
            const int s_reload = s + 2 < ns ? s + 2 : ns - 1;
            const char *a_hi = cur, *a_lo = cur + kPlane;
            const char *b_hi = cur + 2 * kPlane, *b_lo = cur + 3 * kPlane;
            bf16x8 bh[8], bl[8], ah[2], al[2];
            ah[0] = lds_frag(a_hi, rd_a);
#pragma unroll
            for (int j = 0; j < 8; ++j) bh[j] = lds_frag(b_hi, rd_b + j * 16 * kRowB);
            al[0] = lds_frag(a_lo, rd_a);
#pragma unroll
            for (int j = 0; j < 8; ++j) bl[j] = lds_frag(b_lo, rd_b + j * 16 * kRowB);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int c = i & 1;
                if (i + 1 < 8) {
                    ah[c ^ 1] = lds_frag(a_hi, rd_a + (i + 1) * 16 * kRowB);
                    al[c ^ 1] = lds_frag(a_lo, rd_a + (i + 1) * 16 * kRowB);
                }
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bh[j], ah[c], acc[i][j], 0, 0, 0);
                split_unit(nxt, 2 * i);
                reload_unit(2 * i, s_reload);
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bl[j], ah[c], acc[i][j], 0, 0, 0);
                split_unit(nxt, 2 * i + 1);
                reload_unit(2 * i + 1, s_reload);
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bh[j], al[c], acc[i][j], 0, 0, 0);
                // One wave per SIMD issues in order, so the split's VALU work
                // only overlaps the matrix core if it sits between MFMAs:
                // fragment reads first, then MFMA / 2 VALU pairs, the LDS
                // stores and reloads, then the remaining MFMAs.
                __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
                for (int t = 0; t < HEAL_LARGE_VALU_SLOTS; ++t) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x002, HEAL_LARGE_VALU_PER_MFMA, 0);
                }
                __builtin_amdgcn_sched_group_barrier(0x200, 2, 0);
                __builtin_amdgcn_sched_group_barrier(0x020, 5, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, 24 - HEAL_LARGE_VALU_SLOTS, 0);
                __builtin_amdgcn_sched_barrier(0);
            }
            __syncthreads();
        }

        // ---- epilogue: FP32 accumulators -> FP32 C, no downcast ----------
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int64_t m = m0 + wm * kWT + i * 16 + fr;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int64_t n = n0 + wn * kWT + j * 16 + 4 * fg;
                f32x4 v = acc[i][j];
                if (ALPHA) v = v * p.alpha;
                if (m < M && n < N) *reinterpret_cast<f32x4 *>(C + m * p.ldc + n) = v;
            }
        }
    }
}


// Eight-wave form: two waves per SIMD, wave tiles of 64 x 128 (128 FP32
// accumulators per lane).  A single wave cannot issue 16x16x32 MFMAs back to
// back (it sustains about two thirds of the matrix core's rate); two waves
// per SIMD can.  Same LDS layout, loads, split and per-element order as the
// four-wave form; the MFMA loop walks the eight 16-column blocks of the wave
// tile with the four A fragment pairs resident.
template <bool TRANS_B, bool ALPHA, bool TAIL>
__global__ void __launch_bounds__(512, 1)
gemm_large8_kernel(GemmArgs p)
{
    constexpr int NT = 512;
    // Thread -> data maps (per stage, 8 loads of 16 bytes per thread):
    //   A, and B stored N x K: quad u (0..3) is row tid/8 + 64u, k-quad tid%8.
    //   B stored K x N: the 4 (k) x 4 (n) block with k-quad (lane>>1)&7 and
    //     column group (lane&1) | (lane>>4)<<1 | wave<<3.
    __shared__ __attribute__((aligned(16))) char smem[2 * kStage];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave & 3, wn = wave >> 2;
    const int fr = lane & 15, fg = lane >> 4;

    const int64_t tiles_m = (p.M + kBM - 1) / kBM;
    const int64_t tiles_n = (p.N + kBN - 1) / kBN;
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
    const int64_t m0 = (first_m + in_group % gm) * kBM;
    const int64_t n0 = (in_group / gm) * kBN;

    const int64_t M = p.M, N = p.N, K = p.K;
    const int rows_a = (int)((M - m0) < kBM ? (M - m0) : kBM);
    const int cols_b = (int)((N - n0) < kBN ? (N - n0) : kBN);
    const int ns = (int)((K + kBK - 1) / kBK);

    const int a_row = tid >> 3, a_kq = tid & 7;
    const int b_kq = (lane >> 1) & 7;
    const int b_nq = (lane & 1) | ((lane >> 4) << 1) | (wave << 3);
    const int st_a = quad_off(a_row, a_kq);
    int st_b[4];
#pragma unroll
    for (int nn = 0; nn < 4; ++nn) st_b[nn] = TRANS_B ? st_a : quad_off(brow(4 * b_nq + nn), b_kq);
    const int rd_a = chunk_off(wm * 64 + fr, fg);
    const int rd_b = chunk_off(TRANS_B ? wn * kWT + fr : brow(wn * kWT + fr), fg);

    for (int64_t b = blockIdx.y; b < p.batch; b += gridDim.y) {
        const float *__restrict__ A = p.A + b * p.strideA + m0 * p.lda;
        const float *__restrict__ B = p.B + b * p.strideB + (TRANS_B ? n0 * p.ldb : n0);
        float *__restrict__ C = p.C + b * p.strideC;

        const __amdgpu_buffer_rsrc_t ra_src = make_rsrc(A, ((int64_t)(rows_a - 1) * p.lda + K) * 4);
        const __amdgpu_buffer_rsrc_t rb_src =
            TRANS_B ? make_rsrc(B, ((int64_t)(cols_b - 1) * p.ldb + K) * 4)
                    : make_rsrc(B, ((K - 1) * p.ldb + cols_b) * 4);
        uint32_t va[4], vb[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            va[u] = a_row + 64 * u < rows_a ? (uint32_t)(((a_row + 64 * u) * p.lda + 4 * a_kq) * 4) : kOOB;
        if (TRANS_B) {
#pragma unroll
            for (int u = 0; u < 4; ++u)
                vb[u] = a_row + 64 * u < cols_b ? (uint32_t)(((a_row + 64 * u) * p.ldb + 4 * a_kq) * 4) : kOOB;
        } else {
            const int n = 4 * b_nq;
            vb[0] = n < cols_b ? (uint32_t)((4 * b_kq * p.ldb + n) * 4) : kOOB;
        }
        const int ldb4 = (int)(p.ldb * 4);
        const int k_end = (int)K;

        f32x4 ra[4], rb[4];
        auto load_a = [&](int u, int s) {
            uint32_t v = va[u];
            if (TAIL && s * kBK + 4 * a_kq >= k_end) v = kOOB;
            ra[u] = bload(ra_src, v, s * kBK * 4);
        };
        auto load_b = [&](int u, int s) {
            if (TRANS_B) {
                uint32_t v = vb[u];
                if (TAIL && s * kBK + 4 * a_kq >= k_end) v = kOOB;
                rb[u] = bload(rb_src, v, s * kBK * 4);
            } else {
                const int kk = u;            // row kk of the block
                uint32_t v = vb[0];
                if (TAIL && s * kBK + 4 * b_kq + kk >= k_end) v = kOOB;
                rb[u] = bload(rb_src, v, (s * kBK + kk) * ldb4);
            }
        };
        auto split_unit = [&](char *s, int u) {
            uint32_t h0, l0, h1, l1;
            if (u < 4) {
                split2(ra[u].x, ra[u].y, h0, l0);
                split2(ra[u].z, ra[u].w, h1, l1);
                lds_store2(s, st_a + u * 64 * kRowB, h0, h1);
                lds_store2(s + kPlane, st_a + u * 64 * kRowB, l0, l1);
            } else if (TRANS_B) {
                const int v = u - 4;
                split2(rb[v].x, rb[v].y, h0, l0);
                split2(rb[v].z, rb[v].w, h1, l1);
                lds_store2(s + 2 * kPlane, st_a + v * 64 * kRowB, h0, h1);
                lds_store2(s + 3 * kPlane, st_a + v * 64 * kRowB, l0, l1);
            } else {
                const int nn = u - 4;
                split2(rb[0][nn], rb[1][nn], h0, l0);
                split2(rb[2][nn], rb[3][nn], h1, l1);
                lds_store2(s + 2 * kPlane, st_b[nn], h0, h1);
                lds_store2(s + 3 * kPlane, st_b[nn], l0, l1);
            }
        };
        auto reload_unit = [&](int u, int s) {
            if (u < 4) {
                load_a(u, s);
            } else if (TRANS_B) {
                load_b(u - 4, s);
            } else if (u == 7) {
#pragma unroll
                for (int kk = 0; kk < 4; ++kk) load_b(kk, s);
            }
        };

        f32x4 acc[8][4];
#pragma unroll
        for (int j = 0; j < 8; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[j][i] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

        if (ns > 0) {
#pragma unroll
            for (int u = 0; u < 4; ++u) load_a(u, 0);
#pragma unroll
            for (int u = 0; u < 4; ++u) load_b(u, 0);
#pragma unroll
            for (int u = 0; u < 8; ++u) split_unit(smem, u);
            const int s1 = ns > 1 ? 1 : 0;
#pragma unroll
            for (int u = 0; u < 4; ++u) load_a(u, s1);
#pragma unroll
            for (int u = 0; u < 4; ++u) load_b(u, s1);
            __syncthreads();
        }

        for (int s = 0; s < ns; ++s) {
            const char *cur = smem + (s & 1) * kStage;
            char *nxt = smem + ((s + 1) & 1) * kStage;
            const int s_reload = s + 2 < ns ? s + 2 : ns - 1;
            const char *a_hi = cur, *a_lo = cur + kPlane;
            const char *b_hi = cur + 2 * kPlane, *b_lo = cur + 3 * kPlane;
            bf16x8 ah[4], al[4], bh[2], bl[2];
            bh[0] = lds_frag(b_hi, rd_b);
#pragma unroll
            for (int i = 0; i < 4; ++i) ah[i] = lds_frag(a_hi, rd_a + i * 16 * kRowB);
            bl[0] = lds_frag(b_lo, rd_b);
#pragma unroll
            for (int i = 0; i < 4; ++i) al[i] = lds_frag(a_lo, rd_a + i * 16 * kRowB);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int c = j & 1;
                if (j + 1 < 8) {
                    bh[c ^ 1] = lds_frag(b_hi, rd_b + (j + 1) * 16 * kRowB);
                    bl[c ^ 1] = lds_frag(b_lo, rd_b + (j + 1) * 16 * kRowB);
                }
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bh[c], ah[i], acc[j][i], 0, 0, 0);
                split_unit(nxt, j);
                reload_unit(j, s_reload);
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bl[c], ah[i], acc[j][i], 0, 0, 0);
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bh[c], al[i], acc[j][i], 0, 0, 0);
#if HEAL_L8_PATTERN == 1
                __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
                for (int t = 0; t < 6; ++t) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
                }
                __builtin_amdgcn_sched_group_barrier(0x200, 2, 0);
                __builtin_amdgcn_sched_group_barrier(0x020, 4, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, 6, 0);
#elif HEAL_L8_PATTERN == 2
                __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
                for (int t = 0; t < 12; ++t) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);
                }
                __builtin_amdgcn_sched_group_barrier(0x200, 2, 0);
                __builtin_amdgcn_sched_group_barrier(0x020, 4, 0);
#elif HEAL_L8_PATTERN == 3
                __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
                for (int t = 0; t < 10; ++t) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
                }
                __builtin_amdgcn_sched_group_barrier(0x200, 2, 0);
                __builtin_amdgcn_sched_group_barrier(0x020, 4, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
#elif HEAL_L8_PATTERN == 4
                __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
                for (int t = 0; t < HEAL_L8_NV; ++t) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x002, HEAL_L8_VPM, 0);
                }
#if HEAL_L8_VMEM_FIRST
                __builtin_amdgcn_sched_group_barrier(0x020, 4, 0);
                __builtin_amdgcn_sched_group_barrier(0x200, 2, 0);
#else
                __builtin_amdgcn_sched_group_barrier(0x200, 2, 0);
                __builtin_amdgcn_sched_group_barrier(0x020, 4, 0);
#endif
                __builtin_amdgcn_sched_group_barrier(0x008, 12 - HEAL_L8_NV, 0);
#endif
                __builtin_amdgcn_sched_barrier(0);
            }
            __syncthreads();
        }

#if HEAL_LARGE_C_LINES
        // whole 128-byte lines per store (two adjacent 16-column blocks),
        // non-temporal: C is written once and would only evict A and B
        // from L2
#pragma unroll
        for (int j = 0; j < 8; j += 2) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                f32x4 r0 = acc[j][i], r1 = acc[j + 1][i];
                if (ALPHA) {
                    r0 = r0 * p.alpha;
                    r1 = r1 * p.alpha;
                }
                f32x4 x, y;
                whole_lines(r0, r1, fr, x, y);
                const int64_t mx = m0 + wm * 64 + i * 16 + (fr & 7), my = mx + 8;
                const int64_t n = n0 + wn * kWT + j * 16 + 16 * (fr >> 3) + 4 * fg;
                if (mx < M && n < N)
                    __builtin_nontemporal_store(x, reinterpret_cast<f32x4 *>(C + mx * p.ldc + n));
                if (my < M && n < N)
                    __builtin_nontemporal_store(y, reinterpret_cast<f32x4 *>(C + my * p.ldc + n));
            }
        }
#else
#pragma unroll
        for (int j = 0; j < 8; ++j) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int64_t m = m0 + wm * 64 + i * 16 + fr;
                const int64_t n = n0 + wn * kWT + j * 16 + 4 * fg;
                f32x4 v = acc[j][i];
                if (ALPHA) v = v * p.alpha;
                if (m < M && n < N) *reinterpret_cast<f32x4 *>(C + m * p.ldc + n) = v;
            }
        }
#endif
    }
}

template <bool TRANS_B, bool ALPHA>
hipError_t launch(const GemmArgs &a, hipStream_t stream)
{
    const int64_t tiles = ((a.M + kBM - 1) / kBM) * ((a.N + kBN - 1) / kBN);
    const unsigned gy = (unsigned)(a.batch < 65535 ? a.batch : 65535);
    const dim3 grid((unsigned)tiles, gy);
#if HEAL_LARGE_WAVES == 8
    if (a.K % kBK)
        hipLaunchKernelGGL((gemm_large8_kernel<TRANS_B, ALPHA, true>), grid, dim3(512), 0, stream, a);
    else
        hipLaunchKernelGGL((gemm_large8_kernel<TRANS_B, ALPHA, false>), grid, dim3(512), 0, stream, a);
#else
    if (a.K % kBK)
        hipLaunchKernelGGL((gemm_large_kernel<TRANS_B, ALPHA, true>), grid, dim3(kNT), 0, stream, a);
    else
        hipLaunchKernelGGL((gemm_large_kernel<TRANS_B, ALPHA, false>), grid, dim3(kNT), 0, stream, a);
#endif
    return hipGetLastError();
}

}  // namespace

bool large_kernel_applies(const GemmArgs &a, bool trans_b)
{
    // 16-byte rows, whole quads along K (and along N for B stored K x N),
    // all buffer offsets of a tile below 2^31, and a grid that fits.
    if (!(a.vecA && a.vecB && a.vecC) || a.K % 4 != 0) return false;
    if (!trans_b && a.N % 4 != 0) return false;
    if (a.N % 4 != 0) return false;   // 16-byte stores of C
    const int64_t lim = 0x7fffffffLL;
    if (((int64_t)(kBM - 1) * a.lda + a.K) * 4 >= lim) return false;
    if (trans_b ? ((int64_t)(kBN - 1) * a.ldb + a.K) * 4 >= lim
                : ((a.K + kBK - 1) * a.ldb + kBN) * 4 >= lim)
        return false;
    const int64_t tiles = ((a.M + kBM - 1) / kBM) * ((a.N + kBN - 1) / kBN);
    return tiles <= 0x7fffffffLL;
}

hipError_t launch_gemm_large(const GemmArgs &a, bool trans_b, bool use_alpha, hipStream_t stream)
{
    if (trans_b)
        return use_alpha ? launch<true, true>(a, stream) : launch<true, false>(a, stream);
    return use_alpha ? launch<false, true>(a, stream) : launch<false, false>(a, stream);
}

}  // namespace heal
