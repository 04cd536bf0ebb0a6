// The short-K panel kernel for gfx950 (MI355X): products whose K is at most
// 128 with B stored N x K, the shape of attention scores (Q K^T over a head
// dimension of 128).  Two products run on it:
//
//  * bf16x3 (HEAL Section 4, GEMM paragraph and its displayed expansion):
//    FP32 operands split into bf16 (hi, lo), C = hiA*hiB + hiA*loB + loA*hiB;
//  * the INT16 scores (HEAL Section 4, Q/K/V paragraph): INT16 codes split
//    into two exact FP16 parts (hi, q - hi), four products, the sum scaled
//    by alpha (maxQ/32767)(maxK/32767).
//
// Such products are bound by writing C: every output element costs 4 bytes
// of HBM writes against 2K or 4K multiply-adds, so the kernel is built to
// keep the write stream busy.  A workgroup owns a panel of 128 or 256 rows
// of A (one batch entry), splits it once into LDS, and then walks its share
// of the columns of C in steps of 128: each of its four waves loads the B
// fragments of its 32 columns straight from global memory (B stored N x K:
// a lane's 8 consecutive k of one column are 32 contiguous bytes), splits
// them in registers, multiplies them against the whole panel and stores its
// block of C in whole 128-byte lines, non-temporal (streamed past the
// caches, which the output would only pollute).  The loads of the next
// step are issued before the multiplies
// of the current one, so they have a whole step to arrive, and the stores of
// a step drain while the next one is multiplied.  B goes from L2 to
// registers once per workgroup (no LDS round trip), and the panel is read
// from LDS once per 32 columns.
//
// Workgroups are numbered so that each XCD owns a contiguous range of
// panels: the panels of one batch entry share its B in that XCD's L2.
//
// Reduction order: identical to every other instance (K in 32-deep chunks
// ascending; per chunk hiA*hiB, hiA*loB, loA*hiB for bf16x3 and hiQ*hiK,
// hiQ*loK, loQ*hiK, loQ*loK for the scores; one FP32 accumulator, the B
// fragment as the MFMA's first source, the K tail zero-filled), so results
// are bitwise equal to theirs.
#include "heal.h"
#include "heal_device.h"
#include "heal_internal.h"

namespace heal {

namespace {

constexpr int PKMAX = 128;          // deepest K a panel holds
constexpr int PRP = 2 * PKMAX;      // LDS row pitch of a 16-bit plane, bytes
constexpr int PNT = 256;            // four waves
constexpr int PWN = 32;             // columns per wave and step
constexpr int PBN = 4 * PWN;        // columns per step
constexpr uint32_t kOOB = 0x80000000u;  // beyond every buffer range: loads read zeros

// Panel rows (bf16x3, scores), workgroups per panel (each walking half of
// the columns with 2) and steps of B loads in flight per wave.  Measured on
// the attention scores (32 heads, 2048 x 2048 x 128): bf16x3 150 us with
// 256-row panels against 155 us with 128; the scores 128 us with 128-row
// panels against 136 us with 256; two workgroups per panel 1.05x faster
// than one, four slower; two steps of loads in flight slower than one.
#ifndef HEAL_PANEL_BM
#define HEAL_PANEL_BM 256
#endif
#ifndef HEAL_PANEL_BM_SCORES
#define HEAL_PANEL_BM_SCORES 128
#endif
#ifndef HEAL_PANEL_CSPLIT
#define HEAL_PANEL_CSPLIT 2
#endif
#ifndef HEAL_PANEL_PD
#define HEAL_PANEL_PD 1
#endif
#ifndef HEAL_PANEL_PD_SCORES
#define HEAL_PANEL_PD_SCORES 1
#endif
// C stores: with HEAL_PANEL_LINES each store instruction writes whole
// 128-byte lines (8 rows x 32 columns, the two 16 x 16 results of a row
// block traded between lane halves), and HEAL_PANEL_STORE_AUX 2 marks them
// non-temporal.  Measured on the attention scores: bf16x3 135 us and the
// INT16 scores 117 us, against 151 and 135 us for the 16-row x 64-byte
// stores of one result each with the default policy; whole lines with the
// default policy 154 / 135 us; non-temporal stores of 64-byte pieces
// 184 / 173 us (their lines reach HBM in halves).
#ifndef HEAL_PANEL_STORE_AUX
#define HEAL_PANEL_STORE_AUX 2
#endif
#ifndef HEAL_PANEL_LINES
#define HEAL_PANEL_LINES 1
#endif

struct PanelArgs {
    int64_t M, N, K;
    const char *A;
    int64_t lda, strideA;   // elements
    const char *B;          // N x K rows
    int64_t ldb, strideB;
    float *C;
    int64_t ldc, strideC;
    int64_t batch;
    float alpha;            // bf16x3: output scale (SCALE); scores: alpha
    const float *maxA, *maxB;  // scores: max|Q|, max|K| (device)
    int csplit;             // workgroups per panel, each walking its share of the columns
};

__device__ __forceinline__ u32x4 bload(__amdgpu_buffer_rsrc_t r, uint32_t voff)
{
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, 0, 0));
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const char *base, int64_t bytes)
{
    // raw buffer; `bytes` < 2^31 is checked on the host
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(base), (short)0, (int)bytes,
                                             0x00020000);
}

// 16-byte chunk c (8 values of k) of panel row r, XOR-swizzled so that the
// 16 rows of a fragment read fall in 16 different bank groups.
__device__ __forceinline__ int panel_off(int r, int c) { return r * PRP + ((c ^ (r & 15)) << 4); }

template <bool SCORES>
__device__ __forceinline__ f32x4 mma(u32x4 b, u32x4 a, f32x4 c)
{
    if constexpr (SCORES)
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, b),
                                                      __builtin_bit_cast(f16x8, a), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, b),
                                                       __builtin_bit_cast(bf16x8, a), c, 0, 0, 0);
}

// Two parts of 8 consecutive values: bf16 (hi, lo) of 8 FP32 (two quads),
// or FP16 (hi, q - hi) of 8 INT16 codes (one 16-byte unit).
template <bool SCORES>
__device__ __forceinline__ void split8(const u32x4 *raw, u32x4 &h, u32x4 &l)
{
    if constexpr (SCORES) {
        const u32x4 v = raw[0];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            uint32_t hh, ll;
            unpack2_i16((int)(int16_t)(v[t] & 0xffffu), (int)(int16_t)(v[t] >> 16), hh, ll);
            h[t] = hh;
            l[t] = ll;
        }
    } else {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const f32x4 v = __builtin_bit_cast(f32x4, raw[q]);
            uint32_t h0, l0, h1, l1;
            split2(v.x, v.y, h0, l0);
            split2(v.z, v.w, h1, l1);
            h[2 * q] = h0;
            h[2 * q + 1] = h1;
            l[2 * q] = l0;
            l[2 * q + 1] = l1;
        }
    }
}

// KC: 32-deep chunks of K (K <= 32 KC).  SCALE: multiply the bf16x3 result
// by alpha.  PD: steps of B loads in flight per wave.  PBM: rows of the
// panel (128: two workgroups per CU; 256: one, B read from L2 half as often).
template <bool SCORES, bool SCALE, int KC, int PD, int PBM>
__global__ void __launch_bounds__(PNT, PBM <= 128 ? 2 : 1) gemm_panel_kernel(PanelArgs p)
{
    constexpr int PRB = PBM / 16;               // 16-row blocks of the panel
    constexpr int PPLANE = PBM * PRP;           // one LDS plane of the panel
    static_assert(KC >= 1 && 32 * KC <= PKMAX, "K chunks of a panel");
    constexpr int ES = SCORES ? 2 : 4;          // bytes per operand element
    constexpr int RQ = SCORES ? 1 : 2;          // 16-byte loads per 8 values
    constexpr int UPR = 32 * KC * ES / 16;      // 16-byte units per panel row
    constexpr int PU = PBM * UPR / PNT;         // panel units per thread
    static_assert(PU * PNT == PBM * UPR, "whole panel units per thread");

    __shared__ __attribute__((aligned(16))) char smem[2 * PPLANE];
    char *const ph = smem;                      // hi plane
    char *const pl = smem + PPLANE;             // lo plane

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int fr = lane & 15, fg = lane >> 4;

    // ---- panel: XCD-grouped numbering, then (batch entry, row panel) -----
    const int64_t panels = (p.M + PBM - 1) / PBM;
    int64_t L = blockIdx.x;
    {
        const int64_t nb = gridDim.x, x = L & 7, i = L >> 3, q = nb >> 3, r = nb & 7;
        L = x * q + (x < r ? x : r) + i;
    }
    const int64_t pid = L / p.csplit;
    const int cs = (int)(L - pid * p.csplit);
    const int64_t b = pid / panels;
    const int64_t m0 = (pid - b * panels) * PBM;
    const int64_t M = p.M, N = p.N, K = p.K;
    const int rows = (int)(M - m0 < PBM ? M - m0 : PBM);

    const __amdgpu_buffer_rsrc_t ra =
        make_rsrc(p.A + (b * p.strideA + m0 * p.lda) * ES, ((rows - 1) * p.lda + K) * ES);
    const __amdgpu_buffer_rsrc_t rb = make_rsrc(p.B + b * p.strideB * ES, ((N - 1) * p.ldb + K) * ES);
    const __amdgpu_buffer_rsrc_t rc =
        make_rsrc(reinterpret_cast<const char *>(p.C + b * p.strideC), ((M - 1) * p.ldc + N) * 4);

    // ---- issue the panel loads, then the first step's B loads ------------
    u32x4 pa[PU];
#pragma unroll
    for (int u = 0; u < PU; ++u) {
        const int q = tid + PNT * u, r = q / UPR, c = q % UPR;   // row, 16-byte unit
        const bool ok = r < rows && (int64_t)c * (16 / ES) < K;
        pa[u] = bload(ra, ok ? (uint32_t)((r * p.lda) * ES + c * 16) : kOOB);
    }

    // B fragment of lane (fr, fg) at step s, column block j, chunk c:
    // column 128 s + 32 wave + 16 j + fr, k = 32 c + 8 fg .. + 7
    const int64_t all_steps = (N + PBN - 1) / PBN;
    const int s_begin = (int)(all_steps * cs / p.csplit);
    const int s_end = (int)(all_steps * (cs + 1) / p.csplit);
    // The panels of a batch entry walk their columns from different starts
    // (panel i from its i-th step, wrapping around): the workgroups running
    // at one time then write to many column ranges of C rather than all to
    // the same 512 bytes of every row (attention scores: bf16x3 1.2x, INT16
    // 1.07x faster).  The order of the steps changes no result.
    const int cnt = s_end - s_begin;
    const int rot = cnt > 0 ? (int)(pid % cnt) : 0;
    auto step_of = [&](int t) {
        const int u = t + rot;
        return s_begin + (u >= cnt ? u - cnt : u);
    };
    u32x4 raw[PD][2][KC][RQ];
    auto clamp = [&](int t) { return t < cnt ? t : (cnt > 0 ? cnt - 1 : 0); };
    auto load_b = [&](int set, int s) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t n = (int64_t)s * PBN + wave * PWN + j * 16 + fr;
#pragma unroll
            for (int c = 0; c < KC; ++c) {
#pragma unroll
                for (int h = 0; h < RQ; ++h) {
                    const int k = 32 * c + 8 * fg + 4 * h;
                    const bool ok = n < N && k < K;
                    raw[set][j][c][h] = bload(rb, ok ? (uint32_t)((n * p.ldb + k) * ES) : kOOB);
                }
            }
        }
    };
#pragma unroll
    for (int d = 0; d < PD; ++d) {
        __builtin_amdgcn_sched_barrier(0);
        load_b(d, step_of(clamp(d)));
    }
    __builtin_amdgcn_sched_barrier(0);

    // ---- split the panel into LDS ----------------------------------------
#pragma unroll
    for (int u = 0; u < PU; ++u) {
        const int q = tid + PNT * u, r = q / UPR, c = q % UPR;
        if constexpr (SCORES) {
            u32x4 h, l;
            split8<true>(&pa[u], h, l);
            *reinterpret_cast<u32x4 *>(ph + panel_off(r, c)) = h;
            *reinterpret_cast<u32x4 *>(pl + panel_off(r, c)) = l;
        } else {
            // a quad: half of 16-byte chunk c / 2
            const f32x4 v = __builtin_bit_cast(f32x4, pa[u]);
            uint32_t h0, l0, h1, l1;
            split2(v.x, v.y, h0, l0);
            split2(v.z, v.w, h1, l1);
            const int off = panel_off(r, c >> 1) + 8 * (c & 1);
            u32x2 hv = {h0, h1}, lv = {l0, l1};
            *reinterpret_cast<u32x2 *>(ph + off) = hv;
            *reinterpret_cast<u32x2 *>(pl + off) = lv;
        }
    }
    __syncthreads();

    float scale = 1.0f;
    if constexpr (SCORES)
        // alpha (maxQ / 32767)(maxK / 32767) evaluated in FP64, rounded once
        scale = (float)((double)p.alpha * (double)*p.maxA * (double)*p.maxB / (32767.0 * 32767.0));
    else if constexpr (SCALE)
        scale = p.alpha;

    // ---- walk the columns of C -------------------------------------------
    // Step t splits register set t % PD and reloads it with step t + PD, so
    // each load has PD steps to arrive, and at least PD - 1 steps of stores
    // issued after it do not hold it up.  The loop runs whole groups of PD
    // steps (register sets are compile-time choices and every wait stays
    // exact); a step past the last one multiplies clamped copies and stores
    // nothing.
    auto step = [&](int set, int t) {
        const bool live = t < cnt;
        const int s = step_of(clamp(t));
        u32x4 bh[2][KC], bl[2][KC];
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int c = 0; c < KC; ++c) split8<SCORES>(raw[set][j][c], bh[j][c], bl[j][c]);
        // The reload goes into the registers just split (steps past the end
        // reload the last step: loads whose data is never used), after the
        // split: the scheduling barriers keep the compiler from hoisting
        // them into another register set, which it then copies back with a
        // wait for every outstanding store.
        __builtin_amdgcn_sched_barrier(0);
        load_b(set, step_of(clamp(t + PD)));
        __builtin_amdgcn_sched_barrier(0);

        // Row blocks one after another: the panel fragments of block i + 1
        // are read while block i is multiplied, and the block's two 16 x 16
        // results are stored as soon as their chains end, as two stores of
        // whole 128-byte lines (or, without HEAL_PANEL_LINES, one store of
        // 16 rows x 64 bytes per result).  The scheduling barriers keep the
        // compiler from hoisting every LDS read of the step to its top,
        // which would not fit the registers.
        u32x4 ah[KC], al[KC];
        auto read_a = [&](int i, u32x4 *h, u32x4 *l) {
#pragma unroll
            for (int c = 0; c < KC; ++c) {
                const int off = panel_off(16 * i + fr, 4 * c + fg);
                h[c] = *reinterpret_cast<const u32x4 *>(ph + off);
                l[c] = *reinterpret_cast<const u32x4 *>(pl + off);
            }
        };
        read_a(0, ah, al);
#pragma unroll
        for (int i = 0; i < PRB; ++i) {
            u32x4 nh[KC], nl[KC];
            if (i + 1 < PRB) read_a(i + 1, nh, nl);
#if HEAL_PANEL_LINES
            // both 16 x 16 results of the row block, then whole 128-byte
            // lines per store: one store holds rows 0..7 of the block, 32
            // columns each, the other rows 8..15
            f32x4 r[2];
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                f32x4 a = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int c = 0; c < KC; ++c) {
                    a = mma<SCORES>(bh[j][c], ah[c], a);
                    a = mma<SCORES>(bl[j][c], ah[c], a);
                    a = mma<SCORES>(bh[j][c], al[c], a);
                    if constexpr (SCORES) a = mma<SCORES>(bl[j][c], al[c], a);
                }
                if (SCORES || SCALE) a = a * scale;   // FP32 C, no downcast
                r[j] = a;
            }
            f32x4 x, y;
            whole_lines(r[0], r[1], fr, x, y);
            {
                const int64_t mx = m0 + 16 * i + (fr & 7), my = mx + 8;
                const int64_t n = (int64_t)s * PBN + wave * PWN + 16 * (fr >> 3) + 4 * fg;
                const uint32_t ox = live && mx < M && n < N ? (uint32_t)((mx * p.ldc + n) * 4) : kOOB;
                const uint32_t oy = live && my < M && n < N ? (uint32_t)((my * p.ldc + n) * 4) : kOOB;
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, x), rc, (int)ox, 0,
                                                       HEAL_PANEL_STORE_AUX);
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, y), rc, (int)oy, 0,
                                                       HEAL_PANEL_STORE_AUX);
            }
#else
            const int64_t m = m0 + 16 * i + fr;
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                f32x4 a = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int c = 0; c < KC; ++c) {
                    a = mma<SCORES>(bh[j][c], ah[c], a);
                    a = mma<SCORES>(bl[j][c], ah[c], a);
                    a = mma<SCORES>(bh[j][c], al[c], a);
                    if constexpr (SCORES) a = mma<SCORES>(bl[j][c], al[c], a);
                }
                // FP32 C, no downcast
                if (SCORES || SCALE) a = a * scale;
                const int64_t n = (int64_t)s * PBN + wave * PWN + j * 16 + 4 * fg;
                // buffer store, lanes outside C (and every lane of a step
                // past the end) at an offset beyond its range: no branch
                // around the store, so that each wait for a reload counts the
                // stores exactly and does not wait for them
                const uint32_t off =
                    live && m < M && n < N ? (uint32_t)((m * p.ldc + n) * 4) : kOOB;
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, a), rc, (int)off, 0,
                                                       HEAL_PANEL_STORE_AUX);
            }
#endif
            if (i + 1 < PRB) {
#pragma unroll
                for (int c = 0; c < KC; ++c) {
                    ah[c] = nh[c];
                    al[c] = nl[c];
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    for (int t0 = 0; t0 < cnt; t0 += PD) {
#pragma unroll
        for (int d = 0; d < PD; ++d) step(d, t0 + d);
    }
}

template <bool SCORES, bool SCALE>
hipError_t launch_kc(const PanelArgs &a, hipStream_t stream)
{
    constexpr int PD = SCORES ? HEAL_PANEL_PD_SCORES : HEAL_PANEL_PD;
    constexpr int BM = SCORES ? HEAL_PANEL_BM_SCORES : HEAL_PANEL_BM;
    const dim3 grid((unsigned)(a.batch * ((a.M + BM - 1) / BM) * a.csplit));
    const int kc = (int)((a.K + 31) / 32);
    switch (kc) {
    case 1: hipLaunchKernelGGL((gemm_panel_kernel<SCORES, SCALE, 1, PD, BM>), grid, dim3(PNT), 0, stream, a); break;
    case 2: hipLaunchKernelGGL((gemm_panel_kernel<SCORES, SCALE, 2, PD, BM>), grid, dim3(PNT), 0, stream, a); break;
    case 3: hipLaunchKernelGGL((gemm_panel_kernel<SCORES, SCALE, 3, PD, BM>), grid, dim3(PNT), 0, stream, a); break;
    case 4: hipLaunchKernelGGL((gemm_panel_kernel<SCORES, SCALE, 4, PD, BM>), grid, dim3(PNT), 0, stream, a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// Shape conditions shared by both products (es: bytes per operand element).
// K at most 128 and nonzero, whole 16-byte units along K (quads of FP32,
// eights of INT16), 16-byte rows of A, B and C, N % 4 == 0 (whole 16-byte
// stores), at least one full panel of rows, every byte offset a lane may
// address within a panel of A or a batch entry of B below 2^31, and one
// workgroup per (batch entry, panel) within the grid limit; C written with
// buffer stores, so a batch entry of C spans less than 2^31 bytes.
bool panel_shape_ok(int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldb, int64_t ldc,
                    int64_t batch, int es, int PBM, int csplit)
{
    if (K <= 0 || K > PKMAX || (K * es) % 16 != 0 || N % 4 != 0 || M < PBM) return false;
    const int64_t lim = 0x7fffffffLL;
    if (((int64_t)(PBM - 1) * lda + K) * es >= lim) return false;
    if (((N - 1) * ldb + K) * es >= lim) return false;
    if (((M - 1) * ldc + N) * 4 >= lim) return false;
    return batch * ((M + PBM - 1) / PBM) * csplit <= lim;
}

}  // namespace

bool panel_kernel_applies(const GemmArgs &a, bool trans_b)
{
    return trans_b && a.vecA && a.vecB && a.vecC &&
           panel_shape_ok(a.M, a.N, a.K, a.lda, a.ldb, a.ldc, a.batch, 4, HEAL_PANEL_BM,
                          HEAL_PANEL_CSPLIT);
}

hipError_t launch_gemm_panel(const GemmArgs &g, bool use_alpha, hipStream_t stream)
{
    PanelArgs a = {};
    a.M = g.M;
    a.N = g.N;
    a.K = g.K;
    a.A = reinterpret_cast<const char *>(g.A);
    a.lda = g.lda;
    a.strideA = g.strideA;
    a.B = reinterpret_cast<const char *>(g.B);
    a.ldb = g.ldb;
    a.strideB = g.strideB;
    a.C = g.C;
    a.ldc = g.ldc;
    a.strideC = g.strideC;
    a.batch = g.batch;
    a.alpha = g.alpha;
    a.csplit = HEAL_PANEL_CSPLIT;
    return use_alpha ? launch_kc<false, true>(a, stream) : launch_kc<false, false>(a, stream);
}

bool scores_panel_applies(const OpArgs &a)
{
    return a.vecA && a.vecB && a.vecC && panel_shape_ok(a.M, a.N, a.K, a.lda, a.ldb, a.ldc, a.batch, 2,
                                                     HEAL_PANEL_BM_SCORES, HEAL_PANEL_CSPLIT);
}

hipError_t launch_scores_panel(const OpArgs &o, hipStream_t stream)
{
    PanelArgs a = {};
    a.M = o.M;
    a.N = o.N;
    a.K = o.K;
    a.A = reinterpret_cast<const char *>(o.A);
    a.lda = o.lda;
    a.strideA = o.strideA;
    a.B = reinterpret_cast<const char *>(o.B);
    a.ldb = o.ldb;
    a.strideB = o.strideB;
    a.C = o.C;
    a.ldc = o.ldc;
    a.strideC = o.strideC;
    a.batch = o.batch;
    a.alpha = o.alpha;
    a.maxA = o.maxA;
    a.maxB = o.maxB;
    a.csplit = HEAL_PANEL_CSPLIT;
    return launch_kc<true, false>(a, stream);
}

}  // namespace heal
