// C ABI of libheal.so: argument validation, device check, instance choice.
// Every argument check runs before the first HIP call.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <hip/hip_runtime.h>

#include "heal.h"
#include "heal_internal.h"

namespace {

constexpr int kMaxDevices = 64;
// 0 = unknown, 1 = gfx950, 2 = other architecture
int g_device_arch[kMaxDevices];

heal_status_t check_device()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return HEAL_ERR_LAUNCH;
    if (dev < 0) return HEAL_ERR_LAUNCH;
    int state = dev < kMaxDevices ? __atomic_load_n(&g_device_arch[dev], __ATOMIC_RELAXED) : 0;
    if (state == 0) {
        hipDeviceProp_t prop;
        if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return HEAL_ERR_LAUNCH;
        state = strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 2;
        if (dev < kMaxDevices) __atomic_store_n(&g_device_arch[dev], state, __ATOMIC_RELAXED);
    }
    return state == 1 ? HEAL_OK : HEAL_ERR_UNSUPPORTED_DEVICE;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

// M x N outputs whose element count (and so every tile count) fits in 2^62.
bool product_fits(int64_t M, int64_t N) { return M == 0 || N <= ((int64_t)1 << 62) / M; }

// A dispatch counts work-items in 32 bits per grid dimension.  Every kernel
// here has at most 1024 threads per workgroup and at most one workgroup per
// 16 x 16 block of C (the short-K panel kernel also lays its batch entries
// along the grid), so a launch is held to 2^21 such blocks over its batch
// entries: at most 2^31 work-items.  Larger calls run as several launches,
// each on a range of batch entries, rows and columns of C (rows and columns
// in multiples of 256).  Each output element is summed in the same K order
// by every kernel, so the result bits do not depend on how a call is cut.
constexpr int64_t kLaunchBlocks = (int64_t)1 << 21;
constexpr int64_t kLaunchCols = (int64_t)1 << 20;

template <class F>
heal_status_t for_each_part(int64_t batch, int64_t M, int64_t N, F launch)
{
    auto blocks = [](int64_t x) { return (x + 15) / 16; };
    const int64_t nc = N < kLaunchCols ? N : kLaunchCols;
    int64_t mc = kLaunchBlocks / blocks(nc) * 16;   // at least 512 rows
    mc = mc >= M ? M : mc / 256 * 256;
    int64_t bc = kLaunchBlocks / (blocks(mc) * blocks(nc));
    bc = bc < 1 ? 1 : bc > batch ? batch : bc;
    for (int64_t b0 = 0; b0 < batch; b0 += bc)
        for (int64_t m0 = 0; m0 < M; m0 += mc)
            for (int64_t n0 = 0; n0 < N; n0 += nc) {
                const int64_t bn = batch - b0 < bc ? batch - b0 : bc;
                const int64_t mn = M - m0 < mc ? M - m0 : mc;
                const int64_t nn = N - n0 < nc ? N - n0 : nc;
                if (launch(b0, bn, m0, mn, n0, nn) != hipSuccess) return HEAL_ERR_LAUNCH;
            }
    return HEAL_OK;
}

int select_instance(int64_t M, int64_t N)
{
    (void)N;
    if (M <= 64) return HEAL_INSTANCE_SKINNY;
    if (M * N <= (int64_t)2048 * 2048) return HEAL_INSTANCE_MEDIUM;
    return HEAL_INSTANCE_LARGE;
}

// Validate a strided-batched call; returns HEAL_OK if it may proceed.
heal_status_t validate(int64_t M, int64_t N, int64_t K, const float *A, int64_t lda,
                       int64_t strideA, const float *B, int64_t ldb, int64_t strideB, int trans_b,
                       float *C, int64_t ldc, int64_t strideC, int64_t batch)
{
    if (M < 0 || N < 0 || K < 0 || batch < 0) return HEAL_ERR_INVALID_VALUE;
    if (trans_b != 0 && trans_b != 1) return HEAL_ERR_INVALID_VALUE;
    if (strideA < 0 || strideB < 0 || strideC < 0) return HEAL_ERR_INVALID_VALUE;
    if (lda < (K > 1 ? K : 1)) return HEAL_ERR_INVALID_VALUE;
    if (ldb < (trans_b ? (K > 1 ? K : 1) : (N > 1 ? N : 1))) return HEAL_ERR_INVALID_VALUE;
    if (ldc < (N > 1 ? N : 1)) return HEAL_ERR_INVALID_VALUE;
    // sizes whose element offsets would not fit in int64
    const int64_t lim = (int64_t)1 << 48;
    if (M > lim || N > lim || K > lim || lda > lim || ldb > lim || ldc > lim || batch > lim)
        return HEAL_ERR_INVALID_VALUE;
    if (!product_fits(M, N)) return HEAL_ERR_INVALID_VALUE;
    if (M == 0 || N == 0 || batch == 0) return HEAL_OK;
    if (!C || !aligned4(C)) return HEAL_ERR_INVALID_VALUE;
    if (K > 0 && (!A || !B || !aligned4(A) || !aligned4(B))) return HEAL_ERR_INVALID_VALUE;
    return HEAL_OK;
}

heal_status_t run_gemm(int instance, int64_t M, int64_t N, int64_t K, float alpha, const float *A,
                       int64_t lda, int64_t strideA, const float *B, int64_t ldb, int64_t strideB,
                       int trans_b, float *C, int64_t ldc, int64_t strideC, int64_t batch,
                       hipStream_t stream)
{
    heal_status_t st = validate(M, N, K, A, lda, strideA, B, ldb, strideB, trans_b, C, ldc,
                                strideC, batch);
    if (st != HEAL_OK) return st;
    if (instance < 0 || instance >= HEAL_INSTANCE_COUNT) return HEAL_ERR_INVALID_VALUE;
    if (M == 0 || N == 0 || batch == 0) return HEAL_OK;
    st = check_device();
    if (st != HEAL_OK) return st;

    heal::GemmArgs a;
    a.K = K;
    a.lda = lda;
    a.strideA = strideA;
    a.ldb = ldb;
    a.strideB = strideB;
    a.ldc = ldc;
    a.strideC = strideC;
    a.alpha = alpha;
    // 16-byte paths need every row start aligned: base pointer, leading
    // dimension and batch stride all multiples of 4 elements (the parts of
    // a cut call start at multiples of 256 rows and columns).
    a.vecA = aligned16(A) && lda % 4 == 0 && (batch == 1 || strideA % 4 == 0);
    a.vecB = aligned16(B) && ldb % 4 == 0 && (batch == 1 || strideB % 4 == 0);
    a.vecC = aligned16(C) && ldc % 4 == 0 && (batch == 1 || strideC % 4 == 0);
    const bool use_alpha = alpha != 1.0f;
    return for_each_part(batch, M, N, [&](int64_t b0, int64_t bn, int64_t m0, int64_t mn,
                                         int64_t n0, int64_t nn) {
        a.M = mn;
        a.N = nn;
        a.batch = bn;
        a.A = A ? A + b0 * strideA + m0 * lda : A;   // null only when K == 0
        a.B = B ? B + b0 * strideB + (trans_b ? n0 * ldb : n0) : B;
        a.C = C + b0 * strideC + m0 * ldc + n0;
        const int inst = instance == HEAL_INSTANCE_AUTO ? select_instance(mn, nn) : instance;
        return heal::launch_gemm(inst, a, trans_b != 0, use_alpha, stream);
    });
}

// Packed operands: K bounded so that every byte offset inside one tile of
// packed B stays below 2^31 (16 blocks x ceil(K/32) chunks x 2 planes x 1 KiB).
constexpr int64_t kMaxPackedK = (int64_t)1 << 20;
constexpr int32_t kMaxExponent = 300;

// Products of an FP32 A with a packed B (HEAL-Base / HEAL-Full weights, the
// pre-split bf16 operand).
heal_status_t run_packed(int op, int instance, int64_t M, int64_t N, int64_t K, const float *A,
                         int64_t lda, const uint16_t *Bp, int32_t e, float *C, int64_t ldc,
                         hipStream_t stream)
{
    if (M < 0 || N < 0 || K < 0 || K > kMaxPackedK) return HEAL_ERR_INVALID_VALUE;
    const int64_t lim = (int64_t)1 << 48;
    if (M > lim || N > ((int64_t)1 << 40) || lda > lim || ldc > lim) return HEAL_ERR_INVALID_VALUE;
    if (lda < (K > 1 ? K : 1) || ldc < (N > 1 ? N : 1)) return HEAL_ERR_INVALID_VALUE;
    if (!product_fits(M, N)) return HEAL_ERR_INVALID_VALUE;
    if (instance < 0 || instance >= HEAL_INSTANCE_COUNT) return HEAL_ERR_INVALID_VALUE;
    if (M == 0 || N == 0) return HEAL_OK;
    if (!C || !aligned4(C)) return HEAL_ERR_INVALID_VALUE;
    if (K > 0 && (!A || !Bp || !aligned4(A) || !aligned16(Bp))) return HEAL_ERR_INVALID_VALUE;
    heal_status_t st = check_device();
    if (st != HEAL_OK) return st;
    heal::OpArgs a = {};
    a.K = K;
    a.lda = lda;
    a.ldc = ldc;
    a.batch = 1;
    a.e = e;
    a.alpha = 1.0f;
    a.vecA = aligned16(A) && lda % 4 == 0;
    a.vecC = aligned16(C) && ldc % 4 == 0;
    // packed B: a part starting at column n0 (a multiple of 16) starts at
    // column block n0 / 16, ceil(K/32) chunks of planes x 512 values each
    const int64_t block_vals = ((K + 31) / 32) * (op == heal::OP_PRESPLIT ? 2 : 1) * 512;
    return for_each_part(1, M, N, [&](int64_t, int64_t, int64_t m0, int64_t mn, int64_t n0,
                                      int64_t nn) {
        a.M = mn;
        a.N = nn;
        a.A = A ? A + m0 * lda : A;   // null only when K == 0
        a.B = Bp ? Bp + (n0 / 16) * block_vals : Bp;
        a.C = C + m0 * ldc + n0;
        return heal::launch_gemm_op(op, instance, a, stream);
    });
}

}  // namespace

extern "C" {

const char *heal_status_string(heal_status_t status)
{
    switch (status) {
    case HEAL_OK: return "HEAL_OK";
    case HEAL_ERR_INVALID_VALUE: return "HEAL_ERR_INVALID_VALUE";
    case HEAL_ERR_UNSUPPORTED_DEVICE: return "HEAL_ERR_UNSUPPORTED_DEVICE";
    case HEAL_ERR_LAUNCH: return "HEAL_ERR_LAUNCH";
    }
    return "HEAL_ERR_UNKNOWN";
}

int heal_version(void) { return 100; }

#ifndef HEAL_BUILD_ID
#define HEAL_BUILD_ID "unknown"
#endif
const char *heal_build_id(void) { return HEAL_BUILD_ID; }

heal_status_t heal_split_f32(const float *x, uint16_t *hi, uint16_t *lo, int64_t n,
                             hipStream_t stream)
{
    if (n < 0) return HEAL_ERR_INVALID_VALUE;
    if (n == 0) return HEAL_OK;
    if (!x || !hi || !lo || !aligned4(x) || (reinterpret_cast<uintptr_t>(hi) & 1u) ||
        (reinterpret_cast<uintptr_t>(lo) & 1u))
        return HEAL_ERR_INVALID_VALUE;
    heal_status_t st = check_device();
    if (st != HEAL_OK) return st;
    return heal::launch_split(x, hi, lo, n, stream) == hipSuccess ? HEAL_OK : HEAL_ERR_LAUNCH;
}

heal_status_t heal_gemm_f32(int64_t M, int64_t N, int64_t K, const float *A, const float *B,
                            float *C, int64_t lda, int64_t ldb, int64_t ldc, hipStream_t stream)
{
    return run_gemm(HEAL_INSTANCE_AUTO, M, N, K, 1.0f, A, lda, 0, B, ldb, 0, 0, C, ldc, 0, 1,
                    stream);
}

heal_status_t heal_gemm_f32_strided_batched(int64_t M, int64_t N, int64_t K, float alpha,
                                            const float *A, int64_t lda, int64_t strideA,
                                            const float *B, int64_t ldb, int64_t strideB,
                                            int trans_b, float *C, int64_t ldc, int64_t strideC,
                                            int64_t batch, hipStream_t stream)
{
    return run_gemm(HEAL_INSTANCE_AUTO, M, N, K, alpha, A, lda, strideA, B, ldb, strideB, trans_b,
                    C, ldc, strideC, batch, stream);
}

heal_status_t heal_gemm_f32_instance(int instance, int64_t M, int64_t N, int64_t K, float alpha,
                                     const float *A, int64_t lda, int64_t strideA, const float *B,
                                     int64_t ldb, int64_t strideB, int trans_b, float *C,
                                     int64_t ldc, int64_t strideC, int64_t batch,
                                     hipStream_t stream)
{
    return run_gemm(instance, M, N, K, alpha, A, lda, strideA, B, ldb, strideB, trans_b, C, ldc,
                    strideC, batch, stream);
}

int heal_gemm_select_instance(int64_t M, int64_t N) { return select_instance(M, N); }

// ---- FP16 forms, pre-split operand, INT16 scores ----------------------------

heal_status_t heal_split_f16(const float *x, uint16_t *hi, uint16_t *lo, int64_t n,
                             hipStream_t stream)
{
    if (n < 0) return HEAL_ERR_INVALID_VALUE;
    if (n == 0) return HEAL_OK;
    if (!x || !hi || !lo || !aligned4(x) || (reinterpret_cast<uintptr_t>(hi) & 1u) ||
        (reinterpret_cast<uintptr_t>(lo) & 1u))
        return HEAL_ERR_INVALID_VALUE;
    heal_status_t st = check_device();
    if (st != HEAL_OK) return st;
    return heal::launch_split_f16(x, hi, lo, n, stream) == hipSuccess ? HEAL_OK : HEAL_ERR_LAUNCH;
}

int64_t heal_packed_size(int64_t K, int64_t N, int planes)
{
    if (K < 0 || N < 0 || (planes != 1 && planes != 2) || K > kMaxPackedK || N > ((int64_t)1 << 40))
        return -1;
    return ((N + 15) / 16) * ((K + 31) / 32) * planes * 512;
}

heal_status_t heal_maxabs_f32(const float *x, int64_t rows, int64_t cols, int64_t ld,
                              float *maxabs, hipStream_t stream)
{
    if (rows < 0 || cols < 0 || ld < (cols > 1 ? cols : 1) || !maxabs || !aligned4(maxabs))
        return HEAL_ERR_INVALID_VALUE;
    if (rows > ((int64_t)1 << 40) || ld > ((int64_t)1 << 40) || !product_fits(rows, ld))
        return HEAL_ERR_INVALID_VALUE;
    if (rows > 0 && cols > 0 && (!x || !aligned4(x))) return HEAL_ERR_INVALID_VALUE;
    heal_status_t st = check_device();
    if (st != HEAL_OK) return st;
    return heal::launch_maxabs(x, rows, cols, ld, maxabs, stream) == hipSuccess ? HEAL_OK
                                                                                 : HEAL_ERR_LAUNCH;
}

heal_status_t heal_f16_weight_exponent(float maxabs, int32_t *e)
{
    if (!e || !(maxabs >= 0.0f) || maxabs > 3.4028235e38f) return HEAL_ERR_INVALID_VALUE;
    if (maxabs == 0.0f) {
        *e = 0;
        return HEAL_OK;
    }
    // maxabs = f * 2^E with f in [1/2, 1), and 65504 = (1 - 2^-11) * 2^16.
    // If f <= 1 - 2^-11, then f * 2^16 <= 65504 while f * 2^17 >= 2^16 does
    // not fit: the exponent is 16 - E.  Otherwise f * 2^16 > 65504 and
    // f * 2^15 < 2^15 fits: it is 15 - E.
    int E = 0;
    const float f = frexpf(maxabs, &E);
    *e = (f <= 1.0f - 0x1p-11f ? 16 : 15) - E;
    return HEAL_OK;
}

heal_status_t heal_pack_f16_weight(const float *W, int64_t N, int64_t K, int64_t ldw, int32_t e,
                                   uint16_t *W16, hipStream_t stream)
{
    if (N < 0 || K < 0 || K > kMaxPackedK || N > ((int64_t)1 << 40) ||
        ldw < (K > 1 ? K : 1) || e < -kMaxExponent || e > kMaxExponent)
        return HEAL_ERR_INVALID_VALUE;
    if (N == 0 || K == 0) return HEAL_OK;
    if (!W || !W16 || !aligned4(W) || !aligned16(W16)) return HEAL_ERR_INVALID_VALUE;
    heal_status_t st = check_device();
    if (st != HEAL_OK) return st;
    return heal::launch_pack(0, W, K, N, ldw, true, e, W16, stream) == hipSuccess
               ? HEAL_OK
               : HEAL_ERR_LAUNCH;
}

heal_status_t heal_presplit_b(const float *B, int64_t K, int64_t N, int64_t ldb, int trans_b,
                              uint16_t *Bp, hipStream_t stream)
{
    if (N < 0 || K < 0 || K > kMaxPackedK || N > ((int64_t)1 << 40) ||
        (trans_b != 0 && trans_b != 1))
        return HEAL_ERR_INVALID_VALUE;
    if (ldb < (trans_b ? (K > 1 ? K : 1) : (N > 1 ? N : 1))) return HEAL_ERR_INVALID_VALUE;
    if (N == 0 || K == 0) return HEAL_OK;
    if (!B || !Bp || !aligned4(B) || !aligned16(Bp)) return HEAL_ERR_INVALID_VALUE;
    heal_status_t st = check_device();
    if (st != HEAL_OK) return st;
    return heal::launch_pack(1, B, K, N, ldb, trans_b != 0, 0, Bp, stream) == hipSuccess
               ? HEAL_OK
               : HEAL_ERR_LAUNCH;
}

heal_status_t heal_gemm_f16w_instance(int instance, int products, int64_t M, int64_t N,
                                      int64_t K, const float *A, int64_t lda,
                                      const uint16_t *W16, int32_t e, float *C, int64_t ldc,
                                      hipStream_t stream)
{
    if (products != 1 && products != 2) return HEAL_ERR_INVALID_VALUE;
    if (e < -kMaxExponent || e > kMaxExponent) return HEAL_ERR_INVALID_VALUE;
    return run_packed(products == 1 ? heal::OP_BASE : heal::OP_FULL, instance, M, N, K, A, lda,
                      W16, e, C, ldc, stream);
}

heal_status_t heal_gemm_f16w(int products, int64_t M, int64_t N, int64_t K, const float *A,
                             int64_t lda, const uint16_t *W16, int32_t e, float *C, int64_t ldc,
                             hipStream_t stream)
{
    return heal_gemm_f16w_instance(HEAL_INSTANCE_AUTO, products, M, N, K, A, lda, W16, e, C, ldc,
                                   stream);
}

heal_status_t heal_gemm_f32_presplit_instance(int instance, int64_t M, int64_t N, int64_t K,
                                              const float *A, int64_t lda, const uint16_t *Bp,
                                              float *C, int64_t ldc, hipStream_t stream)
{
    return run_packed(heal::OP_PRESPLIT, instance, M, N, K, A, lda, Bp, 0, C, ldc, stream);
}

heal_status_t heal_gemm_f32_presplit(int64_t M, int64_t N, int64_t K, const float *A, int64_t lda,
                                     const uint16_t *Bp, float *C, int64_t ldc, hipStream_t stream)
{
    return run_packed(heal::OP_PRESPLIT, HEAL_INSTANCE_AUTO, M, N, K, A, lda, Bp, 0, C, ldc,
                      stream);
}

heal_status_t heal_quantize_i16(const float *x, int64_t n, int16_t *q, float *maxabs,
                                hipStream_t stream)
{
    if (n < 0 || n > ((int64_t)1 << 40) || !maxabs || !aligned4(maxabs))
        return HEAL_ERR_INVALID_VALUE;
    if (n > 0 && (!x || !q || !aligned4(x) || (reinterpret_cast<uintptr_t>(q) & 1u)))
        return HEAL_ERR_INVALID_VALUE;
    heal_status_t st = check_device();
    if (st != HEAL_OK) return st;
    return heal::launch_quantize(x, n, q, maxabs, stream) == hipSuccess ? HEAL_OK
                                                                        : HEAL_ERR_LAUNCH;
}

heal_status_t heal_scores_i16(int64_t M, int64_t N, int64_t K, const int16_t *Q, int64_t ldq,
                              int64_t strideQ, const float *maxQ, const int16_t *Kt, int64_t ldk,
                              int64_t strideK, const float *maxK, float alpha, float *S,
                              int64_t lds, int64_t strideS, int64_t batch, hipStream_t stream)
{
    if (M < 0 || N < 0 || K < 0 || batch < 0) return HEAL_ERR_INVALID_VALUE;
    if (strideQ < 0 || strideK < 0 || strideS < 0) return HEAL_ERR_INVALID_VALUE;
    if (ldq < (K > 1 ? K : 1) || ldk < (K > 1 ? K : 1) || lds < (N > 1 ? N : 1))
        return HEAL_ERR_INVALID_VALUE;
    const int64_t lim = (int64_t)1 << 48;
    if (M > lim || N > lim || K > lim || ldq > lim || ldk > lim || lds > lim || batch > lim)
        return HEAL_ERR_INVALID_VALUE;
    if (!product_fits(M, N)) return HEAL_ERR_INVALID_VALUE;
    if (M == 0 || N == 0 || batch == 0) return HEAL_OK;
    if (!S || !aligned4(S) || !maxQ || !maxK || !aligned4(maxQ) || !aligned4(maxK))
        return HEAL_ERR_INVALID_VALUE;
    if (K > 0 && (!Q || !Kt || (reinterpret_cast<uintptr_t>(Q) & 1u) ||
                  (reinterpret_cast<uintptr_t>(Kt) & 1u)))
        return HEAL_ERR_INVALID_VALUE;
    heal_status_t st = check_device();
    if (st != HEAL_OK) return st;
    heal::OpArgs a = {};
    a.K = K;
    a.lda = ldq;
    a.strideA = strideQ;
    a.ldb = ldk;
    a.strideB = strideK;
    a.ldc = lds;
    a.strideC = strideS;
    a.maxA = maxQ;
    a.maxB = maxK;
    a.alpha = alpha;
    a.vecA = aligned16(Q) && ldq % 8 == 0 && (batch == 1 || strideQ % 8 == 0);
    a.vecB = aligned16(Kt) && ldk % 8 == 0 && (batch == 1 || strideK % 8 == 0);
    a.vecC = aligned16(S) && lds % 4 == 0 && (batch == 1 || strideS % 4 == 0);
    return for_each_part(batch, M, N, [&](int64_t b0, int64_t bn, int64_t m0, int64_t mn,
                                          int64_t n0, int64_t nn) {
        a.M = mn;
        a.N = nn;
        a.batch = bn;
        a.A = Q ? Q + b0 * strideQ + m0 * ldq : Q;   // null only when K == 0
        a.B = Kt ? Kt + b0 * strideK + n0 * ldk : Kt;
        a.C = S + b0 * strideS + m0 * lds + n0;
        return heal::launch_gemm_op(heal::OP_SCORES, HEAL_INSTANCE_AUTO, a, stream);
    });
}

}  // extern "C"
