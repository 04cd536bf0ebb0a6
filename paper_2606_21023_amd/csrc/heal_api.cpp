// C ABI of libheal.so: argument validation, device check, instance choice.
// Every argument check runs before the first HIP call.
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
    if (instance == HEAL_INSTANCE_AUTO) instance = select_instance(M, N);

    heal::GemmArgs a;
    a.M = M;
    a.N = N;
    a.K = K;
    a.A = A;
    a.lda = lda;
    a.strideA = strideA;
    a.B = B;
    a.ldb = ldb;
    a.strideB = strideB;
    a.C = C;
    a.ldc = ldc;
    a.strideC = strideC;
    a.batch = batch;
    a.alpha = alpha;
    // 16-byte paths need every row start aligned: base pointer, leading
    // dimension and batch stride all multiples of 4 elements.
    a.vecA = aligned16(A) && lda % 4 == 0 && (batch == 1 || strideA % 4 == 0);
    a.vecB = aligned16(B) && ldb % 4 == 0 && (batch == 1 || strideB % 4 == 0);
    a.vecC = aligned16(C) && ldc % 4 == 0 && (batch == 1 || strideC % 4 == 0);
    const bool use_alpha = alpha != 1.0f;
    hipError_t e = heal::launch_gemm(instance, a, trans_b != 0, use_alpha, stream);
    return e == hipSuccess ? HEAL_OK : HEAL_ERR_LAUNCH;
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

}  // extern "C"
