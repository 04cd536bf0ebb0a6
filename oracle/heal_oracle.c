/*
 * heal_oracle.c -- plain, slow CPU oracle for the bf16x3 compensated GEMM.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or
 * load this file or the library built from it; only the test-suite, the smoke
 * check and the CPU-baseline leg of the benchmark use it.  It shares no code,
 * header, table or helper with the HIP library.
 *
 * What it computes (HEAL, Section 4 "Hybrid Error ALleviation", paragraph on
 * GEMM compensation, and its displayed GEMM expansion):
 *   - an FP32 operand is decomposed into a 16-bit head and a 16-bit residual;
 *     here the 16-bit format is bfloat16 for both operands, so
 *         hi = RNE_bf16(x),   lo = RNE_bf16(x - hi)
 *     (rounding is round-to-nearest-even, the hardware default the paper
 *     relies on in Section 3.3; bf16 keeps 7 explicit significand bits,
 *     Appendix A "Baselines");
 *   - the product is expanded into 16-bit products summed in high precision:
 *         S = hiA*hiB + hiA*loB + loA*hiB     (the loA*loB term is dropped),
 *     accumulated here in FP64, k ascending, the three terms in that order;
 *   - the output stays FP32 (Appendix "HEAL Implementation", HEAL-Base and
 *     HEAL-Full: GEMM outputs are kept in FP32):  C = (float)(alpha * S).
 *
 * Readings where the paper is silent (each is listed in the design notes):
 *   - the residual is evaluated exactly as defined, in IEEE arithmetic, for
 *     every input: an infinite x gives hi = x and lo = RNE(inf - inf) = NaN,
 *     a finite x that rounds to infinity gives lo = -/+inf, a NaN x gives NaN
 *     for both; so every output such an input reaches is NaN;
 *   - a NaN is rounded to the canonical quiet NaN with the NaN's sign;
 *   - no scaling of lo (bf16 has the FP32 exponent range, unlike the FP16
 *     variant of the paper, which scales its residual by 2^10).
 *
 * Pins (tests/test_oracle_pins.py): exhaustive comparison of the split against
 * an independent library RNE conversion over all 2^32 inputs; hand-derived
 * golden split and GEMM cases; bf16-representable inputs reduce to the plain
 * product; a constructed split gives exact(A*B) - S = sum lA*lB in closed form;
 * integer inputs give the exact integer GEMM; a brute-force error bound against
 * the exact product on tiny sizes.
 *
 * The second half of the file holds the FP16 forms of the method (HEAL-Base,
 * HEAL-Full) and the INT16 storage with dual-FP16 scores (HEAL+); their pins:
 * binary16 rounding against numpy's casts at every value and tie of the format,
 * the HEAL-Full pair exhaustively over all 2^32 FP32 inputs against library
 * casts, hand-derived golden pairs, the defining property of the weight
 * exponent, integer GEMMs, brute-force error bounds against exact rational
 * products, the exact identity hi + lo/2^10 = q over all INT16 codes, and the
 * paper's INT16 error and MSE-ratio bounds.
 * Build: gcc -O2 -fopenmp -ffp-contract=off.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

static uint32_t bits_of(float x) { uint32_t u; memcpy(&u, &x, 4); return u; }
static float float_of(uint32_t u) { float x; memcpy(&x, &u, 4); return x; }

/* Round an FP32 value to bfloat16, round-to-nearest, ties to even.  A bf16 is
 * the upper 16 bits of an FP32 pattern, so rounding looks at the 16 discarded
 * bits: above half an ulp rounds up, below rounds down, exactly half rounds to
 * the neighbour whose last kept bit is 0.  A carry out of the significand moves
 * into the exponent, which is how the largest values round up to infinity. */
uint16_t oracle_bf16_rne(float x)
{
    uint32_t u = bits_of(x);
    if ((u & 0x7fffffffu) > 0x7f800000u)              /* NaN: quiet, keep sign */
        return (uint16_t)(((u >> 16) & 0x8000u) | 0x7fc0u);
    uint32_t kept = u >> 16;
    uint32_t dropped = u & 0xffffu;
    if (dropped > 0x8000u || (dropped == 0x8000u && (kept & 1u)))
        kept += 1u;
    return (uint16_t)kept;
}

float oracle_bf16_to_float(uint16_t h) { return float_of((uint32_t)h << 16); }

/* The split of one element into (hi, lo) bf16 bit patterns. */
static void split_one(float x, uint16_t *hi, uint16_t *lo)
{
    uint16_t h = oracle_bf16_rne(x);
    float hf = oracle_bf16_to_float(h);
    float r = x - hf;   /* exact for finite hi: |r| <= half a bf16 step of x, on x's grid */
    *hi = h;
    *lo = oracle_bf16_rne(r);
}

void oracle_split(const float *x, uint16_t *hi, uint16_t *lo, int64_t n)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        split_one(x[i], &hi[i], &lo[i]);
}

/* Split the bit-pattern range [start, start+n) of FP32, for exhaustive tests. */
void oracle_split_range(uint32_t start, int64_t n, uint16_t *hi, uint16_t *lo)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        split_one(float_of(start + (uint32_t)i), &hi[i], &lo[i]);
}

/* Compensated product.  A is M x K (row stride lda), B is K x N (row stride
 * ldb), both row-major FP32.  If rows != NULL only the n_rows listed rows of A
 * are computed, and output row r corresponds to A row rows[r]; otherwise all M
 * rows are computed (n_rows is ignored).  S (FP64) and C (FP32) are n_out x N
 * row-major, contiguous.  Returns 0, or -1 on allocation failure. */
int oracle_gemm3(int64_t M, int64_t N, int64_t K,
                 const float *A, int64_t lda,
                 const float *B, int64_t ldb,
                 float alpha,
                 const int64_t *rows, int64_t n_rows,
                 double *S, float *C)
{
    int64_t n_out = rows ? n_rows : M;
    if (n_out <= 0 || N <= 0) return 0;
    float *bh = (float *)malloc(sizeof(float) * (size_t)(K > 0 ? K : 1) * (size_t)N);
    float *bl = (float *)malloc(sizeof(float) * (size_t)(K > 0 ? K : 1) * (size_t)N);
    if (!bh || !bl) { free(bh); free(bl); return -1; }

    /* split every element of B once */
#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < K; ++k) {
        for (int64_t j = 0; j < N; ++j) {
            uint16_t h, l;
            split_one(B[k * ldb + j], &h, &l);
            bh[k * N + j] = oracle_bf16_to_float(h);
            bl[k * N + j] = oracle_bf16_to_float(l);
        }
    }

    int failed = 0;
#pragma omp parallel
    {
        float *ah = (float *)malloc(sizeof(float) * (size_t)(K > 0 ? K : 1));
        float *al = (float *)malloc(sizeof(float) * (size_t)(K > 0 ? K : 1));
        if (!ah || !al) {
#pragma omp atomic write
            failed = 1;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int64_t r = 0; r < n_out; ++r) {
                int64_t i = rows ? rows[r] : r;
                for (int64_t k = 0; k < K; ++k) {
                    uint16_t h, l;
                    split_one(A[i * lda + k], &h, &l);
                    ah[k] = oracle_bf16_to_float(h);
                    al[k] = oracle_bf16_to_float(l);
                }
                double *s = S + r * N;
                for (int64_t j = 0; j < N; ++j) s[j] = 0.0;
                for (int64_t k = 0; k < K; ++k) {
                    double a_hi = ah[k], a_lo = al[k];
                    const float *bhk = bh + k * N, *blk = bl + k * N;
                    for (int64_t j = 0; j < N; ++j) {
                        double b_hi = bhk[j], b_lo = blk[j];
                        s[j] += a_hi * b_hi + a_hi * b_lo + a_lo * b_hi;
                    }
                }
                float *c = C + r * N;
                for (int64_t j = 0; j < N; ++j) c[j] = (float)((double)alpha * s[j]);
            }
        }
        free(ah);
        free(al);
    }
    free(bh);
    free(bl);
    return failed ? -1 : 0;
}


/* ------------------------------------------------------------------------
 * FP16 forms of the method.
 *
 * HEAL-Base and HEAL-Full (Appendix "HEAL Implementation"; Section 4, GEMM
 * paragraph and its displayed two-product expansion):
 *   - the weight matrix is scaled by a per-matrix power of two 2^e before it
 *     is cast to FP16, and the GEMM output is scaled back by 2^-e;
 *   - Base casts the FP32 activation once:  C = 2^-e * sum_k f16(a)*w16;
 *   - Full pairs two FP16 values per activation, a head h_hi = f16(h) and a
 *     residual shifted up by 2^10, h_lo = f16((h - h_hi) * 2^10), and adds the
 *     two products:  C = 2^-e * (sum_k h_hi*w16 + 2^-10 * sum_k h_lo*w16).
 * HEAL+ (Section 4, paragraph on Q/K/V truncation, and its displayed
 * attention expansion): a tensor X is stored as INT16 codes
 *   q = Round(32767 * x / max|X|)
 * and each code is unpacked into a dual-FP16 pair hi + lo/2^10 for the score
 * product (Q_hi + Q_lo/2^10)(K_hi + K_lo/2^10)^T, all four products kept.
 * ------------------------------------------------------------------------ */

/* Round a double to IEEE binary16, round-to-nearest, ties to even, written
 * from the format's definition: 1 sign bit, 5 exponent bits (bias 15), 10
 * fraction bits; normal numbers cover [2^-14, 65504], below that the spacing
 * is fixed at 2^-24 (subnormals); a magnitude of 65520 or more (half a step
 * above the largest finite value) rounds to infinity. */
uint16_t oracle_f16_rne(double x)
{
    uint16_t sign = signbit(x) ? 0x8000u : 0u;
    if (isnan(x)) return (uint16_t)(sign | 0x7e00u);
    double a = fabs(x);
    if (a >= 65520.0) return (uint16_t)(sign | 0x7c00u);
    if (a < 0x1p-14) {
        /* subnormal (or zero): an integer count of 2^-24 steps, 1024 = 2^-14 */
        double q = rint(a * 0x1p24);   /* exact scaling; rint rounds to even */
        return (uint16_t)(sign | (uint16_t)q);
    }
    int ex;
    frexp(a, &ex);                     /* a = f * 2^ex, f in [0.5, 1) */
    int E = ex - 1;                    /* a in [2^E, 2^(E+1)), -14 <= E <= 15 */
    double q = rint(ldexp(a, 10 - E)); /* significand with 10 fraction bits, in [1024, 2048] */
    if (q == 2048.0) { q = 1024.0; E += 1; }
    if (E > 15) return (uint16_t)(sign | 0x7c00u);
    return (uint16_t)(sign | (uint16_t)((E + 15) << 10) | (uint16_t)(q - 1024.0));
}

/* The value of a binary16 bit pattern. */
double oracle_f16_value(uint16_t h)
{
    int s = h >> 15, E = (h >> 10) & 0x1f, f = h & 0x3ff;
    double v;
    if (E == 0x1f) v = f ? NAN : INFINITY;
    else if (E == 0) v = ldexp((double)f, -24);
    else v = ldexp((double)(1024 + f), E - 25);
    return s ? -v : v;
}

/* HEAL-Full activation pair of one FP32 value.  The residual h - h_hi and its
 * 2^10 shift are evaluated exactly (FP64 holds them); an infinite or NaN head
 * makes the residual follow IEEE arithmetic (inf - inf = NaN). */
static void split_f16_one(float x, uint16_t *hi, uint16_t *lo)
{
    uint16_t h = oracle_f16_rne((double)x);
    double r = ((double)x - oracle_f16_value(h)) * 1024.0;
    *hi = h;
    *lo = oracle_f16_rne(r);
}

void oracle_split_f16(const float *x, uint16_t *hi, uint16_t *lo, int64_t n)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        split_f16_one(x[i], &hi[i], &lo[i]);
}

void oracle_split_f16_range(uint32_t start, int64_t n, uint16_t *hi, uint16_t *lo)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        split_f16_one(float_of(start + (uint32_t)i), &hi[i], &lo[i]);
}

/* The per-matrix weight exponent: the largest integer e with
 * maxabs * 2^e <= 65504 (the largest finite FP16), so the scaled weights use
 * the top of the FP16 range and none overflows; 0 for an all-zero matrix.
 * maxabs must be finite and >= 0. */
int32_t oracle_f16_weight_exponent(double maxabs)
{
    if (!(maxabs > 0.0)) return 0;
    int32_t e = 0;
    while (ldexp(maxabs, e) > 65504.0) --e;
    while (ldexp(maxabs, e + 1) <= 65504.0) ++e;
    return e;
}

/* The FP16 weight of one FP32 entry: RNE_f16(w * 2^e), the scaling exact in FP64. */
uint16_t oracle_f16_weight(float w, int32_t e) { return oracle_f16_rne(ldexp((double)w, e)); }

/* HEAL-Base (products == 1) or HEAL-Full (products == 2) GEMM.  A is M x K
 * FP32 (row stride lda); W is the FP32 weight, N x K (row stride ldw, the
 * layout of a linear layer's weight), so the product is A * W^T; e is the
 * weight exponent.  Sums run k ascending in FP64, head and residual sums kept
 * apart and combined at the end; C = (float)(2^-e * S).  Rows as in
 * oracle_gemm3.  Returns 0, or -1 on allocation failure / bad argument. */
int oracle_gemm_f16w(int products, int64_t M, int64_t N, int64_t K,
                     const float *A, int64_t lda, const float *W, int64_t ldw, int32_t e,
                     const int64_t *rows, int64_t n_rows, double *S, float *C)
{
    if (products != 1 && products != 2) return -1;
    int64_t n_out = rows ? n_rows : M;
    if (n_out <= 0 || N <= 0) return 0;
    double *w16 = (double *)malloc(sizeof(double) * (size_t)N * (size_t)(K > 0 ? K : 1));
    if (!w16) return -1;
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < N; ++j)
        for (int64_t k = 0; k < K; ++k)
            w16[j * K + k] = oracle_f16_value(oracle_f16_weight(W[j * ldw + k], e));

    int failed = 0;
#pragma omp parallel
    {
        double *ah = (double *)malloc(sizeof(double) * (size_t)(K > 0 ? K : 1));
        double *al = (double *)malloc(sizeof(double) * (size_t)(K > 0 ? K : 1));
        if (!ah || !al) {
#pragma omp atomic write
            failed = 1;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int64_t r = 0; r < n_out; ++r) {
                int64_t i = rows ? rows[r] : r;
                for (int64_t k = 0; k < K; ++k) {
                    uint16_t h, l;
                    split_f16_one(A[i * lda + k], &h, &l);
                    ah[k] = oracle_f16_value(h);
                    al[k] = oracle_f16_value(l);
                }
                for (int64_t j = 0; j < N; ++j) {
                    const double *w = w16 + j * K;
                    double s_hi = 0.0, s_lo = 0.0;
                    for (int64_t k = 0; k < K; ++k) s_hi += ah[k] * w[k];
                    if (products == 2)
                        for (int64_t k = 0; k < K; ++k) s_lo += al[k] * w[k];
                    double s = ldexp(s_hi + ldexp(s_lo, -10), -e);
                    S[r * N + j] = s;
                    C[r * N + j] = (float)s;
                }
            }
        }
        free(ah);
        free(al);
    }
    free(w16);
    return failed ? -1 : 0;
}

/* max|x| over n FP32 values (0 for n == 0). */
float oracle_maxabs(const float *x, int64_t n)
{
    float m = 0.0f;
    for (int64_t i = 0; i < n; ++i) {
        float a = fabsf(x[i]);
        if (a > m) m = a;
    }
    return m;
}

/* INT16 codes of a tensor: q = Round(32767 * x / max|X|), Round taking the
 * real quotient to the nearest integer, ties to even.
 *
 * Evaluated as rint((32767 * x) / m) in FP64, which is that exact rounding:
 *   - 32767 * x is exact (15 by 24 significant bits);
 *   - write x = X 2^a with X an integer, |X| < 2^24, 2^a the last place of x;
 *     |m| >= |x| puts m on the same grid, m = Y 2^a with Y an integer >= |X|;
 *   - a half-integer n + 1/2 that the quotient t = 32767 X / Y does not equal
 *     lies at least 1/(2Y) away from it (their difference is an integer over
 *     2Y), while the one rounding of the FP64 division moves t by at most
 *     2^-53 |t| < 2^-53 2^15 2^24 / Y = 2^-14 / Y;
 *   - a quotient that is a half-integer (at most 17 bits) is representable and
 *     the division returns it exactly, so rint sees the tie and takes the even
 *     neighbour.
 * The quotient never exceeds 32767 in magnitude, so no range is lost for any
 * m, however small.  An all-zero tensor (m == 0) gives all-zero codes.  x
 * must be finite.  Writes max|X| to *maxabs. */
void oracle_quantize_i16(const float *x, int64_t n, int16_t *q, float *maxabs)
{
    float m = oracle_maxabs(x, n);
    for (int64_t i = 0; i < n; ++i) {
        double t = m > 0.0f ? (32767.0 * (double)x[i]) / (double)m : 0.0;
        q[i] = (int16_t)rint(t);
    }
    *maxabs = m;
}

/* The dequantisation of the score product: a code q of a tensor with maximum
 * m stands for q * m / 32767, so the scores of codes qQ, qK are
 *   alpha * (maxQ / 32767) * (maxK / 32767) * sum_k qQ qK;
 * this returns the factor in front of the sum, in FP64 (alpha * maxQ is exact,
 * the rest rounds three times, relative error below 2^-51). */
double oracle_scores_factor(float maxQ, float maxK, float alpha)
{
    return (double)alpha * (double)maxQ * (double)maxK / (32767.0 * 32767.0);
}

/* The dual-FP16 pair of one INT16 code: hi = f16(q), lo = 2^10 * (q - hi);
 * hi is an integer of 11 significant bits, q - hi an integer with
 * |q - hi| <= 8, so hi + lo / 2^10 == q exactly and both are exact FP16. */
void oracle_unpack_i16(int16_t q, uint16_t *hi, uint16_t *lo)
{
    uint16_t h = oracle_f16_rne((double)q);
    *hi = h;
    *lo = oracle_f16_rne(((double)q - oracle_f16_value(h)) * 1024.0);
}

/* Attention scores from INT16 Q (M x K, row stride ldq) and K (N x K, row
 * stride ldk), the contraction over the head dimension K:
 *   S_ij = sum_k (Qhi + Qlo/2^10)(Khi + Klo/2^10), the four products in the
 *          order hi*hi, hi*lo, lo*hi, lo*lo, k ascending, in FP64 (exact: every
 *          term is an integer or a multiple of 2^-20 well inside 2^53);
 *   factor = oracle_scores_factor(maxQ, maxK, alpha), in FP64;
 *   C_ij = (float)(factor * S_ij).
 * Rows as in oracle_gemm3.  Returns 0, or -1 on allocation failure. */
int oracle_scores_i16(int64_t M, int64_t N, int64_t K,
                      const int16_t *Q, int64_t ldq, const int16_t *Kt, int64_t ldk,
                      float maxQ, float maxK, float alpha,
                      const int64_t *rows, int64_t n_rows, double *S, float *C)
{
    int64_t n_out = rows ? n_rows : M;
    if (n_out <= 0 || N <= 0) return 0;
    double factor = oracle_scores_factor(maxQ, maxK, alpha);
    size_t kk = (size_t)(K > 0 ? K : 1);
    double *kh = (double *)malloc(sizeof(double) * (size_t)N * kk);
    double *kl = (double *)malloc(sizeof(double) * (size_t)N * kk);
    if (!kh || !kl) { free(kh); free(kl); return -1; }
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < N; ++j)
        for (int64_t k = 0; k < K; ++k) {
            uint16_t h, l;
            oracle_unpack_i16(Kt[j * ldk + k], &h, &l);
            kh[j * K + k] = oracle_f16_value(h);
            kl[j * K + k] = oracle_f16_value(l) / 1024.0;
        }
    int failed = 0;
#pragma omp parallel
    {
        double *qh = (double *)malloc(sizeof(double) * kk);
        double *ql = (double *)malloc(sizeof(double) * kk);
        if (!qh || !ql) {
#pragma omp atomic write
            failed = 1;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int64_t r = 0; r < n_out; ++r) {
                int64_t i = rows ? rows[r] : r;
                for (int64_t k = 0; k < K; ++k) {
                    uint16_t h, l;
                    oracle_unpack_i16(Q[i * ldq + k], &h, &l);
                    qh[k] = oracle_f16_value(h);
                    ql[k] = oracle_f16_value(l) / 1024.0;
                }
                for (int64_t j = 0; j < N; ++j) {
                    const double *bh = kh + j * K, *bl = kl + j * K;
                    double s = 0.0;
                    for (int64_t k = 0; k < K; ++k)
                        s += qh[k] * bh[k] + qh[k] * bl[k] + ql[k] * bh[k] + ql[k] * bl[k];
                    S[r * N + j] = s;
                    C[r * N + j] = (float)(factor * s);
                }
            }
        }
        free(qh);
        free(ql);
    }
    free(kh);
    free(kl);
    return failed ? -1 : 0;
}

/* Element-wise helpers for the tests: binary16 rounding of doubles, and the
 * FP16 weights RNE_f16(W * 2^e) of an N x K weight (row stride ldw), written
 * N x K contiguous. */
void oracle_f16_rne_array(const double *x, uint16_t *out, int64_t n)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_f16_rne(x[i]);
}

void oracle_f16_weights(const float *W, int64_t N, int64_t K, int64_t ldw, int32_t e,
                        uint16_t *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < N; ++j)
        for (int64_t k = 0; k < K; ++k) out[j * K + k] = oracle_f16_weight(W[j * ldw + k], e);
}

void oracle_unpack_i16_array(const int16_t *q, uint16_t *hi, uint16_t *lo, int64_t n)
{
    for (int64_t i = 0; i < n; ++i) oracle_unpack_i16(q[i], &hi[i], &lo[i]);
}

int oracle_num_threads(void) { return omp_get_max_threads(); }
