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
 * the exact product on tiny sizes.  Build: gcc -O2 -fopenmp -ffp-contract=off.
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

int oracle_num_threads(void) { return omp_get_max_threads(); }
