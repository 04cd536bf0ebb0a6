/* Plain-C user of include/heal.h: compiles as C11 against the header, links
 * libheal.so, and exercises the host-side contract that needs no GPU
 * (status strings, version, argument validation, packed sizes, the weight
 * exponent).  Exit status 0 on success; prints the first failed check. */
#include <stdio.h>
#include <string.h>

#include "heal.h"

#define CHECK(cond)                                                      \
    do {                                                                 \
        if (!(cond)) {                                                   \
            fprintf(stderr, "abi_check: failed: %s (line %d)\n", #cond, __LINE__); \
            return 1;                                                    \
        }                                                                \
    } while (0)

int main(void)
{
    float *fake = (float *)(void *)0x10000;   /* never dereferenced */
    uint16_t *fake16 = (uint16_t *)(void *)0x10000;
    int32_t e = 0;

    CHECK(heal_version() >= 100);
    CHECK(strcmp(heal_status_string(HEAL_OK), "HEAL_OK") == 0);
    CHECK(strcmp(heal_status_string(HEAL_ERR_INVALID_VALUE), "HEAL_ERR_INVALID_VALUE") == 0);

    /* validation happens before any HIP call */
    CHECK(heal_gemm_f32(4, 4, 8, fake, fake, fake, 7, 4, 4, 0) == HEAL_ERR_INVALID_VALUE);
    CHECK(heal_gemm_f32(0, 4, 4, 0, 0, 0, 4, 4, 4, 0) == HEAL_OK);
    CHECK(heal_gemm_f32_strided_batched(4, 8, 16, 1.0f, fake, 16, 64, fake, 8, 128, 2, fake, 8, 32,
                                        1, 0) == HEAL_ERR_INVALID_VALUE);
    CHECK(heal_gemm_f32_instance(HEAL_INSTANCE_COUNT, 4, 4, 4, 1.0f, fake, 4, 0, fake, 4, 0, 0,
                                 fake, 4, 0, 1, 0) == HEAL_ERR_INVALID_VALUE);
    CHECK(heal_split_f32(fake, fake16, fake16, -1, 0) == HEAL_ERR_INVALID_VALUE);
    CHECK(heal_gemm_select_instance(16, 4096) == HEAL_INSTANCE_SKINNY);
    CHECK(heal_gemm_select_instance(8192, 8192) == HEAL_INSTANCE_LARGE);

    CHECK(heal_packed_size(33, 17, 1) == 2 * 2 * 1 * 512);
    CHECK(heal_packed_size(4096, 4096, 2) == 256 * 128 * 2 * 512);
    CHECK(heal_packed_size(10, 10, 3) == -1);
    CHECK(heal_f16_weight_exponent(1.0f, &e) == HEAL_OK && e == 15);
    CHECK(heal_f16_weight_exponent(65504.0f, &e) == HEAL_OK && e == 0);
    CHECK(heal_f16_weight_exponent(-1.0f, &e) == HEAL_ERR_INVALID_VALUE);
    CHECK(heal_gemm_f16w(3, 4, 8, 16, fake, 16, fake16, 0, fake, 8, 0) == HEAL_ERR_INVALID_VALUE);
    CHECK(heal_gemm_f16w(2, 0, 8, 16, 0, 16, 0, 0, 0, 8, 0) == HEAL_OK);
    CHECK(heal_gemm_f32_presplit(4, 8, 16, fake, 15, fake16, fake, 8, 0) == HEAL_ERR_INVALID_VALUE);
    CHECK(heal_quantize_i16(fake, -1, (int16_t *)fake16, fake, 0) == HEAL_ERR_INVALID_VALUE);
    CHECK(heal_scores_i16(4, 8, 16, (int16_t *)fake16, 15, 0, fake, (int16_t *)fake16, 16, 0,
                          fake, 1.0f, fake, 8, 0, 1, 0) == HEAL_ERR_INVALID_VALUE);
    printf("abi_check: ok\n");
    return 0;
}
