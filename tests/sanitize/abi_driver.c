/* Sanitizer driver for the C ABI's host side (test infrastructure): every
 * entry point called with arguments its validation must reject before any
 * HIP call (so no GPU is needed), plus the size and name queries; each status
 * is checked.  Built and run by tests/test_sanitizers.py against a build of
 * the library whose host code carries AddressSanitizer and
 * UndefinedBehaviorSanitizer. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "../../include/reqat.h"

static int fails = 0;
#define EXPECT(call, st)                                                                        \
    do {                                                                                        \
        reqat_status got_ = (call);                                                             \
        if (got_ != (st)) {                                                                     \
            printf("line %d: %s -> %d, expected %d\n", __LINE__, #call, (int)got_, (int)(st)); \
            ++fails;                                                                            \
        }                                                                                       \
    } while (0)

int main(void)
{
    /* never dereferenced: validation rejects before any use */
    void *P = (void *)(uintptr_t)(1u << 20);
    uint8_t *U = (uint8_t *)P;
    float *F = (float *)P;
    const reqat_format NV = REQAT_FMT_NVFP4, MX = REQAT_FMT_MXFP4;
    int s;
    for (s = 0; s < 9; s++)
        if (!reqat_status_str((reqat_status)s) || !strlen(reqat_status_str((reqat_status)s))) ++fails;
    if (reqat_abi_version() != REQAT_ABI_VERSION) ++fails;
    if (reqat_workspace_bytes() == 0) ++fails;
    if (reqat_linear_workspace_bytes(NV, 16, 5120) == 0 || reqat_linear_workspace_bytes(NV, 16, 100) != 0) ++fails;
    if (reqat_linear_workspace_bytes((reqat_format)7, 16, 5120) != 0) ++fails;
    if (reqat_w4a16_workspace_bytes(-1, 5, 128) != 0) ++fails;
    (void)reqat_w4a16_workspace_bytes(16, 5120, 27648);

    EXPECT(reqat_quantize_fp4((reqat_format)3, P, 4, 64, 64, U, U, F, REQAT_TS_COMPUTE, P, 0), REQAT_E_ENUM);
    EXPECT(reqat_quantize_fp4(NV, P, -1, 64, 64, U, U, F, REQAT_TS_COMPUTE, P, 0), REQAT_E_SHAPE);
    EXPECT(reqat_quantize_fp4(NV, P, 4, 40, 64, U, U, F, REQAT_TS_COMPUTE, P, 0), REQAT_E_SHAPE);
    EXPECT(reqat_quantize_fp4(NV, P, 4, 64, 32, U, U, F, REQAT_TS_COMPUTE, P, 0), REQAT_E_SHAPE);
    EXPECT(reqat_quantize_fp4(MX, P, 4, 64, 64, U, U, F, REQAT_TS_COMPUTE, 0, 0), REQAT_E_UNSUPPORTED);
    EXPECT(reqat_quantize_fp4(NV, P, 4, 64, 64, U, U, 0, REQAT_TS_COMPUTE, P, 0), REQAT_E_NULL);
    EXPECT(reqat_quantize_fp4(NV, (char *)P + 2, 4, 64, 64, U, U, F, REQAT_TS_COMPUTE, P, 0), REQAT_E_ALIGN);
    EXPECT(reqat_quantize_fp4(NV, P, 4, 64, 68, U, U, F, REQAT_TS_COMPUTE, P, 0), REQAT_E_ALIGN);
    EXPECT(reqat_fakequant_fp4(NV, P, 4, 64, 64, 0, 64, F, REQAT_TS_GIVEN, 0, 0), REQAT_E_NULL);
    EXPECT(reqat_fakequant_fp4(NV, P, 4, 64, 64, P, 64, F, REQAT_TS_COMPUTE, P, 0), REQAT_E_UNSUPPORTED);
    EXPECT(reqat_quantize_fakequant_fp4(NV, P, 4, 64, 64, U, U, P, 64, F, REQAT_TS_COMPUTE, P, 0),
           REQAT_E_UNSUPPORTED);
    EXPECT(reqat_quantize_mxfp4_rht(P, 4, 48, 48, 1u, U, U, 0), REQAT_E_SHAPE);
    EXPECT(reqat_quantize_mxfp4_rht(0, 4, 64, 64, 1u, U, U, 0), REQAT_E_NULL);
    EXPECT(reqat_fakequant_mxfp4_rht(P, 4, 64, 64, 1u, (char *)P + 2, 64, 0), REQAT_E_ALIGN);
    EXPECT(reqat_gemm_w4a4((reqat_format)9, 4, 8, 128, U, U, F, U, U, F, P, REQAT_DT_F32, 8, 0), REQAT_E_ENUM);
    EXPECT(reqat_gemm_w4a4(NV, 4, 8, 96, U, U, F, U, U, F, P, REQAT_DT_F32, 8, 0), REQAT_E_SHAPE);
    EXPECT(reqat_gemm_w4a4(NV, 4, 8, 128, U, U, F, U, U, F, P, REQAT_DT_F32, 4, 0), REQAT_E_SHAPE);
    EXPECT(reqat_gemm_w4a4(NV, 4, 8, 128, 0, U, F, U, U, F, P, REQAT_DT_F32, 8, 0), REQAT_E_NULL);
    EXPECT(reqat_gemm_w4a4(MX, 4, 8, 128, U, U, F, U, U, 0, P, REQAT_DT_F32, 8, 0), REQAT_E_UNSUPPORTED);
    EXPECT(reqat_gemm_w4a4(NV, 4, 8, 128, U + 4, U, F, U, U, F, P, REQAT_DT_F32, 8, 0), REQAT_E_ALIGN);
    EXPECT(reqat_gemm_w4a4(NV, 4, 8, 128, U, U, F, U, U, F, P, (reqat_dtype)5, 8, 0), REQAT_E_ENUM);
    EXPECT(reqat_gemm_w4a16(4, 8, 96, P, 96, U, U, P, REQAT_DT_F32, 8, 0, 0), REQAT_E_SHAPE);
    EXPECT(reqat_gemm_w4a16(4, 8, 128, 0, 128, U, U, P, REQAT_DT_F32, 8, 0, 0), REQAT_E_NULL);
    EXPECT(reqat_quantize_kv4(P, 4, 40, 40, 0, U, U, F, REQAT_TS_COMPUTE, P, 0), REQAT_E_SHAPE);
    EXPECT(reqat_quantize_kv4(P, 4, 64, 64, (float *)((char *)P + 4), U, U, F, REQAT_TS_COMPUTE, P, 0),
           REQAT_E_ALIGN);
    EXPECT(reqat_fakequant_kv4(P, 4, 64, 64, 0, P, 64, 0, REQAT_TS_GIVEN, 0, 0), REQAT_E_NULL);
    EXPECT(reqat_sem_loss(P, 4, 100, 104, (int32_t *)P, 0.5f, 1e-6f, F, F, F, 0), REQAT_E_SHAPE);
    EXPECT(reqat_sem_loss(0, 4, 128, 128, (int32_t *)P, 0.5f, 1e-6f, F, F, F, 0), REQAT_E_NULL);
    EXPECT(reqat_sem_loss_backward(P, 4, 128, 128, (int32_t *)P, F, F, 0.5f, 1.0f, P, (reqat_dtype)4, 128, 0),
           REQAT_E_ENUM);
    EXPECT(reqat_linear_w4a4(NV, 4, 8, 128, P, 128, F, REQAT_TS_COMPUTE, U, U, F, P, REQAT_DT_F32, 8, 0, 0),
           REQAT_E_NULL);
    EXPECT(reqat_linear_w4a4(NV, 4, 8, 128, P, 128, F, REQAT_TS_COMPUTE, U, U, F, P, REQAT_DT_F32, 8,
                             (char *)P + 16, 0),
           REQAT_E_ALIGN);
    EXPECT(reqat_linear_w4a4_noalloc(NV, 4, 8, 100, P, 128, F, REQAT_TS_COMPUTE, U, U, F, P, REQAT_DT_F32, 8, 0),
           REQAT_E_SHAPE);
    EXPECT(reqat_linear_w4a4_noalloc(NV, 1 << 20, 8, 5120, P, 5120, F, REQAT_TS_COMPUTE, U, U, F, P, REQAT_DT_F32,
                                     8, 0),
           REQAT_E_TOO_LARGE);
    /* packed weight images: sizes, and every rejection before a launch (overlap included) */
    if (reqat_w4a16_packed_bytes(17, 256) != 2 * 2 * 1088 || reqat_w4a16_packed_bytes(16, 100) != 0) ++fails;
    if (reqat_w4a4_packed_bytes(NV, 8960, 1536) != (size_t)560 * 6 * 2304 ||
        reqat_w4a4_packed_bytes(MX, 17, 384) != (size_t)2 * 2 * 2176 ||
        reqat_w4a4_packed_bytes((reqat_format)7, 16, 128) != 0 || reqat_w4a4_packed_bytes(NV, -1, 128) != 0)
        ++fails;
    EXPECT(reqat_pack_w4a16(U, U, 8, 96, P, 0), REQAT_E_SHAPE);
    EXPECT(reqat_pack_w4a16(0, U, 8, 128, P, 0), REQAT_E_NULL);
    EXPECT(reqat_pack_w4a16(U, U + 2, 8, 128, U + 4096, 0), REQAT_E_ALIGN);
    EXPECT(reqat_pack_w4a16(U, U + 4096, 8, 128, U + 256, 0), REQAT_E_UNSUPPORTED);
    EXPECT(reqat_gemm_w4a16_packed(4, 8, 128, P, 128, 0, P, REQAT_DT_F32, 8, 0, 0), REQAT_E_NULL);
    EXPECT(reqat_pack_w4a4((reqat_format)7, U, U, 8, 128, P, 0), REQAT_E_ENUM);
    EXPECT(reqat_pack_w4a4(NV, U, U, 8, 96, P, 0), REQAT_E_SHAPE);
    EXPECT(reqat_pack_w4a4(NV, U, 0, 8, 128, P, 0), REQAT_E_NULL);
    EXPECT(reqat_pack_w4a4(NV, U, U + 8, 8, 128, U + 8192, 0), REQAT_E_ALIGN);
    EXPECT(reqat_pack_w4a4(NV, U, U + 8192, 8, 128, U + 256, 0), REQAT_E_UNSUPPORTED);
    EXPECT(reqat_pack_w4a4(MX, U + 8192, U, 8, 128, U + 16, 0), REQAT_E_UNSUPPORTED);
    EXPECT(reqat_gemm_w4a4_packed(NV, 65, 8, 128, U, U, F, P, F, P, REQAT_DT_F32, 8, 0), REQAT_E_UNSUPPORTED);
    EXPECT(reqat_gemm_w4a4_packed(MX, 4, 8, 128, U, U, F, P, 0, P, REQAT_DT_F32, 8, 0), REQAT_E_UNSUPPORTED);
    EXPECT(reqat_gemm_w4a4_packed(NV, 4, 8, 128, U, U, F, 0, F, P, REQAT_DT_F32, 8, 0), REQAT_E_NULL);
    EXPECT(reqat_gemm_w4a4_packed(NV, 4, 8, 128, U, U, F, U + 8, F, P, REQAT_DT_F32, 8, 0), REQAT_E_ALIGN);
    EXPECT(reqat_gemm_w4a4_packed(NV, 4, 8, 128, U, U, F, P, F, P, REQAT_DT_F32, 4, 0), REQAT_E_SHAPE);
    EXPECT(reqat_linear_w4a4_packed(NV, 65, 8, 128, P, 128, F, REQAT_TS_GIVEN, P, F, P, REQAT_DT_F32, 8, P, 0),
           REQAT_E_UNSUPPORTED);
    EXPECT(reqat_linear_w4a4_packed(NV, 4, 8, 128, P, 128, F, REQAT_TS_GIVEN, P, F, P, REQAT_DT_F32, 8, 0, 0),
           REQAT_E_NULL);
    EXPECT(reqat_linear_w4a4_packed(NV, 4, 8, 128, P, 128, F, REQAT_TS_GIVEN, P, F, P, REQAT_DT_F32, 8,
                                    (char *)P + 16, 0),
           REQAT_E_ALIGN);
    EXPECT(reqat_linear_w4a4_packed(NV, 4, 8, 128, P, 128, F, (reqat_tscale_mode)3, P, F, P, REQAT_DT_F32, 8, P, 0),
           REQAT_E_ENUM);
    if (fails) {
        printf("%d failures\n", fails);
        return 1;
    }
    printf("abi driver ok\n");
    return 0;
}
