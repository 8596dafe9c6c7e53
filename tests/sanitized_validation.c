/* Argument validation of the C ABI under AddressSanitizer and
 * UndefinedBehaviorSanitizer (linked against libmasq_sanitized.so).  Every
 * call below is rejected (or is an empty batch) before the library touches
 * the GPU, so no device is needed.  Fake device addresses are never
 * dereferenced.  Prints "ok" and exits 0 when every status matches. */
#include <stdint.h>
#include <stdio.h>

#include "masq.h"

static int failures = 0;

static void expect(const char* what, masq_status got, masq_status want) {
    if (got != want) {
        printf("FAIL %s: got %d want %d\n", what, (int)got, (int)want);
        ++failures;
    }
}

int main(void) {
    void* P = (void*)(uintptr_t)(1u << 20); /* 256-byte aligned fake address */
    void* Pm = (void*)((uintptr_t)P + 4);
    const size_t big = (size_t)1 << 30;
    expect("fused null x",
           masq_linear_fused(NULL, MASQ_BF16, P, P, P, P, P, P, MASQ_BF16, 16, 64, 64, 16, 2, P,
                             MASQ_BF16, P, big, NULL), MASQ_ERR_NULL);
    expect("fused bad K",
           masq_linear_fused(P, MASQ_BF16, P, P, P, P, P, P, MASQ_BF16, 16, 40, 64, 16, 2, P,
                             MASQ_BF16, P, big, NULL), MASQ_ERR_SHAPE);
    expect("fused K past exact int32",
           masq_linear_fused(P, MASQ_BF16, P, P, P, P, P, P, MASQ_BF16, 16, 133136 + 16, 64, 16,
                             2, P, MASQ_BF16, P, big, NULL), MASQ_ERR_SHAPE);
    expect("fused huge T",
           masq_linear_fused(P, MASQ_BF16, P, P, P, P, P, P, MASQ_BF16, (int64_t)1 << 40, 64, 64,
                             16, 2, P, MASQ_BF16, P, big, NULL), MASQ_ERR_SHAPE);
    expect("fused misaligned",
           masq_linear_fused(Pm, MASQ_BF16, P, P, P, P, P, P, MASQ_BF16, 16, 64, 64, 16, 2, P,
                             MASQ_BF16, P, big, NULL), MASQ_ERR_ALIGN);
    expect("fused small workspace",
           masq_linear_fused(P, MASQ_BF16, P, P, P, P, P, P, MASQ_BF16, 4096, 3584, 18944, 64, 2,
                             P, MASQ_BF16, P, 1024, NULL), MASQ_ERR_WORKSPACE);
    expect("fused empty",
           masq_linear_fused(NULL, MASQ_BF16, NULL, NULL, NULL, NULL, NULL, NULL, MASQ_BF16, 0,
                             64, 64, 16, 2, NULL, MASQ_BF16, NULL, 0, NULL), MASQ_OK);
    expect("noalloc past scratch",
           masq_linear_fused_noalloc(P, MASQ_BF16, P, P, P, P, P, P, MASQ_BF16, 20000, 3584, 512,
                                     64, 3, P, MASQ_BF16, NULL), MASQ_ERR_SCRATCH);
    expect("noalloc bad dtype",
           masq_linear_fused_noalloc(P, (masq_dtype)9, P, P, P, P, P, P, MASQ_BF16, 16, 64, 64,
                                     16, 2, P, MASQ_BF16, NULL), MASQ_ERR_DTYPE);
    expect("smooth_quant bad n_mod",
           masq_smooth_quant(P, MASQ_BF16, P, P, 16, 64, 5, P, P, NULL), MASQ_ERR_SHAPE);
    expect("gemm no output",
           masq_w8a8_gemm(P, P, P, P, 16, 64, 64, NULL, NULL, MASQ_F32, NULL), MASQ_ERR_NULL);
    expect("w4 gemm ragged",
           masq_w4a8_gemm(P, P, P, P, 16, 96, 64, P, NULL, MASQ_F32, NULL), MASQ_ERR_SHAPE);
    expect("lowrank bad rank",
           masq_lowrank_comp(P, MASQ_BF16, P, P, P, P, MASQ_BF16, 16, 64, 64, 24, 2, P, MASQ_BF16,
                             NULL), MASQ_ERR_SHAPE);
    expect("mas-only ragged K",
           masq_mas_only_linear(P, MASQ_BF16, P, P, P, P, 16, 96, 64, 3, P, MASQ_BF16, P, big,
                                NULL), MASQ_ERR_UNSUPPORTED);
    expect("mas-only small workspace",
           masq_mas_only_linear(P, MASQ_BF16, P, P, P, P, 4096, 3584, 3584, 3, P, MASQ_BF16, P, 64,
                                NULL), MASQ_ERR_WORKSPACE);
    expect("dgemm negative m",
           masq_dgemm(-1, 4, 4, P, 4, 1, P, 4, 1, 0.0, P, 4, NULL), MASQ_ERR_SHAPE);
    expect("cholesky lda < n", masq_cholesky(8, (double*)P, 4, 0.0, (int32_t*)P, NULL, NULL),
           MASQ_ERR_SHAPE);
    expect("cholesky empty", masq_cholesky(0, NULL, 0, 0.0, (int32_t*)P, NULL, NULL), MASQ_OK);
    expect("trsm bad trans",
           masq_trsm_right(4, 8, (const double*)P, 8, 2, (double*)P, 8, NULL), MASQ_ERR_SHAPE);
    expect("jacobi too wide",
           masq_jacobi_svd(4, 1025, (double*)P, (double*)P, (double*)P, (double*)P, (double*)P, 0,
                           10, NULL, NULL), MASQ_ERR_SHAPE);
    expect("mae loss negative count", masq_mae_loss((const double*)P, -1, (double*)P, NULL),
           MASQ_ERR_SHAPE);
    expect("adam bad beta",
           masq_adam_log_step((double*)P, (double*)P, (double*)P, (const double*)P, (float*)P,
                              (float*)P, 8, 1.0, 1e-2, 1.0, 0.999, 1e-8, 1, NULL),
           MASQ_ERR_SHAPE);
    expect("channel range bad dtype",
           masq_channel_range(P, (masq_dtype)7, P, 8, 64, 2, P, NULL), MASQ_ERR_DTYPE);
    if (masq_linear_fused_workspace_bytes(-1, 64, 64, 16, 2) != 0) {
        printf("FAIL workspace query of a negative batch\n");
        ++failures;
    }
    if (masq_mas_only_workspace_bytes(16, 128, 64, 9) != 0) {
        printf("FAIL mas-only workspace query of 9 modalities\n");
        ++failures;
    }
    for (int c = -1; c < 10; ++c)
        if (masq_status_str((masq_status)c) == NULL) {
            printf("FAIL status string %d\n", c);
            ++failures;
        }
    if (failures == 0) printf("ok\n");
    return failures == 0 ? 0 : 1;
}
