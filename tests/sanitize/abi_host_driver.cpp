// Drives the host side of libmpgemm (argument checks, kernel selection,
// split and workspace planning, the host view of the INT4 encodings) under
// AddressSanitizer + UndefinedBehaviorSanitizer, without a GPU: every call
// here returns before touching a device (invalid arguments are refused on the
// host; the query functions never launch anything). Any sanitizer report, or
// a documented result that does not hold, makes the process fail.
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "mpgemm.h"

static int bad = 0;
#define CHECK(c)                                                                    \
    do {                                                                            \
        if (!(c)) {                                                                 \
            fprintf(stderr, "FAIL line %d: %s\n", __LINE__, #c);                    \
            bad = 1;                                                                \
        }                                                                           \
    } while (0)

int main() {
    const void *A = (const void *)(uintptr_t(1) << 20), *B = (const void *)(uintptr_t(1) << 40);
    void *C = (void *)(uintptr_t(1) << 44);
    const int sizes[] = {0, 1, 2, 3, 16, 31, 33, 100, 128, 255, 256, 257, 512, 1000, 1024, 4096, 8192, 65536};
    long checked = 0;
    for (int dt = 0; dt < 3; ++dt) {
        const int nv = mpgemm_num_variants(dt);
        CHECK(nv > 1);
        for (int M : sizes)
            for (int N : sizes)
                for (int K : {0, 2, 64, 256, 1000, 4096, 8192, 70000}) {
                    const int v = mpgemm_select_variant(dt, M, N, K, A, B, C);
                    const int vw = mpgemm_select_variant_ws(dt, M, N, K, A, B, C);
                    CHECK(v >= 0 && v < nv && vw >= 0 && vw < nv);
                    CHECK(mpgemm_variant_supports(dt, v, M, N, K, A, B, C) == 1);
                    size_t bytes = 1;
                    CHECK(mpgemm_workspace_size(dt, -1, 0, M, N, K, nullptr, &bytes) == hipSuccess);
                    CHECK(mpgemm_workspace_size(dt, v, 1, M, N, K, nullptr, &bytes) == hipSuccess);
                    CHECK(mpgemm_select_splits(dt, v, M, N, K) >= 1);
                    ++checked;
                }
        for (int v = -1; v <= nv; ++v) {
            const char *name = mpgemm_variant_name(dt, v);
            CHECK(name != nullptr);
            size_t bytes = 0;
            (void)mpgemm_workspace_size(dt, v, 2, 512, 640, 2048, nullptr, &bytes);
        }
    }
    // argument errors: refused on the host, nothing enqueued
    const hipError_t inv = hipErrorInvalidValue;
    CHECK(gemm_s8_s32(-1, 8, 8, (const int8_t *)A, (const int8_t *)B, (int32_t *)C, nullptr) == inv);
    CHECK(gemm_s4_s32(8, 8, 7, (const uint8_t *)A, (const uint8_t *)B, (int32_t *)C, nullptr) == inv);
    CHECK(gemm_f16_f32(8, 8, 8, (const char *)A + 1, B, (float *)C, nullptr) == inv);
    CHECK(gemm_s8_s32(8, 8, 8, (const int8_t *)A, (const int8_t *)B, (int32_t *)A, nullptr) == inv);
    CHECK(gemm_scaled(1, 8, 8, 8, A, B, C, nullptr, nullptr) == inv);
    mpgemm_epilogue zp = {nullptr, nullptr, (const int32_t *)(uintptr_t(1) << 30), nullptr, MPGEMM_OUT_F16};
    CHECK(gemm_scaled(1, 64, 64, 64, A, B, C, &zp, nullptr) == inv);
    CHECK(mpgemm_gemm_ws(1, 64, 64, 64, A, B, C, nullptr, (void *)((uintptr_t(1) << 46) + 16), 1 << 20, nullptr) == inv);
    CHECK(mpgemm_gemm_ws(1, 64, 64, 64, A, B, C, &zp, (void *)(uintptr_t(1) << 46), 256, nullptr) == inv);
    CHECK(mpgemm_run_variant_ws(1, 0, 2, 64, 64, 64, A, B, C, nullptr, nullptr, 0, nullptr) == inv);
    CHECK(mpgemm_run_variant(7, 1, 8, 8, 8, A, B, C, nullptr) == inv);
    CHECK(mpgemm_gemm_noalloc(1, -1, 8, 8, A, B, C, nullptr, nullptr) == inv);
    CHECK(mpgemm_gemm_bt(2, 256, 256, 64, A, B, C, nullptr) == inv);
    size_t bytes = 0;
    CHECK(mpgemm_workspace_size(1, -1, 0, -1, 8, 8, nullptr, &bytes) == inv);
    CHECK(mpgemm_workspace_size(1, -1, 0, 8, 8, 8, nullptr, nullptr) == inv);
    CHECK(mpgemm_select_variant(9, 8, 8, 8, A, B, C) == -1);
    // host views of the INT4 encodings
    uint8_t run[16];
    uint32_t out[6];
    for (int t = 0; t < 1000; ++t) {
        for (int i = 0; i < 16; ++i) run[i] = (uint8_t)(rand() & 0xFF);
        mpgemm_s4_run_to_fp6(run, out);
        mpgemm_s4_run_to_e2m3(run, out);
    }
    printf("abi host driver: %ld shape checks, %s\n", checked, bad ? "FAILED" : "ok");
    return bad;
}
