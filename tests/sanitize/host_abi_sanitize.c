/*
 * The host-side code of libf3s.so under AddressSanitizer and
 * UndefinedBehaviorSanitizer, on a machine without a GPU (built and run by
 * tests/test_sanitize_host.py): every entry point's argument checks, the
 * scratch sizing of plan builds over the whole int32 range of N and of the
 * CSR length, status strings, and the failure paths of plan builds when the
 * HIP runtime finds no device (the plan object is created and released on
 * the way).  Any out-of-bounds access, leak in the library, integer overflow
 * or other undefined behaviour aborts the run.  Prints "ok" on success.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "f3s.h"
#include "f3s_probe.h"

#define CHECK(c)                                                           \
    do {                                                                   \
        if (!(c)) {                                                        \
            fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
            return 1;                                                      \
        }                                                                  \
    } while (0)

int main(void)
{
    for (int s = -1; s <= 7; ++s) CHECK(f3s_status_string((f3s_status_t)s) != NULL);
    CHECK(strcmp(f3s_status_string(F3S_ERR_TOO_LARGE), "F3S_ERR_TOO_LARGE") == 0);
    CHECK(f3s_last_error() == F3S_OK);

    /* scratch sizing: non-decreasing in nnz and N, at least 6 bytes per entry,
       no overflow up to the int32 limits */
    const int32_t Ns[] = {0, 1, 15, 16, 17, 1000, 1 << 20, 1 << 30, 2147483632, 2147483647};
    const int64_t nnzs[] = {0, 1, 17, 1 << 20, 1ll << 30, 2147483647ll};
    for (size_t a = 0; a < sizeof Ns / sizeof Ns[0]; ++a) {
        size_t prev = 0;
        for (size_t b = 0; b < sizeof nnzs / sizeof nnzs[0]; ++b) {
            const size_t w = f3s_plan_workspace_bytes(Ns[a], nnzs[b]);
            CHECK(w >= (size_t)(6 * nnzs[b]));
            CHECK(w >= prev);
            prev = w;
        }
    }
    CHECK(f3s_plan_workspace_bytes(-1, 5) == 0 && f3s_plan_workspace_bytes(5, -1) == 0);

    /* argument errors, no device needed */
    CHECK(f3s_plan(NULL, NULL, -1) == NULL && f3s_last_error() == F3S_ERR_INVALID_VALUE);
    CHECK(f3s_plan(NULL, NULL, 5) == NULL && f3s_last_error() == F3S_ERR_INVALID_VALUE);
    int32_t rp[3] = {0, 1, 2}, ci[2] = {0, 1};
    CHECK(f3s_plan_ws(rp, ci, 2, NULL, 0) == NULL && f3s_last_error() == F3S_ERR_INVALID_VALUE);
    f3s_plan_info_t info;
    CHECK(f3s_plan_info(NULL, &info) == F3S_ERR_INVALID_VALUE);
    CHECK(f3s_plan_info(NULL, NULL) == F3S_ERR_INVALID_VALUE);
    f3s_destroy(NULL);
    CHECK(f3s_plan_export(NULL, NULL, NULL, NULL, NULL, NULL) == F3S_ERR_INVALID_VALUE);
    CHECK(f3s_run(NULL, NULL, NULL, NULL, NULL, 64, 1.0f, NULL) == F3S_ERR_INVALID_VALUE);
    CHECK(f3s_run_mh(NULL, NULL, NULL, NULL, NULL, 2, 64, 1.0f, NULL) == F3S_ERR_INVALID_VALUE);
    CHECK(f3s_forward(NULL, NULL, NULL, NULL, NULL, NULL, 1, 64, 1.0f, NULL) ==
          F3S_ERR_INVALID_VALUE);
    CHECK(f3s_forward_typed(NULL, NULL, NULL, NULL, F3S_DTYPE_F16, NULL, F3S_DTYPE_F32, NULL, 1,
                            64, 1.0f, NULL) == F3S_ERR_INVALID_VALUE);
    CHECK(f3s_backward(NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL,
                       1, 64, 1.0f, NULL) == F3S_ERR_INVALID_VALUE);
    CHECK(f3s_backward_typed(NULL, NULL, NULL, NULL, NULL, F3S_DTYPE_FP8_E4M3, NULL, NULL,
                             NULL, NULL, NULL, NULL, NULL, 1, 64, 1.0f, NULL) ==
          F3S_ERR_UNSUPPORTED);
    CHECK(f3s_backward_noalloc(NULL, NULL, NULL, NULL, NULL, F3S_DTYPE_F16, NULL, NULL, NULL,
                               NULL, NULL, NULL, 1, 64, 1.0f, NULL) == F3S_ERR_INVALID_VALUE);
    CHECK(f3s_backward_noalloc_max_records() == (int64_t)1 << 21);
    CHECK(f3s_plan_transpose(NULL) == NULL && f3s_last_error() == F3S_ERR_INVALID_VALUE);
    CHECK(f3s_plan_window_rows(NULL, NULL) == F3S_ERR_INVALID_VALUE);
    /* batch segmentations: malformed ones are rejected; the windows of valid
       ones are computed (on the host) before the null CSR is rejected */
    {
        const int32_t bad[][4] = {{1, 2, 3, 4}, {0, 3, 2, 4}, {0, 1, 2, 3}};
        for (int k = 0; k < 3; ++k)
            CHECK(f3s_plan_segments(NULL, NULL, 4, bad[k], 3) == NULL &&
                  f3s_last_error() == F3S_ERR_INVALID_VALUE);
        CHECK(f3s_plan_segments(NULL, NULL, 4, NULL, 3) == NULL &&
              f3s_last_error() == F3S_ERR_INVALID_VALUE);
        CHECK(f3s_plan_segments(NULL, NULL, 4, bad[0], -1) == NULL &&
              f3s_last_error() == F3S_ERR_INVALID_VALUE);
        int32_t seg[40];
        seg[0] = 0;
        for (int g = 0; g < 39; ++g) seg[g + 1] = seg[g] + (g * 7) % 41;  /* 0 .. 40 rows */
        const int32_t n = seg[39];
        CHECK(f3s_plan_segments(NULL, NULL, n, seg, 39) == NULL &&
              f3s_last_error() == F3S_ERR_INVALID_VALUE);
        const int32_t one[2] = {0, 1 << 24};
        CHECK(f3s_plan_segments(NULL, NULL, 1 << 24, one, 1) == NULL &&
              f3s_last_error() == F3S_ERR_INVALID_VALUE);
    }
    CHECK(f3s_plan_transpose_workspace_bytes(NULL) == 0);
    CHECK(f3s_plan_transpose_ws(NULL, NULL, 0) == NULL);
    CHECK(f3s_probe_read(NULL, 16, NULL, NULL) == F3S_ERR_INVALID_VALUE);
    CHECK(f3s_probe_copy(NULL, NULL, 16, NULL) == F3S_ERR_INVALID_VALUE);
    CHECK(f3s_probe_write(NULL, 16, 0u, NULL) == F3S_ERR_INVALID_VALUE);
    CHECK(f3s_probe_gather(NULL, NULL, NULL, NULL, NULL, 64, NULL) == F3S_ERR_INVALID_VALUE);
    CHECK(f3s_probe_gather_lds(NULL, NULL, NULL, NULL, NULL, 64, NULL) ==
          F3S_ERR_INVALID_VALUE);
    CHECK(f3s_probe_rows(NULL, 16, 128, 8, 1, 1, NULL, NULL) == F3S_ERR_INVALID_VALUE);
    CHECK(f3s_run_trace(NULL, NULL, NULL, NULL, NULL, 64, 1.0f, NULL, 0, NULL) ==
          F3S_ERR_INVALID_VALUE);

    /* without a device every build fails, releasing the plan object it made */
    for (int k = 0; k < 3; ++k) {
        CHECK(f3s_plan(rp, ci, 2) == NULL);
        CHECK(f3s_last_error() != F3S_OK);
        CHECK(f3s_plan(rp, ci, 0) == NULL);
    }
    (void)f3s_wall_clock_khz(-1);
    printf("ok\n");
    return 0;
}
