/*
 * Sanitizer driver for the C ABI's host code (CPU only, no GPU needed): linked with
 * an AddressSanitizer / UndefinedBehaviorSanitizer build of api.hip, it calls every
 * entry point on paths that return before any HIP call: the host rung table over the
 * workload alphas and bad bases, the workspace sizes, and the refusals of invalid
 * arguments (null or misaligned pointers, bad sizes, layouts, alpha, rope base, W, K,
 * grouped-head counts, a too-small workspace, a problem beyond the static scratch).
 * Any out-of-bounds access or undefined operation aborts the run.
 */
#include <math.h>
#include <stdio.h>
#include <string.h>

#include "fibattn.h"

static int bad = 0;
static const int32_t *unsorted_base() {
    static const int32_t b[3] = {5, 3, 8};
    return b;
}
#define EXPECT(cond)                                                   \
    do {                                                               \
        if (!(cond)) { fprintf(stderr, "line %d: %s\n", __LINE__, #cond); bad = 1; } \
    } while (0)

int main() {
    const int32_t fib[15] = {1, 2, 3, 5, 8, 13, 21, 34, 55, 89, 144, 233, 377, 610, 987};
    const int32_t pow2[11] = {1, 2, 4, 8, 16, 32, 64, 128, 256, 512, 1024};
    int32_t many[40];
    for (int a = 0; a < 40; ++a) many[a] = 1 + a;
    int32_t d0[FIBATTN_MAX_RUNGS], f[FIBATTN_MAX_RUNGS];
    float w[FIBATTN_MAX_RUNGS];
    int n = -7;

    // host rung table: every kept rung lies beyond the window, in increasing distance
    const float alphas[] = {0.5f, 0.7310586f, 0.9666667f, 1.0f, 1.2333333f, 1.5f, 0.01f, 3.7f, 1e30f};
    for (float a : alphas)
        for (int W = 0; W <= FIBATTN_MAX_WINDOW; W += 4) {
            for (int base = 0; base < 2; ++base) {
                const int32_t *b = base ? pow2 : fib;
                const int K = base ? 11 : 15;
                const fibattn_status_t st = fibattn_rung_table(a, b, K, W, d0, w, f, &n);
                if (a > 1e29f) { EXPECT(st == FIBATTN_ERR_INVALID_ARG); continue; }
                EXPECT(st == FIBATTN_OK && n >= 0 && n <= K);
                for (int r = 0; r < n; ++r) {
                    EXPECT(w[r] >= 0.f && w[r] < 1.f);
                    EXPECT(d0[r] + w[r] > (float)W);
                    if (r) EXPECT(d0[r] + w[r] > d0[r - 1] + w[r - 1]);
                }
            }
        }
    EXPECT(fibattn_rung_table(1.f, many, 32, 0, d0, w, f, &n) == FIBATTN_OK && n == 32);
    EXPECT(fibattn_rung_table(1.f, many, 33, 0, d0, w, f, &n) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_rung_table(NAN, fib, 15, 8, d0, w, f, &n) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_rung_table(1.f, nullptr, 3, 8, d0, w, f, &n) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_rung_table(1.f, fib, 15, 8, nullptr, w, f, &n) == FIBATTN_ERR_INVALID_ARG);

    // workspace sizes
    EXPECT(fibattn_backward_workspace_bytes(8, 8, 1024, 64, 8, 15) > 0);
    EXPECT(fibattn_backward_workspace_bytes(0, 8, 1024, 64, 8, 15) == 0);
    EXPECT(fibattn_backward_workspace_bytes(1, 1, 1 << 24, 64, 8, 15) == 0);
    EXPECT(fibattn_backward_workspace_bytes(1, 1, 100, 96, 8, 15) == 0);

    // refusals before any launch
    void *p = (void *)(uintptr_t)256, *mis = (void *)(uintptr_t)258;
    float *fp = (float *)p;
    const float one = 1.f;
    EXPECT(fibattn_forward(nullptr, p, p, p, fp, 1, 1, 8, 64, 8, fib, 15, one, FIBATTN_BF16, 0) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_forward(mis, p, p, p, fp, 1, 1, 8, 64, 8, fib, 15, one, FIBATTN_BF16, 0) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_forward(p, p, p, p, fp, 1, 1, 8, 96, 8, fib, 15, one, FIBATTN_BF16, 0) == FIBATTN_ERR_UNSUPPORTED);
    EXPECT(fibattn_forward(p, p, p, p, fp, 1, 1, 8, 64, 129, fib, 15, one, FIBATTN_BF16, 0) == FIBATTN_ERR_UNSUPPORTED);
    EXPECT(fibattn_forward(p, p, p, p, fp, 1, 1, 8, 64, 8, fib, 15, -one, FIBATTN_BF16, 0) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_forward(p, p, p, p, fp, 1, 1, 8, 64, 8, many, 33, one, FIBATTN_BF16, 0) == FIBATTN_ERR_UNSUPPORTED);
    EXPECT(fibattn_forward(p, p, p, p, fp, 1, 1, 8, 64, 8, fib, 15, one, (fibattn_dtype_t)7, 0) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_forward_gqa(p, p, p, p, fp, 1, 8, 3, 8, 64, 8, fib, 15, one, FIBATTN_BF16, 0) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_backward(p, p, p, p, fp, p, p, p, p, fp, p, 16, 1, 1, 64, 64, 8, fib, 15, one, 0.f,
                            FIBATTN_BF16, 0) == FIBATTN_ERR_WORKSPACE);
    EXPECT(fibattn_backward(p, p, p, p, fp, p, p, p, p, fp, p, 1 << 30, 1, 1, 64, 64, 8, fib, 15, one, 0.5f,
                            FIBATTN_BF16, 0) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_backward_gqa(p, p, p, p, fp, p, p, p, p, nullptr, p, 1 << 30, 1, 4, 2, 64, 64, 8, fib, 15,
                                one, 0.f, FIBATTN_BF16, 0) == FIBATTN_ERR_INVALID_ARG);
    fibattn_layout_t lay[8];
    for (auto &l : lay) l = {64 * 64, 64 * 64, 64};
    lay[2].pos = 60;  // rows no longer 16-byte aligned
    EXPECT(fibattn_forward_strided(p, p, p, p, fp, lay, 1, 1, 1, 64, 64, 8, fib, 15, one, FIBATTN_BF16, 0) ==
           FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_backward_strided(p, p, p, p, fp, p, p, p, p, fp, p, 1 << 30, lay, 1, 1, 1, 64, 64, 8, fib,
                                    15, one, 0.f, FIBATTN_BF16, 0) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_forward_strided(p, p, p, p, fp, nullptr, 1, 1, 1, 64, 64, 8, fib, 15, one, FIBATTN_BF16, 0) ==
           FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_device_table(fp, fib, 15, 8, nullptr, 0) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_device_table(fp, fib, 15, -1, p, 0) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_forward_dt(p, p, p, p, fp, 1, 2, 2, 64, 64, 8, nullptr, FIBATTN_BF16, 0) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_device_table_theta(nullptr, fp, fib, 15, 8, p, 0) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_rope_qk_table(p, p, p, p, 1, 8, 3, 64, 64, 1e4f, nullptr, nullptr, fib, 15, 8, nullptr,
                                 FIBATTN_BF16, 0) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_rope_qk_table(p, p, p, p, 1, 8, 2, 64, 64, 1e4f, fp, nullptr, unsorted_base(), 3, 8, p,
                                 FIBATTN_BF16, 0) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_device_table_theta(fp, nullptr, fib, 15, 8, mis, 0) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_backward_dt(p, p, p, p, fp, p, p, p, p, fp, nullptr, p, 16, 1, 2, 2, 64, 64, 8, p, 0.f, FIBATTN_BF16,
                               0) == FIBATTN_ERR_WORKSPACE);
    EXPECT(fibattn_alpha_from_theta(fp, fp, 0, 0) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_dtheta(fp, nullptr, fp, 4, 0) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_rope(p, p, 1, 1, 64, 64, 0.5f, 0, FIBATTN_BF16, 0) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_rope_qk(p, p, p, mis, 1, 1, 64, 64, 1e4f, FIBATTN_BF16, 0) == FIBATTN_ERR_INVALID_ARG);
    EXPECT(fibattn_backward_noalloc(p, p, p, p, fp, p, p, p, p, fp, 32, 8, 8, 16384, 64, 8, fib, 15, one, 0.f,
                                    FIBATTN_BF16, 0) == FIBATTN_ERR_SCRATCH);
    EXPECT(fibattn_timing_begin(99, 4) == FIBATTN_ERR_INVALID_ARG);
    float ms = -1.f;
    int cnt = -1;
    EXPECT(fibattn_timing_end(&ms, &cnt) == FIBATTN_OK && cnt == 0);
    for (int s = -3; s <= 9; ++s) EXPECT(strlen(fibattn_status_string((fibattn_status_t)s)) > 0);
    EXPECT(fibattn_forward(p, p, p, p, fp, 1, 1, 8, 64, 8, fib, 15, one, (fibattn_dtype_t)-1, 0) ==
           FIBATTN_ERR_INVALID_ARG);
    puts(bad ? "FAIL" : "OK");
    return bad;
}
