/*
 * Sanitizer driver for the oracle (CPU only): built with AddressSanitizer and
 * UndefinedBehaviorSanitizer together with oracle/fibattn_oracle.c, it runs every
 * oracle entry point over small inputs that reach the edge cases of the attended set
 * (T = 1, W = 0, no rungs, rungs inside the window or before position 0, a rung landing
 * on row 0, grouped heads, K = 32) and checks that every output is finite.  Any
 * out-of-bounds access, leak or undefined operation aborts the run.
 */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_rungs(float alpha, const int *base, int K, int W, int *d0, float *w, int *f, float *d);
int oracle_forward(int B, int H, int Hkv, int T, int D, int W, const int *base, int K, float alpha,
                   const double *q, const double *k, const double *v, double *o, double *lse);
int oracle_backward(int B, int H, int Hkv, int T, int D, int W, const int *base, int K, float alpha,
                    const double *q, const double *k, const double *v, const double *dO,
                    double *dq, double *dk, double *dv, double *dalpha, double *l1);
void oracle_rope(int B, int H, int T, int D, double rope_base, int transpose, const double *x, double *y);

static unsigned long long rng = 88172645463325252ull;
static double urand(void) { /* xorshift64, values in [-1, 1) */
    rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17;
    return (double)(rng >> 11) / (double)(1ull << 52) - 1.0;
}

static int all_finite(const double *x, size_t n) {
    for (size_t a = 0; a < n; ++a)
        if (!isfinite(x[a])) return 0;
    return 1;
}

static int run_case(int B, int H, int Hkv, int T, int D, int W, const int *base, int K, float alpha) {
    size_t nq = (size_t)B * H * T * D, nk = (size_t)B * Hkv * T * D;
    double *q = malloc(nq * sizeof(double)), *dO = malloc(nq * sizeof(double));
    double *k = malloc(nk * sizeof(double)), *v = malloc(nk * sizeof(double));
    double *o = malloc(nq * sizeof(double)), *lse = malloc((size_t)B * H * T * sizeof(double));
    double *dq = malloc(nq * sizeof(double)), *dk = malloc(nk * sizeof(double));
    double *dv = malloc(nk * sizeof(double)), *y = malloc(nq * sizeof(double));
    double da = 0.0, l1 = 0.0;
    int ok = 1;
    for (size_t a = 0; a < nq; ++a) { q[a] = urand(); dO[a] = urand(); }
    for (size_t a = 0; a < nk; ++a) { k[a] = urand(); v[a] = urand(); }
    if (oracle_forward(B, H, Hkv, T, D, W, base, K, alpha, q, k, v, o, lse) != 0) ok = 0;
    if (oracle_backward(B, H, Hkv, T, D, W, base, K, alpha, q, k, v, dO, dq, dk, dv, &da, &l1) != 0) ok = 0;
    oracle_rope(B, H, T, D, 10000.0, 0, q, y);
    oracle_rope(B, H, T, D, 10000.0, 1, y, y);
    ok = ok && all_finite(o, nq) && all_finite(lse, (size_t)B * H * T) && all_finite(dq, nq) &&
         all_finite(dk, nk) && all_finite(dv, nk) && isfinite(da) && isfinite(l1) && all_finite(y, nq);
    free(q); free(dO); free(k); free(v); free(o); free(lse); free(dq); free(dk); free(dv); free(y);
    return ok;
}

int main(void) {
    static const int fib[15] = {1, 2, 3, 5, 8, 13, 21, 34, 55, 89, 144, 233, 377, 610, 987};
    static const int pow2[11] = {1, 2, 4, 8, 16, 32, 64, 128, 256, 512, 1024};
    static const int row0[3] = {1, 13, 40};
    int many[32];
    for (int a = 0; a < 32; ++a) many[a] = 3 + 3 * a;
    struct { int B, H, Hkv, T, D, W; const int *base; int K; float alpha; } cases[] = {
        {1, 2, 2, 128, 32, 8, fib, 15, 1.0f},
        {2, 3, 3, 70, 8, 3, fib, 15, 0.7310586f},
        {1, 4, 2, 50, 4, 2, pow2, 11, 1.3f},
        {1, 4, 1, 33, 8, 0, fib, 8, 0.9f},
        {1, 1, 1, 1, 8, 8, fib, 15, 1.0f},
        {1, 2, 2, 5, 4, 8, fib, 15, 1.0f},
        {1, 2, 2, 20, 4, 0, fib, 0, 1.0f},
        {1, 2, 2, 64, 4, 2, row0, 3, 1.0f},
        {1, 1, 1, 120, 4, 0, many, 32, 0.9f},
        {1, 2, 2, 40, 4, 12, fib, 5, 1.0f},
    };
    int bad = 0;
    for (size_t c = 0; c < sizeof cases / sizeof cases[0]; ++c) {
        if (!run_case(cases[c].B, cases[c].H, cases[c].Hkv, cases[c].T, cases[c].D, cases[c].W,
                      cases[c].base, cases[c].K, cases[c].alpha)) {
            fprintf(stderr, "case %zu: non-finite output or refused input\n", c);
            bad = 1;
        }
    }
    /* the rung table refuses bad input without touching the output arrays past K */
    int d0[64], f[64];
    float w[64], d[64];
    static const int unsorted[3] = {3, 2, 5};
    if (oracle_rungs(1.0f, unsorted, 3, 2, d0, w, f, d) != -1) bad = 1;
    if (oracle_rungs(-1.0f, fib, 15, 2, d0, w, f, d) != -1) bad = 1;
    if (oracle_rungs(1.0f, many, 32, 2, d0, w, f, d) != 32) bad = 1;
    puts(bad ? "FAIL" : "OK");
    return bad;
}
