/*
 * fp64 CPU oracle for Fibonacci-offset sparse attention.
 *
 * TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's
 * CPU-baseline leg load this library.  It shares no code, header or table with the
 * HIP library; both read the same seeded inputs and nothing else.
 *
 * What it computes is the plain definition of the paper's attended set
 * (Section 2, "Attended set"), written out one query at a time:
 *
 *   - query i attends to window distances delta = 0..W, truncated at position 0;
 *   - and to rung distances d_k = alpha * f_k for the base f (Fibonacci or
 *     power-of-2, Section 2 "Control base");
 *   - a rung is read at the continuous row i - d_k, i.e. as the linear blend of
 *     rows i - floor(d_k) (weight 1 - w) and i - floor(d_k) - 1 (weight w), where
 *     w = d_k - floor(d_k); keys and values are blended with the same weights;
 *   - logits tau * <q_i, key>, tau = 1/sqrt(D); softmax over the entries; the
 *     output is the weighted sum of the (blended) values; lse is saved.
 *
 * Readings of points the paper leaves open (each is listed in the design notes):
 *   - d_k is one IEEE float32 product fl32(alpha * f_k) (round to nearest even);
 *   - a rung with d_k <= W lies inside the window: the attended set is a union,
 *     so it is dropped rather than counted twice;
 *   - a rung with d_k > i reaches before position 0 and is masked; d_k == i is
 *     kept (weight on row 0);
 *   - "floor" is taken on the distance, so the two rows are i - floor(d) and
 *     i - floor(d) - 1; the row -1 (only reached when w == 0) is a zero vector;
 *   - equal rung distances are kept once.
 *
 * Backward: the exact gradient of that forward, with the inclusion masks held
 * constant (a hard mask carries no gradient to alpha, Section 2 "Implementation
 * note"): dw_k/dalpha = f_k and d floor(d_k)/dalpha = 0.
 *
 * RoPE (Section 3 "Model and training": theta_rope = 1e4; Section 2: applied at the
 * true positions before gathering): rotate-half pairing (j, j + D/2) with inverse
 * frequency base^(-2j/D); angles in float64.
 *
 * Grouped key/value heads (Section 3 "Model and training": 8 query heads share 2
 * key/value heads): q, o, dO, dq are [B, H, T, D], k, v, dk, dv are [B, Hkv, T, D]
 * with H a multiple of Hkv; query head h reads key/value head h / (H / Hkv), and
 * dk, dv sum the contributions of the H / Hkv query heads of the group.
 *
 * Tensors are float64, C-contiguous.  Work is split with OpenMP over (b, h) in the
 * forward and over (b, key/value head) in the backward, each unit written by one
 * thread in a fixed order, so results do not depend on the thread count.
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_MAX_RUNGS 64

/* ------------------------------------------------------------------------- */
/* Rung table: offsets shared by every query (Section 2).                    */
/* ------------------------------------------------------------------------- */

/* Returns the number of rungs kept; writes floor(d), w = d - floor(d) (exact in
 * float32), f and d itself, in increasing d.  base must be strictly increasing and
 * alpha > 0, so d is non-decreasing in k. Returns -1 on bad input. */
int oracle_rungs(float alpha, const int *base, int K, int W,
                 int *d0_out, float *w_out, int *f_out, float *d_out)
{
    int n = 0;
    if (K < 0 || K > ORACLE_MAX_RUNGS || !(alpha > 0.0f)) return -1;
    for (int k = 0; k < K; ++k) {
        if (base[k] < 1) return -1;
        if (k > 0 && base[k] <= base[k - 1]) return -1;
        volatile float fk = (float)base[k];
        volatile float d = alpha * fk;          /* one float32 multiply */
        if (!(d > (float)W)) continue;          /* inside the window: already attended */
        if (n > 0 && d == d_out[n - 1]) continue; /* equal distance: keep once */
        float fl = floorf(d);
        d0_out[n] = (int)fl;
        w_out[n] = d - fl;
        f_out[n] = base[k];
        d_out[n] = d;
        ++n;
    }
    return n;
}

/* ------------------------------------------------------------------------- */
/* Per-query entry list.                                                      */
/* ------------------------------------------------------------------------- */

typedef struct {
    int r0, r1;      /* rows; r1 may be -1 (zero row) or unused (w1 == 0, window) */
    double w0, w1;   /* blend weights */
    int f;           /* base value for rung entries, 0 for window entries */
} entry_t;

/* Entries of query i.  Rung k is included when d_k <= i, i.e. floor(d_k) < i, or
 * floor(d_k) == i with w_k == 0. */
static int query_entries(int i, int W, int n, const int *d0, const double *w, const int *f,
                         entry_t *e)
{
    int m = 0;
    for (int delta = 0; delta <= W && delta <= i; ++delta) {
        e[m].r0 = i - delta; e[m].r1 = -1; e[m].w0 = 1.0; e[m].w1 = 0.0; e[m].f = 0;
        ++m;
    }
    for (int k = 0; k < n; ++k) {
        int incl = (d0[k] < i) || (d0[k] == i && w[k] == 0.0);
        if (!incl) continue;
        e[m].r0 = i - d0[k];
        e[m].r1 = i - d0[k] - 1;
        e[m].w0 = 1.0 - w[k];
        e[m].w1 = w[k];
        e[m].f = f[k];
        ++m;
    }
    return m;
}

static double dot(const double *a, const double *b, int D)
{
    double s = 0.0;
    for (int c = 0; c < D; ++c) s += a[c] * b[c];
    return s;
}

/* <x, row r> with row -1 the zero vector */
static double dot_row(const double *x, const double *M, int r, int D)
{
    return r < 0 ? 0.0 : dot(x, M + (size_t)r * D, D);
}

/* ------------------------------------------------------------------------- */
/* Forward on an explicit rung table (w in float64).                          */
/* ------------------------------------------------------------------------- */

void oracle_forward_table(int B, int H, int Hkv, int T, int D, int W,
                          int n, const int *d0, const double *w, const int *f,
                          const double *q, const double *k, const double *v,
                          double *o, double *lse)
{
    const double tau = 1.0 / sqrt((double)D);
    const int BH = B * H;
    const int G = H / Hkv;  /* query heads per key/value head */
#pragma omp parallel
    {
        entry_t *e = (entry_t *)malloc(sizeof(entry_t) * (size_t)(W + 1 + n));
        double *s = (double *)malloc(sizeof(double) * (size_t)(W + 1 + n));
#pragma omp for schedule(dynamic, 1)
        for (int bh = 0; bh < BH; ++bh) {
            const size_t off = (size_t)bh * T * D;
            const size_t kvoff = (size_t)((bh / H) * Hkv + (bh % H) / G) * T * D;
            const double *Q = q + off, *Kx = k + kvoff, *V = v + kvoff;
            for (int i = 0; i < T; ++i) {
                const double *qi = Q + (size_t)i * D;
                int m = query_entries(i, W, n, d0, w, f, e);
                double mx = -INFINITY;
                for (int a = 0; a < m; ++a) {
                    s[a] = tau * (e[a].w0 * dot_row(qi, Kx, e[a].r0, D) +
                                  e[a].w1 * dot_row(qi, Kx, e[a].r1, D));
                    if (s[a] > mx) mx = s[a];
                }
                double z = 0.0;
                for (int a = 0; a < m; ++a) z += exp(s[a] - mx);
                double L = mx + log(z);
                lse[(size_t)bh * T + i] = L;
                double *oi = o + off + (size_t)i * D;
                for (int c = 0; c < D; ++c) oi[c] = 0.0;
                for (int a = 0; a < m; ++a) {
                    double p = exp(s[a] - L);
                    for (int c = 0; c < D; ++c) {
                        double vh = e[a].w0 * V[(size_t)e[a].r0 * D + c];
                        if (e[a].r1 >= 0) vh += e[a].w1 * V[(size_t)e[a].r1 * D + c];
                        oi[c] += p * vh;
                    }
                }
            }
        }
        free(e);
        free(s);
    }
}

/* ------------------------------------------------------------------------- */
/* Backward on an explicit rung table.                                        */
/* dq, dk, dv are overwritten.  dalpha = sum over b,h,i and rung entries of    */
/* f_k * dL/dw; l1 = sum of |f_k * dL/dw| (the magnitude of the terms).        */
/* ------------------------------------------------------------------------- */

void oracle_backward_table(int B, int H, int Hkv, int T, int D, int W,
                           int n, const int *d0, const double *w, const int *f,
                           const double *q, const double *k, const double *v,
                           const double *dO,
                           double *dq, double *dk, double *dv,
                           double *dalpha, double *l1)
{
    const double tau = 1.0 / sqrt((double)D);
    const int BHkv = B * Hkv;
    const int G = H / Hkv;  /* query heads sharing one key/value head */
    double *part = (double *)calloc((size_t)BHkv * 2, sizeof(double));
    memset(dk, 0, sizeof(double) * (size_t)BHkv * T * D);
    memset(dv, 0, sizeof(double) * (size_t)BHkv * T * D);
#pragma omp parallel
    {
        const int cap = W + 1 + n;
        entry_t *e = (entry_t *)malloc(sizeof(entry_t) * (size_t)cap);
        double *s = (double *)malloc(sizeof(double) * (size_t)cap);
        double *p = (double *)malloc(sizeof(double) * (size_t)cap);
        double *dP = (double *)malloc(sizeof(double) * (size_t)cap);
        double *oi = (double *)malloc(sizeof(double) * (size_t)D);
        /* one key/value head at a time: its G query heads scatter into the same dk, dv */
#pragma omp for schedule(dynamic, 1)
        for (int bk = 0; bk < BHkv; ++bk) {
          const size_t kvoff = (size_t)bk * T * D;
          const double *Kx = k + kvoff, *V = v + kvoff;
          double *DK = dk + kvoff, *DV = dv + kvoff;
          double acc = 0.0, acc1 = 0.0;
          for (int hg = 0; hg < G; ++hg) {
            const int bh = (bk / Hkv) * H + (bk % Hkv) * G + hg;
            const size_t off = (size_t)bh * T * D;
            const double *Q = q + off, *Gd = dO + off;
            double *DQ = dq + off;
            for (int i = 0; i < T; ++i) {
                const double *qi = Q + (size_t)i * D;
                const double *gi = Gd + (size_t)i * D;
                int m = query_entries(i, W, n, d0, w, f, e);
                /* forward recomputed exactly */
                double mx = -INFINITY;
                for (int a = 0; a < m; ++a) {
                    s[a] = tau * (e[a].w0 * dot_row(qi, Kx, e[a].r0, D) +
                                  e[a].w1 * dot_row(qi, Kx, e[a].r1, D));
                    if (s[a] > mx) mx = s[a];
                }
                double z = 0.0;
                for (int a = 0; a < m; ++a) z += exp(s[a] - mx);
                double L = mx + log(z);
                for (int c = 0; c < D; ++c) oi[c] = 0.0;
                for (int a = 0; a < m; ++a) {
                    p[a] = exp(s[a] - L);
                    for (int c = 0; c < D; ++c) {
                        double vh = e[a].w0 * V[(size_t)e[a].r0 * D + c];
                        if (e[a].r1 >= 0) vh += e[a].w1 * V[(size_t)e[a].r1 * D + c];
                        oi[c] += p[a] * vh;
                    }
                }
                /* Delta_i = <dO_i, o_i>; dP_e = <dO_i, vhat_e>; dS_e = p_e (dP_e - Delta_i) */
                double delta = dot(gi, oi, D);
                for (int a = 0; a < m; ++a)
                    dP[a] = e[a].w0 * dot_row(gi, V, e[a].r0, D) + e[a].w1 * dot_row(gi, V, e[a].r1, D);
                double *dqi = DQ + (size_t)i * D;
                for (int c = 0; c < D; ++c) dqi[c] = 0.0;
                for (int a = 0; a < m; ++a) {
                    double dS = p[a] * (dP[a] - delta);
                    for (int c = 0; c < D; ++c) {
                        double kh = e[a].w0 * Kx[(size_t)e[a].r0 * D + c];
                        if (e[a].r1 >= 0) kh += e[a].w1 * Kx[(size_t)e[a].r1 * D + c];
                        dqi[c] += tau * dS * kh;
                    }
                    /* scatter through the blend weights */
                    for (int c = 0; c < D; ++c) {
                        DK[(size_t)e[a].r0 * D + c] += e[a].w0 * tau * dS * qi[c];
                        DV[(size_t)e[a].r0 * D + c] += e[a].w0 * p[a] * gi[c];
                    }
                    if (e[a].r1 >= 0 && e[a].w1 != 0.0) {
                        for (int c = 0; c < D; ++c) {
                            DK[(size_t)e[a].r1 * D + c] += e[a].w1 * tau * dS * qi[c];
                            DV[(size_t)e[a].r1 * D + c] += e[a].w1 * p[a] * gi[c];
                        }
                    }
                    if (e[a].f != 0) {
                        /* dL/dw: the logit moves by tau<q, k[r1]-k[r0]>, the value by v[r1]-v[r0] */
                        double ds_dw = tau * (dot_row(qi, Kx, e[a].r1, D) - dot_row(qi, Kx, e[a].r0, D));
                        double dv_dw = dot_row(gi, V, e[a].r1, D) - dot_row(gi, V, e[a].r0, D);
                        double g = dS * ds_dw + p[a] * dv_dw;
                        acc += (double)e[a].f * g;
                        acc1 += fabs((double)e[a].f * g);
                    }
                }
            }
          }
          part[2 * bk] = acc;
          part[2 * bk + 1] = acc1;
        }
        free(e); free(s); free(p); free(dP); free(oi);
    }
    double sa = 0.0, s1 = 0.0;
    for (int bk = 0; bk < BHkv; ++bk) { sa += part[2 * bk]; s1 += part[2 * bk + 1]; }
    free(part);
    *dalpha = sa;
    *l1 = s1;
}

/* ------------------------------------------------------------------------- */
/* Entry points taking alpha: build the float32 rung table, then run.         */
/* ------------------------------------------------------------------------- */

static int table_from_alpha(float alpha, const int *base, int K, int W,
                            int *d0, double *w, int *f)
{
    float wf[ORACLE_MAX_RUNGS], df[ORACLE_MAX_RUNGS];
    int n = oracle_rungs(alpha, base, K, W, d0, wf, f, df);
    for (int a = 0; a < n; ++a) w[a] = (double)wf[a];
    return n;
}

int oracle_forward(int B, int H, int Hkv, int T, int D, int W, const int *base, int K, float alpha,
                   const double *q, const double *k, const double *v, double *o, double *lse)
{
    int d0[ORACLE_MAX_RUNGS], f[ORACLE_MAX_RUNGS];
    double w[ORACLE_MAX_RUNGS];
    int n = table_from_alpha(alpha, base, K, W, d0, w, f);
    if (n < 0) return -1;
    if (Hkv < 1 || H % Hkv != 0) return -1;
    oracle_forward_table(B, H, Hkv, T, D, W, n, d0, w, f, q, k, v, o, lse);
    return 0;
}

int oracle_backward(int B, int H, int Hkv, int T, int D, int W, const int *base, int K, float alpha,
                    const double *q, const double *k, const double *v, const double *dO,
                    double *dq, double *dk, double *dv, double *dalpha, double *l1)
{
    int d0[ORACLE_MAX_RUNGS], f[ORACLE_MAX_RUNGS];
    double w[ORACLE_MAX_RUNGS];
    int n = table_from_alpha(alpha, base, K, W, d0, w, f);
    if (n < 0) return -1;
    if (Hkv < 1 || H % Hkv != 0) return -1;
    oracle_backward_table(B, H, Hkv, T, D, W, n, d0, w, f, q, k, v, dO, dq, dk, dv, dalpha, l1);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* RoPE at true positions 0..T-1 (rotate-half).  transpose != 0 applies R^T,  */
/* the map the backward uses to carry gradients back to the unrotated input. */
/* ------------------------------------------------------------------------- */

void oracle_rope(int B, int H, int T, int D, double rope_base, int transpose,
                 const double *x, double *y)
{
    const int half = D / 2;
    const int BH = B * H;
#pragma omp parallel for schedule(static)
    for (int bh = 0; bh < BH; ++bh) {
        for (int t = 0; t < T; ++t) {
            const double *xr = x + ((size_t)bh * T + t) * D;
            double *yr = y + ((size_t)bh * T + t) * D;
            for (int j = 0; j < half; ++j) {
                double inv_freq = pow(rope_base, -2.0 * (double)j / (double)D);
                double ang = (double)t * inv_freq;
                double c = cos(ang), s = sin(ang);
                double a = xr[j], b = xr[j + half];
                if (!transpose) {
                    yr[j] = a * c - b * s;
                    yr[j + half] = b * c + a * s;
                } else {
                    yr[j] = a * c + b * s;
                    yr[j + half] = b * c - a * s;
                }
            }
        }
    }
}

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
