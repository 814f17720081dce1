// Backward kernels: dq + dalpha (query-stationary), dk/dv (key-stationary, no
// atomics), and the fixed-order dalpha reduction.
//
// The gradient is that of the forward in fwd.hip with the inclusion masks held
// constant (Section 2 "Implementation note": a hard mask carries no gradient to
// alpha, so alpha acts only through the blend weights, dw_k/dalpha = f_k).
// With p_e = exp(s_e - lse_i), Delta_i = <dO_i, o_i>, dP_e = <dO_i, vhat_e> and
// dS_e = p_e (dP_e - Delta_i):
//   dq_i   = tau sum_e dS_e khat_e
//   dk_j   = sum over entries e that read row j of  weight_e(j) tau dS_e q_i
//   dv_j   = sum over entries e that read row j of  weight_e(j) p_e dO_i
//   dL/dw  = tau dS_e <q_i, k[r1] - k[r0]> + p_e <dO_i, v[r1] - v[r0]>  (rung entries)
//   dalpha = sum_{b,h,i,rungs} f_k dL/dw
// The row -1 (reached only when w == 0) is a zero vector.
// dalpha is a sum with heavy cancellation (its magnitude is a small fraction of the
// sum of its terms' magnitudes), so it does not take Delta from the stored o (rounded
// to the storage type) but from the entries themselves, Delta_i = sum_e p_e dP_e (the
// same quantity, since o_i = sum_e p_e vhat_e): per query it accumulates
// Xa = sum f p dP <q, k[r1]-k[r0]>, Xb = sum f p <dO, v[r1]-v[r0]>, Y = sum f p <q, k[r1]-k[r0]>
// and the entries' sum of p dP, and adds tau (Xa - Delta Y) + Xb.
//
// Because every rung offset is shared, the queries that read key row j are again a
// fixed set of shifted positions: j .. j+W through the window, and j + floor(d_k)
// (as the row r0, weight 1-w) and j + floor(d_k) + 1 (as r1, weight w) through rung k.
// The dk/dv kernel therefore owns one key row per lane group and gathers its
// contributions, so every dk/dv row is written once, without atomics.
#include "launch.h"

namespace fibattn {

// ---------------------------------------------------------------------------
// dq, Delta and per-workgroup dalpha partials.
// ---------------------------------------------------------------------------
// DEV: the rung table is the one at rtp, built on the device (rt_arg unused).
template <typename S, int D, bool DEV>
__global__ __launch_bounds__(256) void bwd_dq_kernel(
    const S *__restrict__ q, const S *__restrict__ k, const S *__restrict__ v,
    const S *__restrict__ o, const float *__restrict__ lse, const S *__restrict__ dO,
    S *__restrict__ dq, float *__restrict__ delta_out, double *__restrict__ partials, int T,
    int W, RungTable rt_arg, const RungTable *__restrict__ rtp, float tau, Heads hd, Layouts lay) {
    const RungTable &rt = DEV ? *rtp : rt_arg;
    const bool bad = DEV && table_unusable(rt, W);  // bad device alpha, or another W
    constexpr int VN = Vec<S>::N;
    constexpr int LPQ = D / VN;
    constexpr int QPB = 256 / LPQ;
    __shared__ double red[256];

    const int g = threadIdx.x / LPQ;
    const int sub = threadIdx.x % LPQ;
    const int i = blockIdx.x * QPB + g;
    const int bk = hd.kv_of(blockIdx.y);
    const S *Q = q + lay.q.head(blockIdx.y, hd.H);
    const S *K = k + lay.k.head(bk, hd.kv_heads());
    const S *V = v + lay.v.head(bk, hd.kv_heads());
    const long long sq = lay.q.st, sk = lay.k.st, sv = lay.v.st;  // row strides
    const int col = sub * VN;
    const float sl2 = tau * kLog2e;

    double dal = 0.0;
    if (i < T) {
        float qv[VN], gv[VN], kv[VN], vv[VN], acc[VN];
        Vec<S>::load(Q + i * sq + col, qv);
        Vec<S>::load(dO + lay.g.head(blockIdx.y, hd.H) + i * lay.g.st + col, gv);
        Vec<S>::load(o + lay.o.head(blockIdx.y, hd.H) + i * lay.o.st + col, kv);
        const float delta = group_sum<LPQ>(dot<VN>(gv, kv));
        if (sub == 0) delta_out[(size_t)blockIdx.y * T + i] = bad ? NAN : delta;
        const float lse2 = lse[(size_t)blockIdx.y * T + i] * kLog2e;
#pragma unroll
        for (int c = 0; c < VN; ++c) acc[c] = 0.f;

        double xa = 0.0, xb = 0.0, y = 0.0, dsum = 0.0;  // dalpha parts, Delta from the entries
        const int wmax = min(W, i);
        for (int d = 0; d <= wmax; ++d) {
            Vec<S>::load(K + (i - d) * sk + col, kv);
            Vec<S>::load(V + (i - d) * sv + col, vv);
            const float s = group_sum<LPQ>(dot<VN>(qv, kv));
            const float dP = group_sum<LPQ>(dot<VN>(gv, vv));
            const float p = exp2f(s * sl2 - lse2);
            const float c = tau * p * (dP - delta);
            dsum += (double)p * (double)dP;
#pragma unroll
            for (int x = 0; x < VN; ++x) acc[x] = fmaf(c, kv[x], acc[x]);
        }
        for (int r = 0; r < rt.n; ++r) {
            const int d0 = rt.d0[r];
            const float w = rt.w[r];
            if (!(d0 < i || (d0 == i && w == 0.f))) break;
            const int r0 = i - d0;
            float k1[VN], v1[VN];
            Vec<S>::load(K + r0 * sk + col, kv);
            Vec<S>::load(V + r0 * sv + col, vv);
            if (r0 >= 1) {
                Vec<S>::load(K + (r0 - 1) * sk + col, k1);
                Vec<S>::load(V + (r0 - 1) * sv + col, v1);
            } else {
#pragma unroll
                for (int x = 0; x < VN; ++x) { k1[x] = 0.f; v1[x] = 0.f; }
            }
            const float s0 = group_sum<LPQ>(dot<VN>(qv, kv));
            const float s1 = group_sum<LPQ>(dot<VN>(qv, k1));
            const float dP0 = group_sum<LPQ>(dot<VN>(gv, vv));
            const float dP1 = group_sum<LPQ>(dot<VN>(gv, v1));
            const float s = (1.f - w) * s0 + w * s1;
            const float dP = (1.f - w) * dP0 + w * dP1;
            const float p = exp2f(s * sl2 - lse2);
            const float dS = p * (dP - delta);
            const float c = tau * dS;
            const float c0 = c * (1.f - w);
            const float c1 = c * w;
#pragma unroll
            for (int x = 0; x < VN; ++x) acc[x] = fmaf(c0, kv[x], fmaf(c1, k1[x], acc[x]));
            const double fp = (double)rt.f[r] * (double)p;
            xa += fp * (double)dP * (double)(s1 - s0);
            xb += fp * (double)(dP1 - dP0);
            y += fp * (double)(s1 - s0);
            dsum += (double)p * (double)dP;
        }
        dal = (double)tau * (xa - dsum * y) + xb;
        if (bad) {
#pragma unroll
            for (int x = 0; x < VN; ++x) acc[x] = NAN;
            dal = NAN;
        }
        Vec<S>::store(dq + lay.dq.head(blockIdx.y, hd.H) + i * lay.dq.st + col, acc);
    }
    red[threadIdx.x] = (sub == 0 && i < T) ? dal : 0.0;
    __syncthreads();
#pragma unroll
    for (int st = 128; st >= 1; st >>= 1) {
        if ((int)threadIdx.x < st) red[threadIdx.x] += red[threadIdx.x + st];
        __syncthreads();
    }
    if (threadIdx.x == 0) partials[(size_t)blockIdx.y * gridDim.x + blockIdx.x] = red[0];
}

// ---------------------------------------------------------------------------
// dk, dv: one key row per lane group.
// ---------------------------------------------------------------------------
template <typename S, int D, bool DEV>
__global__ __launch_bounds__(256) void bwd_dkdv_kernel(
    const S *__restrict__ q, const S *__restrict__ k, const S *__restrict__ v,
    const float *__restrict__ lse, const S *__restrict__ dO, const float *__restrict__ delta_in,
    S *__restrict__ dk, S *__restrict__ dv, int T, int W, RungTable rt_arg,
    const RungTable *__restrict__ rtp, float tau, Heads hd, Layouts lay) {
    const RungTable &rt = DEV ? *rtp : rt_arg;
    constexpr int VN = Vec<S>::N;
    constexpr int LPQ = D / VN;
    constexpr int QPB = 256 / LPQ;

    const int g = threadIdx.x / LPQ;
    const int sub = threadIdx.x % LPQ;
    const int j = blockIdx.x * QPB + g;
    if (j >= T) return;  // whole lane groups leave together; no block barrier below
    const int bk = blockIdx.y;  // batch * key/value heads + key/value head
    const S *K = k + lay.k.head(bk, hd.kv_heads());
    const S *V = v + lay.v.head(bk, hd.kv_heads());
    const long long sq = lay.q.st, sk = lay.k.st, sv = lay.v.st, sg = lay.g.st;  // row strides
    const int col = sub * VN;
    const float sl2 = tau * kLog2e;

    float kj[VN], vj[VN], adk[VN], adv[VN], qv[VN], gv[VN];
    Vec<S>::load(K + j * sk + col, kj);
    Vec<S>::load(V + j * sv + col, vj);
#pragma unroll
    for (int c = 0; c < VN; ++c) { adk[c] = 0.f; adv[c] = 0.f; }

    // every query head of the group reads this key row; their terms add up
    for (int hg = 0; hg < hd.G; ++hg) {
        const int bh = hd.q_of(blockIdx.y, hg);
        const S *Q = q + lay.q.head(bh, hd.H);
        const S *G = dO + lay.g.head(bh, hd.H);
        const float *L = lse + (size_t)bh * T;
        const float *Dl = delta_in + (size_t)bh * T;

        // window: queries i = j .. j+W read row j with weight 1
        const int imax = min(T - 1, j + W);
        for (int i = j; i <= imax; ++i) {
            Vec<S>::load(Q + i * sq + col, qv);
            Vec<S>::load(G + i * sg + col, gv);
            const float s = group_sum<LPQ>(dot<VN>(qv, kj));
            const float dP = group_sum<LPQ>(dot<VN>(gv, vj));
            const float p = exp2f(s * sl2 - L[i] * kLog2e);
            const float c = tau * p * (dP - Dl[i]);
#pragma unroll
            for (int x = 0; x < VN; ++x) {
                adk[x] = fmaf(c, qv[x], adk[x]);
                adv[x] = fmaf(p, gv[x], adv[x]);
            }
        }
        // rungs
        for (int r = 0; r < rt.n; ++r) {
            const int d0 = rt.d0[r];
            const float w = rt.w[r];
            const int i0 = j + d0;
            if (i0 >= T) break;  // d0 increases with r
            float kn[VN], vn[VN];
            // query i0 reads row j as r0 (weight 1-w) and row j-1 as r1; included iff w <= j
            if (w == 0.f || j >= 1) {
                Vec<S>::load(Q + i0 * sq + col, qv);
                Vec<S>::load(G + i0 * sg + col, gv);
                float s = (1.f - w) * dot<VN>(qv, kj);
                float dP = (1.f - w) * dot<VN>(gv, vj);
                if (w != 0.f) {
                    Vec<S>::load(K + (j - 1) * sk + col, kn);
                    Vec<S>::load(V + (j - 1) * sv + col, vn);
                    s = fmaf(w, dot<VN>(qv, kn), s);
                    dP = fmaf(w, dot<VN>(gv, vn), dP);
                }
                s = group_sum<LPQ>(s);
                dP = group_sum<LPQ>(dP);
                const float p = exp2f(s * sl2 - L[i0] * kLog2e);
                const float c = tau * p * (dP - Dl[i0]) * (1.f - w);
                const float pw = p * (1.f - w);
#pragma unroll
                for (int x = 0; x < VN; ++x) {
                    adk[x] = fmaf(c, qv[x], adk[x]);
                    adv[x] = fmaf(pw, gv[x], adv[x]);
                }
            }
            // query i0+1 reads row j+1 as r0 and row j as r1 (weight w); always included
            const int i1 = i0 + 1;
            if (w != 0.f && i1 < T) {
                Vec<S>::load(Q + i1 * sq + col, qv);
                Vec<S>::load(G + i1 * sg + col, gv);
                Vec<S>::load(K + (j + 1) * sk + col, kn);
                Vec<S>::load(V + (j + 1) * sv + col, vn);
                float s = fmaf(1.f - w, dot<VN>(qv, kn), w * dot<VN>(qv, kj));
                float dP = fmaf(1.f - w, dot<VN>(gv, vn), w * dot<VN>(gv, vj));
                s = group_sum<LPQ>(s);
                dP = group_sum<LPQ>(dP);
                const float p = exp2f(s * sl2 - L[i1] * kLog2e);
                const float c = tau * p * (dP - Dl[i1]) * w;
                const float pw = p * w;
#pragma unroll
                for (int x = 0; x < VN; ++x) {
                    adk[x] = fmaf(c, qv[x], adk[x]);
                    adv[x] = fmaf(pw, gv[x], adv[x]);
                }
            }
        }
    }
    if (DEV && table_unusable(rt, W)) {  // bad device alpha, or another W
#pragma unroll
        for (int x = 0; x < VN; ++x) { adk[x] = NAN; adv[x] = NAN; }
    }
    Vec<S>::store(dk + lay.dk.head(bk, hd.kv_heads()) + j * lay.dk.st + col, adk);
    Vec<S>::store(dv + lay.dv.head(bk, hd.kv_heads()) + j * lay.dv.st + col, adv);
}

// ---------------------------------------------------------------------------
// dalpha: one workgroup sums the partials in a fixed order, in float64.
// ---------------------------------------------------------------------------
// dtheta (device tables built from theta): dalpha (as stored) times d alpha / d theta.
__global__ __launch_bounds__(256) void dalpha_reduce_kernel(const double *__restrict__ partials,
                                                            size_t n, float *__restrict__ dalpha,
                                                            float *__restrict__ dtheta,
                                                            const RungTable *__restrict__ rtp) {
    __shared__ double red[256];
    double s = 0.0;
    for (size_t t = threadIdx.x; t < n; t += 256) s += partials[t];
    red[threadIdx.x] = s;
    __syncthreads();
#pragma unroll
    for (int st = 128; st >= 1; st >>= 1) {
        if ((int)threadIdx.x < st) red[threadIdx.x] += red[threadIdx.x + st];
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const float da = (float)red[0];
        *dalpha = da;
        if (dtheta) *dtheta = (float)((double)da * rtp->dadtheta);
    }
}

template <typename S, int D>
static size_t num_partials_t(int BH, int T) {
    constexpr int QPB = 256 / (D / Vec<S>::N);
    return (size_t)((T + QPB - 1) / QPB) * (size_t)BH;
}

size_t bwd_num_partials(int dtype, int D, int BH, int T) {
    if (dtype == 0 && D == 32) return num_partials_t<float, 32>(BH, T);
    if (dtype == 0 && D == 64) return num_partials_t<float, 64>(BH, T);
    if (dtype == 1 && D == 32) return num_partials_t<uint16_t, 32>(BH, T);
    if (dtype == 1 && D == 64) return num_partials_t<uint16_t, 64>(BH, T);
    if (dtype == 0 && D == 128) return num_partials_t<float, 128>(BH, T);
    if (dtype == 1 && D == 128) return num_partials_t<uint16_t, 128>(BH, T);
    return 0;
}

template <typename S, int D>
static hipError_t launch_bwd_t(const void *q, const void *k, const void *v, const void *o,
                               const float *lse, const void *dO, void *dq, void *dk, void *dv,
                               float *dalpha, float *dtheta, float *delta_ws, double *partials, int BH,
                               const Heads &hd, int T, int W, const RungTable &rt,
                               const RungTable *rtp, const Layouts &lay, hipStream_t s) {
    constexpr int QPB = 256 / (D / Vec<S>::N);
    const float tau = 1.f / sqrtf((float)D);
    dim3 grid((T + QPB - 1) / QPB, BH);
    hipError_t e = launch(kBwdDq, rtp ? bwd_dq_kernel<S, D, true> : bwd_dq_kernel<S, D, false>, grid,
                          dim3(256), 0, s, (const S *)q, (const S *)k, (const S *)v, (const S *)o,
                          lse, (const S *)dO, (S *)dq, delta_ws, partials, T, W, rt, rtp, tau, hd, lay);
    if (e != hipSuccess) return e;
    e = launch(kBwdDkDv, rtp ? bwd_dkdv_kernel<S, D, true> : bwd_dkdv_kernel<S, D, false>,
               dim3(grid.x, BH / hd.G), dim3(256), 0, s, (const S *)q, (const S *)k, (const S *)v,
               lse, (const S *)dO, delta_ws, (S *)dk, (S *)dv, T, W, rt, rtp, tau, hd, lay);
    if (e != hipSuccess) return e;
    return launch(kDalphaReduce, dalpha_reduce_kernel, dim3(1), dim3(256), 0, s, partials,
                  (size_t)grid.x * grid.y, dalpha, dtheta, rtp);
}

static hipError_t launch_backward_generic(int dtype, int D, const void *q, const void *k, const void *v,
                                          const void *o, const float *lse, const void *dO, void *dq,
                                          void *dk, void *dv, float *dalpha, float *dtheta, float *delta_ws,
                                          double *partials, int BH, const Heads &hd, int T, int W,
                                          const RungTable &rt, const RungTable *rtp, const Layouts &lay,
                                          hipStream_t s) {
#define FIBATTN_BWD(S_, D_)                                                                  \
    return launch_bwd_t<S_, D_>(q, k, v, o, lse, dO, dq, dk, dv, dalpha, dtheta, delta_ws, partials, \
                                BH, hd, T, W, rt, rtp, lay, s)
    if (dtype == 0 && D == 32) FIBATTN_BWD(float, 32);
    if (dtype == 0 && D == 64) FIBATTN_BWD(float, 64);
    if (dtype == 1 && D == 32) FIBATTN_BWD(uint16_t, 32);
    if (dtype == 1 && D == 64) FIBATTN_BWD(uint16_t, 64);
    if (dtype == 0 && D == 128) FIBATTN_BWD(float, 128);
    if (dtype == 1 && D == 128) FIBATTN_BWD(uint16_t, 128);
#undef FIBATTN_BWD
    return hipErrorInvalidValue;
}


hipError_t launch_backward(int dtype, int D, const void *q, const void *k, const void *v,
                           const void *o, const float *lse, const void *dO, void *dq, void *dk,
                           void *dv, float *dalpha, float *dtheta, float *delta_ws, double *partials,
                           const RungTerms &terms, int BH, const Heads &hd, int T, int W,
                           const RungTable &rt, const RungTable *rtp, const RopeFreq &rf,
                           float rope_base, const Layouts &lay, hipStream_t s) {
    if (backward_mfma_supported(dtype, D, W))
        return launch_backward_mfma(q, k, v, o, lse, dO, dq, dk, dv, dalpha, dtheta, delta_ws, partials,
                                    terms, BH, hd, T, W, rt, rtp, rf, lay, s);
    hipError_t e = launch_backward_generic(dtype, D, q, k, v, o, lse, dO, dq, dk, dv, dalpha, dtheta, delta_ws,
                                           partials, BH, hd, T, W, rt, rtp, lay, s);
    // R^T on dq and dk in place: gradients w.r.t. the unrotated q, k (R^T is linear, so
    // it also carries the group sum in dk)
    if (e == hipSuccess && rf.on) {
        e = launch_rope(dtype, D, dq, dq, lay.dq, lay.dq, dk, dk, lay.dk, lay.dk, BH, hd.H, T, rope_base, 1,
                        s, BH / hd.G, hd.kv_heads());
    }
    return e;
}

}  // namespace fibattn
