// Forward kernel: window band + shared rung offsets, softmax, weighted values, lse.
//
// Section 2 "Attended set": every query i of a (b, h) attends to distances 0..W and to
// the rung distances d_k = alpha f_k, each rung read as the blend of rows
// i - floor(d_k) (weight 1 - w_k) and i - floor(d_k) - 1 (weight w_k).  Because the
// offsets are shared, a block of consecutive queries reads, for each rung, one
// contiguous shifted block of key/value rows.
//
// Layout: a group of LPQ = D / VN lanes owns one query; lane `sub` holds dims
// [sub*VN, sub*VN + VN) (16 bytes of the row), so a row load by a group is one
// coalesced 64- or 128-byte access and consecutive groups read consecutive rows.
// Pass 1 computes the scaled logits (blend done in score space: the logit of a rung
// is (1-w) <q, k[r0]> + w <q, k[r1]>) into LDS and their maximum; pass 2 forms the
// probabilities and the weighted sum of values.  The whole softmax runs in base 2.
#include "launch.h"

namespace fibattn {

// DEV: the rung table is the one at rtp, built on the device (rt_arg unused).
template <typename S, int D, bool DEV>
__global__ __launch_bounds__(256) void fwd_kernel(const S *__restrict__ q, const S *__restrict__ k,
                                                  const S *__restrict__ v, S *__restrict__ o,
                                                  float *__restrict__ lse, int T, int W,
                                                  RungTable rt_arg, const RungTable *__restrict__ rtp,
                                                  float scale_log2, Heads hd, Layouts lay) {
    const RungTable &rt = DEV ? *rtp : rt_arg;
    constexpr int VN = Vec<S>::N;
    constexpr int LPQ = D / VN;
    constexpr int QPB = 256 / LPQ;
    extern __shared__ float smem[];

    const int cap = W + 1 + (DEV ? kMaxRungs : rt.n);  // LDS logits per query
    const int g = threadIdx.x / LPQ;
    const int sub = threadIdx.x % LPQ;
    const int i = blockIdx.x * QPB + g;
    const int bk = hd.kv_of(blockIdx.y);
    const S *Q = q + lay.q.head(blockIdx.y, hd.H);
    const S *K = k + lay.k.head(bk, hd.kv_heads());
    const S *V = v + lay.v.head(bk, hd.kv_heads());
    const long long sq = lay.q.st, sk = lay.k.st, sv = lay.v.st;  // row strides
    float *sc = smem + g * cap;
    const int col = sub * VN;

    float m = -INFINITY;
    if (i < T) {
        float qv[VN], kv[VN];
        Vec<S>::load(Q + i * sq + col, qv);
        int e = 0;
        const int wmax = min(W, i);
        for (int d = 0; d <= wmax; ++d, ++e) {
            Vec<S>::load(K + (i - d) * sk + col, kv);
            const float s = group_sum<LPQ>(dot<VN>(qv, kv)) * scale_log2;
            if (sub == 0) sc[e] = s;
            m = fmaxf(m, s);
        }
        for (int r = 0; r < rt.n; ++r, ++e) {
            const int d0 = rt.d0[r];
            const float w = rt.w[r];
            if (!(d0 < i || (d0 == i && w == 0.f))) break;  // d_k > i: before position 0
            const int r0 = i - d0;
            Vec<S>::load(K + r0 * sk + col, kv);
            float part = (1.f - w) * dot<VN>(qv, kv);
            if (w != 0.f) {
                Vec<S>::load(K + (r0 - 1) * sk + col, kv);
                part = fmaf(w, dot<VN>(qv, kv), part);
            }
            const float s = group_sum<LPQ>(part) * scale_log2;
            if (sub == 0) sc[e] = s;
            m = fmaxf(m, s);
        }
    }
    __syncthreads();
    if (i < T) {
        float acc[VN], vv[VN];
#pragma unroll
        for (int c = 0; c < VN; ++c) acc[c] = 0.f;
        float l = 0.f;
        int e = 0;
        const int wmax = min(W, i);
        for (int d = 0; d <= wmax; ++d, ++e) {
            const float p = exp2f(sc[e] - m);
            l += p;
            Vec<S>::load(V + (i - d) * sv + col, vv);
#pragma unroll
            for (int c = 0; c < VN; ++c) acc[c] = fmaf(p, vv[c], acc[c]);
        }
        for (int r = 0; r < rt.n; ++r, ++e) {
            const int d0 = rt.d0[r];
            const float w = rt.w[r];
            if (!(d0 < i || (d0 == i && w == 0.f))) break;
            const float p = exp2f(sc[e] - m);
            l += p;
            const int r0 = i - d0;
            const float p0 = p * (1.f - w);
            Vec<S>::load(V + r0 * sv + col, vv);
#pragma unroll
            for (int c = 0; c < VN; ++c) acc[c] = fmaf(p0, vv[c], acc[c]);
            if (w != 0.f) {
                const float p1 = p * w;
                Vec<S>::load(V + (r0 - 1) * sv + col, vv);
#pragma unroll
                for (int c = 0; c < VN; ++c) acc[c] = fmaf(p1, vv[c], acc[c]);
            }
        }
        const bool bad = DEV && table_unusable(rt, W);  // bad device alpha, or another W
        const float inv = bad ? NAN : 1.f / l;
#pragma unroll
        for (int c = 0; c < VN; ++c) acc[c] *= inv;
        Vec<S>::store(o + lay.o.head(blockIdx.y, hd.H) + i * lay.o.st + col, acc);
        if (sub == 0) lse[(size_t)blockIdx.y * T + i] = bad ? NAN : (m + log2f(l)) * kLn2;
    }
}

template <typename S, int D>
static hipError_t launch_fwd_t(const void *q, const void *k, const void *v, void *o, float *lse,
                               int BH, const Heads &hd, int T, int W, const RungTable &rt,
                               const RungTable *rtp, const Layouts &lay, hipStream_t s) {
    constexpr int LPQ = D / Vec<S>::N;
    constexpr int QPB = 256 / LPQ;
    dim3 grid((T + QPB - 1) / QPB, BH);
    const size_t lds = sizeof(float) * QPB * (size_t)(W + 1 + (rtp ? kMaxRungs : rt.n));
    const float scale_log2 = kLog2e / sqrtf((float)D);
    return launch(kForward, rtp ? fwd_kernel<S, D, true> : fwd_kernel<S, D, false>, grid, dim3(256),
                  (unsigned)lds, s, (const S *)q, (const S *)k, (const S *)v, (S *)o, lse, T, W, rt,
                  rtp, scale_log2, hd, lay);
}

hipError_t launch_forward(int dtype, int D, const void *q, const void *k, const void *v, void *o,
                          float *lse, int BH, const Heads &hd, int T, int W, const RungTable &rt,
                          const RungTable *rtp, const Layouts &lay, hipStream_t s) {
    if (forward_mfma_supported(dtype, D, W))
        return launch_forward_mfma(q, k, v, o, lse, BH, hd, T, W, rt, rtp, lay, s);
    if (dtype == 0 && D == 32) return launch_fwd_t<float, 32>(q, k, v, o, lse, BH, hd, T, W, rt, rtp, lay, s);
    if (dtype == 0 && D == 64) return launch_fwd_t<float, 64>(q, k, v, o, lse, BH, hd, T, W, rt, rtp, lay, s);
    if (dtype == 1 && D == 32) return launch_fwd_t<uint16_t, 32>(q, k, v, o, lse, BH, hd, T, W, rt, rtp, lay, s);
    if (dtype == 1 && D == 64) return launch_fwd_t<uint16_t, 64>(q, k, v, o, lse, BH, hd, T, W, rt, rtp, lay, s);
    if (dtype == 0 && D == 128) return launch_fwd_t<float, 128>(q, k, v, o, lse, BH, hd, T, W, rt, rtp, lay, s);
    if (dtype == 1 && D == 128) return launch_fwd_t<uint16_t, 128>(q, k, v, o, lse, BH, hd, T, W, rt, rtp, lay, s);
    return hipErrorInvalidValue;
}

}  // namespace fibattn
