// Forward for bfloat16, d_head = 64, W <= 16 on gfx950 matrix cores + VALU.
//
// Section 2 "Attended set": query i attends distances 0..W and the rung distances
// d_k = alpha f_k, shared by all queries.  A workgroup owns 64 consecutive queries of
// one (batch, head) (four waves of 16).  For a wave's queries [t0, t0+16):
//   - the window band lies in the 32 key rows [t0-16, t0+16).  Its logits are one
//     16x32 tile of Q.K^T on the matrix cores, masked to 0 <= i - j <= W; the
//     probability-weighted values are (V^T P^T) on the matrix cores; the band's K
//     and V rows are copied to LDS once per workgroup with direct-to-LDS loads;
//   - every rung is a contiguous shifted block: query t0+n reads rows t0+n-floor(d)
//     and t0+n-floor(d)-1.  Those logits are per-row dot products (bf16 dot2, four
//     lanes per row) blended in score space; the blended values are accumulated on
//     the VALU in the same register layout as the matrix-core output.  With
//     interpolation the staged rows reach 32 rows below the tile, and the short
//     rungs whose two rows lie there are read from LDS instead of the L2.  (With
//     every w == 0 the wider stage does not pay: the first rung read from global
//     memory would start late.)
// Softmax runs in base 2: the band's maximum is the first running reference, then
// rungs are taken a batch at a time (their key and value rows loaded together),
// rescaling the running sum and weighted values only when a logit exceeds the
// reference by a wide margin.  The layer step's instance also applies RoPE to q where
// it loads it (RQ below).
#include "launch.h"
#include "mfma.h"

namespace fibattn {

constexpr int kFwdBQ = 64;                 // queries per workgroup
constexpr float kSlack = 8.f;              // log2 units a logit may exceed the running reference

// INTERP: some rung has w != 0, so the second row r1 is read.  DEV: the rung table
// is the one at rtp, built on the device (rt_arg unused).  STRIDED: rows are placed
// by the layouts' position strides (else every row stride is 64, a constant).
// HS: query heads per workgroup, all reading one key/value head (grouped heads): the
// four waves are HS heads times 4/HS runs of 16 queries at the same positions, so the
// staged band rows serve every head of the group and the rung rows the heads gather
// are the same addresses (HS = 1: one head, 64 queries).
// RQ: q holds the raw (unrotated) queries and k the rotated keys.  Each lane rotates its
// own slice of its query row at the query's position (RoPE, Section 2 "Attended set"),
// attends with the rotated row and, when qrot is not null, writes it there for the
// backward, placed by lay.dq (the forward has no dq of its own).  A query row is used by
// one query only, so rotating it where it is loaded costs no extra row traffic; a key
// row is read by up to 1 + W + K queries and stays with the RoPE launch.  rf: the RoPE
// frequencies (unused without RQ).
template <bool INTERP, bool DEV, bool STRIDED, int HS, bool RQ>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void fwd_bf16_d64_kernel(
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k, const uint16_t *__restrict__ v,
    uint16_t *__restrict__ o, float *__restrict__ lse, int T, int W, RungTable rt_arg,
    const RungTable *__restrict__ rtp, float sl2, int tiles, Heads hd, Layouts lay,
    uint16_t *qrot, RopeFreq rf) {
    const RungTable &rt = DEV ? *rtp : rt_arg;
    constexpr int RB = INTERP ? 1 : 2;  // rungs per load batch; two batches in flight
    constexpr int NS = INTERP ? 2 : 1;  // rows per rung (r0, and r1 when interpolating)
    constexpr int kQ = kFwdBQ / HS;     // queries per workgroup and head
    // staged rows [T0 - kLeadF, T0 + kQ): the band and, interpolating, the short rungs
    constexpr int kLeadF = INTERP ? 32 : 16;
    constexpr int kBandRows = kQ + kLeadF;
    __shared__ __align__(16) uint16_t kr[kBandRows * kD];
    __shared__ __align__(16) uint16_t vr[kBandRows * kD];
    __shared__ double sfreq[RQ ? 32 : 1];  // RoPE frequencies, revolutions per position

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform: scalar work
    const int wv = wave / HS;                  // run of 16 queries
    const int nm = lane & 15, gm = lane >> 4;  // MFMA layout
    const int nq = lane >> 2, gq = lane & 3;   // quad layout
    // Raised issue priority while this wave sets up and issues its row copies, so a
    // starting workgroup's loads are not queued behind resident waves' rung arithmetic.
    __builtin_amdgcn_s_setprio(2);
    const int blk = xcd_remap(blockIdx.x, gridDim.x);
    const int bh = (blk / tiles) * HS + wave % HS;  // this wave's query head
    const int T0 = (blk % tiles) * kQ;
    const int bk = hd.kv_of(bh);
    const uint16_t *Q = q + head_at<STRIDED, kD>(lay.q, bh, hd.H, T);
    const uint16_t *K = k + head_at<STRIDED, kD>(lay.k, bk, hd.kv_heads(), T);
    const uint16_t *V = v + head_at<STRIDED, kD>(lay.v, bk, hd.kv_heads(), T);
    // row strides
    const int stq = STRIDED ? (int)lay.q.st : kD, stk = STRIDED ? (int)lay.k.st : kD;
    const int stv = STRIDED ? (int)lay.v.st : kD, sto = STRIDED ? (int)lay.o.st : kD;

    const int t0 = T0 + 16 * wv;
    const int last = t0 + 15;  // the wave's last query
    // rows [T0-kLeadF, T0+64) of K and V, straight to LDS (rows outside [0, T) are
    // clamped copies: their keys are masked below).  They need no table entry, so they
    // are issued before the wave waits for the rung table's scalar loads (strided rows:
    // after the first rung batch, which keeps the strided instance free of spills).
    auto stage_band = [&]() {
        dma_rows<kBandRows>(kr, K, T0 - kLeadF, T, stk);
        dma_rows<kBandRows>(vr, V, T0 - kLeadF, T, stv);
    };
    if constexpr (!STRIDED) stage_band();
    // rungs some query of this wave includes: a prefix of the table (sorted by d).  A
    // table in device memory is tested entry by entry unconditionally (entries past n are
    // zero), so it is fetched with a few wide scalar loads rather than a chain of
    // dependent ones; a table in the kernel arguments keeps the short-circuit form.
    int nact = 0;
#pragma unroll
    for (int r = 0; r < kMaxRungs; ++r)
        nact += (DEV ? ((r < rt.n) & (rt.d0[r] <= last)) : (r < rt.n && rt.d0[r] <= last)) ? 1 : 0;
    nact = __builtin_amdgcn_readfirstlane(nact);  // wave-uniform: scalar branches
    // rungs whose rows (r0 and, interpolating, r1) for every query of the wave lie in
    // the staged rows: a prefix of the table
    int nlds = 0;
#pragma unroll
    for (int r = 0; r < kMaxRungs; ++r)
        nlds += (INTERP && (DEV ? ((r < rt.n) & (rt.d0[r] + NS - 1 <= kLeadF + 16 * wv))
                                : (r < rt.n && rt.d0[r] + NS - 1 <= kLeadF + 16 * wv))) ? 1 : 0;
    nlds = __builtin_amdgcn_readfirstlane(nlds);

    const int im = t0 + nm;  // query of this lane in the MFMA layout
    const int i = t0 + nq;   // ... in the quad layout
    const int ic = min(i, T - 1);
    Slice qq = load_row(Q, ic, gq, stq);  // raw with RQ, rotated after the wait below
    // RQ: cos and sin of the lane's eight angles (its query's position, frequencies
    // 8 gq .. 8 gq + 7), evaluated while the row copies are in flight
    float rc[RQ ? 8 : 1], rs[RQ ? 8 : 1];
    if constexpr (RQ) {
        stage_freq(sfreq, rf);
        __syncthreads();
#pragma unroll
        for (int d = 0; d < 8; ++d) rope_cs_rev(i, sfreq[8 * gq + d], rc[d], rs[d]);
    }

    // rung rows of a batch: kx[x*NS + s], vx[x*NS + s] = row r_s of rung rb + x
    // (from LDS for the first nlds rungs, else from global memory; `which` selects
    // 1 = global rungs only, 2 = LDS rungs only, 3 = both)
    auto load_batch = [&](int rb, Slice *kx, Slice *vx, int which) {
#pragma unroll
        for (int x = 0; x < RB; ++x) {
            if (rb + x < nlds) {
                if (which & 2) {
                    const int L0 = 16 * wv + nq + kLeadF - rt.d0[rb + x];
#pragma unroll
                    for (int sidx = 0; sidx < NS; ++sidx) {
                        kx[x * NS + sidx] = dma_slice(kr, L0 - sidx, gq);
                        vx[x * NS + sidx] = dma_slice(vr, L0 - sidx, gq);
                    }
                }
            } else if (which & 1) {
                const int R0 = max(ic - rt.d0[rb + x], 0);  // a query past T is masked
#pragma unroll
                for (int sidx = 0; sidx < NS; ++sidx) {
                    const int R = max(R0 - sidx, 0);
                    kx[x * NS + sidx] = load_row(K, R, gq, stk);
                    vx[x * NS + sidx] = load_row(V, R, gq, stv);
                }
            }
        }
    };
    Slice kA[RB * NS], vA[RB * NS], kB[RB * NS], vB[RB * NS];
    if (0 < nact) load_batch(0, kA, vA, 1);  // in flight during the band phase
    if constexpr (STRIDED) stage_band();
    __builtin_amdgcn_s_setprio(0);
    wait_vmem();
    __syncthreads();
    if (0 < nact) load_batch(0, kA, vA, 2);
    if constexpr (RQ) {
        // rotate-half pairs (8g + d, 32 + 8g + d) are slice positions d and d + 8: word w
        // of a holds d = 2w, 2w + 1, word w of b their partners
        uint32_t aw[4] = {qq.a.x, qq.a.y, qq.a.z, qq.a.w}, bw[4] = {qq.b.x, qq.b.y, qq.b.z, qq.b.w};
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            float x0, y0, x1, y1;
            rope_rotate(bf16_lo(aw[w]), bf16_lo(bw[w]), rc[2 * w], rs[2 * w], x0, y0);
            rope_rotate(bf16_hi(aw[w]), bf16_hi(bw[w]), rc[2 * w + 1], rs[2 * w + 1], x1, y1);
            aw[w] = pack_bf16(x0, x1);  // round to nearest even, as the RoPE launch
            bw[w] = pack_bf16(y0, y1);
        }
        qq.a = make_uint4(aw[0], aw[1], aw[2], aw[3]);
        qq.b = make_uint4(bw[0], bw[1], bw[2], bw[3]);
        if (qrot && i < T) {  // read by the backward: ordinary stores
            uint16_t *qr = qrot + head_at<STRIDED, kD>(lay.dq, bh, hd.H, T) +
                           (size_t)i * (STRIDED ? (int)lay.dq.st : kD);
            *reinterpret_cast<uint4 *>(qr + 8 * gq) = qq.a;
            *reinterpret_cast<uint4 *>(qr + 32 + 8 * gq) = qq.b;
        }
    }

    // ---- window band (MFMA layout): logits (log2 units), maximum, probabilities ----
    const Slice qm = slice_from_quad(qq, lane);  // the wave's q rows in the MFMA layout
    float m = -INFINITY;
    f32x4 sb[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        const Slice kb = dma_slice(kr, kLeadF - 16 + 16 * wv + 16 * b + nm, gm);
        sb[b] = mfma_dot64(kb, qm, f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int key = t0 - 16 + 16 * b + 4 * gm + e;
            const bool ok = key >= 0 && key <= im && im - key <= W;
            sb[b][e] = ok ? sb[b][e] * sl2 : -INFINITY;
            m = fmaxf(m, sb[b][e]);
        }
    }
    m = max4(m);  // finite: key im itself is always in the band
    float l = 0.f;
    uint32_t pw[4];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        float p[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            p[e] = fast_exp2(sb[b][e] - m);
            l += p[e];
        }
        pw[2 * b] = pack_bf16(p[0], p[1]);
        pw[2 * b + 1] = pack_bf16(p[2], p[3]);
    }
    l = sum4(l);
    const bf16x8 P = as_bf8(make_uint4(pw[0], pw[1], pw[2], pw[3]));
    // V^T.P^T, the A operand gathered from the row-major staged V
    Acc16 acc;
#pragma unroll
    for (int c = 0; c < 4; ++c)
        acc.c[c] = mfma(dma_operand_t(vr, c, nm, kLeadF - 16 + 16 * wv, gm), P, f32x4{0.f, 0.f, 0.f, 0.f});
    // hand the band results to the quad layout
    acc_to_quad(acc, lane);
    m = to_quad(m, lane);
    l = to_quad(l, lane);

    // ---- rungs (quad layout): logits of a batch, running reference, values ----
    auto compute_batch = [&](int rb, const Slice *kx, const Slice *vx) {
        float s[RB];
        float mb = m;
#pragma unroll
        for (int x = 0; x < RB; ++x) {
            const int r = rb + x;
            const int d0 = rt.d0[r];
            const float w = rt.w[r];
            // with every w == 0 a rung is in the set of query i iff d0 <= i
            const bool incl = r < nact && (INTERP ? (d0 < i || (d0 == i && w == 0.f)) : d0 <= i);
            float part = dot_slice(qq, kx[x * NS]);
            if (INTERP) part = (1.f - w) * part + w * dot_slice(qq, kx[x * NS + 1]);
            part = quad_sum(part) * sl2;
            s[x] = incl ? part : -INFINITY;
            mb = fmaxf(mb, s[x]);
        }
        // The running reference m moves only when a logit exceeds it by more than
        // kSlack (log2 units), so exp2(s - m) <= 2^kSlack stays far inside float32
        // range; o = acc / l and lse = m + log2(l) hold for any reference, and the
        // rescale of acc and l is skipped unless some lane of the wave needs it.
        const bool grow = mb > m + kSlack;
        if (__builtin_amdgcn_ballot_w64(grow)) {
            const float mn = grow ? mb : m;
            const float scale = fast_exp2(m - mn);
            m = mn;
            l *= scale;
#pragma unroll
            for (int c = 0; c < 4; ++c) acc.c[c] *= scale;
        }
        float p[RB];
#pragma unroll
        for (int x = 0; x < RB; ++x) {
            p[x] = fast_exp2(s[x] - m);
            l += p[x];
        }
        if (INTERP) {
            const float w = rt.w[rb];
            acc_axpy2(acc, p[0] * (1.f - w), vx[0], p[0] * w, vx[1]);
        } else {
            acc_axpy2(acc, p[0], vx[0], p[1], vx[1]);
        }
    };

    // two batches in flight: load the next while computing the current
#pragma unroll
    for (int rb = 0; rb < kMaxRungs; rb += 2 * RB) {
        if (rb < nact) {
            if (rb + RB < nact) load_batch(rb + RB, kB, vB, 3);
            compute_batch(rb, kA, vA);
            if (rb + RB < nact) {
                if (rb + 2 * RB < nact) load_batch(rb + 2 * RB, kA, vA, 3);
                compute_batch(rb + RB, kB, vB);
            }
        }
    }

    if (i < T) {
        const bool bad = DEV && table_unusable(rt, W);  // bad device alpha, or another W
        store_acc(o + head_at<STRIDED, kD>(lay.o, bh, hd.H, T) + (size_t)i * sto, gq, acc, bad ? NAN : 1.f / l);
        if (gq == 0) __builtin_nontemporal_store(bad ? NAN : (m + log2f(l)) * kLn2, lse + (size_t)bh * T + i);
    }
}

static bool any_interp(const RungTable &rt) {
    for (int r = 0; r < rt.n; ++r)
        if (rt.w[r] != 0.f) return true;
    return false;
}

bool forward_mfma_supported(int dtype, int D, int W) { return dtype == 1 && D == 64 && W <= 16; }

// Query heads per workgroup for G query heads per key/value head (packed tensors with a
// host table; other launches take one head per workgroup).
static int heads_per_wg(int G) { return G % 4 == 0 ? 4 : G % 2 == 0 ? 2 : 1; }

hipError_t launch_forward_mfma(const void *q, const void *k, const void *v, void *o, float *lse,
                               int BH, const Heads &hd, int T, int W, const RungTable &rt,
                               const RungTable *rtp, const Layouts &lay, hipStream_t s,
                               const RopeFreq *rq, void *q_rot) {
    const float sl2 = kLog2e / sqrtf(64.f);
    // device tables come with packed tensors only; rotation on load places R q by lay.dq
    const int hk = hd.kv_heads();
    const bool strided = !is_packed(lay.q, hd.H, T, kD) || !is_packed(lay.k, hk, T, kD) ||
                         !is_packed(lay.v, hk, T, kD) || !is_packed(lay.o, hd.H, T, kD) ||
                         (rq && q_rot && !is_packed(lay.dq, hd.H, T, kD));
    if (rtp && strided) return hipErrorInvalidValue;
    const bool interp = any_interp(rt);
    const int hs = (rtp || strided) ? 1 : heads_per_wg(hd.G);
    const int tiles = (T + kFwdBQ / hs - 1) / (kFwdBQ / hs);  // runs of 64 / hs queries
#define FIBATTN_FWD(I, H, R) fwd_bf16_d64_kernel<I, false, false, H, R>
#define FIBATTN_FWD_HS(R)                                                                        \
    (hs == 4   ? (interp ? FIBATTN_FWD(true, 4, R) : FIBATTN_FWD(false, 4, R))                \
     : hs == 2 ? (interp ? FIBATTN_FWD(true, 2, R) : FIBATTN_FWD(false, 2, R))                \
               : (interp ? FIBATTN_FWD(true, 1, R) : FIBATTN_FWD(false, 1, R)))
    auto kern = rtp ? (rq ? fwd_bf16_d64_kernel<true, true, false, 1, true> : fwd_bf16_d64_kernel<true, true, false, 1, false>)
              : strided ? (rq ? (interp ? fwd_bf16_d64_kernel<true, false, true, 1, true>
                                        : fwd_bf16_d64_kernel<false, false, true, 1, true>)
                              : (interp ? fwd_bf16_d64_kernel<true, false, true, 1, false>
                                        : fwd_bf16_d64_kernel<false, false, true, 1, false>))
              : rq ? FIBATTN_FWD_HS(true) : FIBATTN_FWD_HS(false);
#undef FIBATTN_FWD_HS
#undef FIBATTN_FWD
    return launch(kForward, kern, dim3(tiles * (BH / hs)), dim3(256), 0, s, q, k, v, o, lse, T, W, rt, rtp,
                  sl2, tiles, hd, lay, (uint16_t *)q_rot, rq ? *rq : RopeFreq{});
}

}  // namespace fibattn
