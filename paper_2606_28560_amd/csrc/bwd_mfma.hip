// Backward for bfloat16, d_head = 64, W <= 16 on gfx950 matrix cores + VALU.
//
// Same gradient as bwd.hip (the forward's exact gradient with the inclusion masks
// held constant, Section 2 "Implementation note"), organised like fwd_mfma.hip:
//
// dq kernel (query-stationary, 64 queries per workgroup, 16 per wave):
//   band:  S^T = K.Q^T and dP^T = V.dO^T on the matrix cores (16x32 tiles),
//          dS = P (dP - Delta), dq^T += K^T (tau dS)^T; the band's K and V rows are
//          copied to LDS with direct-to-LDS loads;
//   rungs: per-row bf16 dot2 products for <q, k[r0]>, <q, k[r1]>, <dO, v[r0]>,
//          <dO, v[r1]> (the r1 terms are needed for dalpha even when w = 0; with
//          interpolation the rows of short rungs come from the staged rows, which
//          then reach 32 rows below the tile),
//          dq += tau dS ((1-w) k[r0] + w k[r1]) on the VALU,
//          dalpha partial += f (tau dS <q, k[r1]-k[r0]> + p <dO, v[r1]-v[r0]>), where
//          the dS of this sum uses Delta_i = sum_e p_e dP_e over the query's entries
//          rather than the one from the stored (bf16) o;
//   writes dq, Delta_i = <dO_i, o_i>, one float64 dalpha partial per workgroup
//   (each query's terms in float32, then float64 across queries) and, for every rung
//   entry, the pair (tau dS, p) as bfloat16 (the rung terms, staged in LDS during the
//   rung loop and copied out by each wave after it);
// dk/dv kernel (key-stationary, 64 keys per workgroup, 16 per wave): the queries
// that read key row j are j..j+W (window) and, for rung k, j+floor(d_k) (as row r0,
// weight 1-w) and j+floor(d_k)+1 (as row r1, weight w):
//   band:  S = Q.K^T and dP = dO.V^T tiles, dk^T += Q^T (tau dS), dv^T += dO^T P with
//          the band's q and dO rows copied to LDS with direct-to-LDS loads;
//   rungs: dk += (tau dS) q and dv += p dO with the dq kernel's rung terms, so a rung
//          reads only the q and dO rows of its queries (bf16 dot2 accumulation, two
//          rungs or one interpolated rung per batch, two batches in flight);
//   each dk/dv row is written once; no atomics.  Workgroup 0 also sums the dalpha
//   partials in a fixed order (float64), after the dq kernel has finished.
#include "launch.h"
#include "mfma.h"

namespace fibattn {

constexpr int kBwdB = 64;                // rows per workgroup

// ---------------------------------------------------------------------------
// INTERP: some rung has w != 0 (rows r0 and r1 both loaded per rung).  DEV: the rung
// table is the one at rtp, built on the device (rt_arg unused).  STRIDED: rows placed
// by the layouts' position strides (else every row stride is 64, a constant).
// HS: query heads per workgroup, all reading one key/value head: the four waves are HS
// heads times 4/HS runs of 16 queries at the same positions (as in the forward), so the
// staged K, V rows serve every head of the group.
template <bool INTERP, bool DEV, bool STRIDED, int HS>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void bwd_dq_bf16_d64_kernel(
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k, const uint16_t *__restrict__ v,
    const uint16_t *__restrict__ o, const float *__restrict__ lse, const uint16_t *__restrict__ dO,
    uint16_t *__restrict__ dq, float *__restrict__ delta_out, double *__restrict__ partials,
    RungTerms terms, int T, int W, RungTable rt_arg, const RungTable *__restrict__ rtp, RopeFreq rf,
    float tau, int tiles, Heads hd, Layouts lay) {
    const RungTable &rt = DEV ? *rtp : rt_arg;
    const bool bad = DEV && table_unusable(rt, W);  // bad device alpha, or another W
    // staged K, V rows [T0 - kLeadQ, T0 + 64): the band and, interpolating, the short rungs
    constexpr int kQ = kBwdB / HS;  // queries per workgroup and head
    constexpr int kLeadQ = INTERP ? 32 : 16;
    constexpr int kStage = kQ + kLeadQ;
    __shared__ __align__(16) uint16_t kr[kStage * kD];
    __shared__ __align__(16) uint16_t vr[kStage * kD];
    __shared__ double sfreq[32];
    __shared__ double red[4];
    // (tau dS, p) of every rung entry of the tile's queries, copied to terms.p at the end
    // (stores inside the rung loop would hold up its loads: they share one counter)
    __shared__ uint32_t sterm[kMaxRungs * kBwdB];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform: scalar work
    const int wv = wave / HS;  // run of 16 queries
    const int nm = lane & 15, gm = lane >> 4;  // MFMA layout
    const int nq = lane >> 2, gq = lane & 3;   // quad layout
    // Raised issue priority while the prologue's loads and row copies are issued (as
    // in the forward); dk/dv keeps the default (measured slower at T = 4096).
    __builtin_amdgcn_s_setprio(2);
    // Each XCD serves its work items last-first, while dk/dv (the next kernel) serves its
    // own first-first and an XCD keeps the same heads in both: the tiles dk/dv starts
    // with are then the ones this kernel touched last, whose rows and rung terms are
    // still in the XCD's L2 (dk/dv -0.4 us, T = 1024 step -1 us, T = 4096 step -1.8 us).
    int blk = xcd_remap(blockIdx.x, gridDim.x);
    if ((gridDim.x & 7) == 0) {
        const int per = gridDim.x >> 3, x = blk / per;
        blk = x * per + (per - 1 - (blk - x * per));
    }
    const int bh = (blk / tiles) * HS + wave % HS;  // this wave's query head
    const int T0 = (blk % tiles) * kQ;
    const int bk = hd.kv_of(bh);
    const uint16_t *Q = q + head_at<STRIDED, kD>(lay.q, bh, hd.H, T);
    const uint16_t *K = k + head_at<STRIDED, kD>(lay.k, bk, hd.kv_heads(), T);
    const uint16_t *V = v + head_at<STRIDED, kD>(lay.v, bk, hd.kv_heads(), T);
    const uint16_t *G = dO + head_at<STRIDED, kD>(lay.g, bh, hd.H, T);
    // row strides
    const int stq = STRIDED ? (int)lay.q.st : kD, stk = STRIDED ? (int)lay.k.st : kD;
    const int stv = STRIDED ? (int)lay.v.st : kD, stg = STRIDED ? (int)lay.g.st : kD;
    const int sto = STRIDED ? (int)lay.o.st : kD, stdq = STRIDED ? (int)lay.dq.st : kD;
    const float *L = lse + (size_t)bh * T;
    const float sl2 = tau * kLog2e;

    const int t0 = T0 + 16 * wv;
    const int im = t0 + nm, imc = min(im, T - 1);  // MFMA layout query
    const int i = t0 + nq, ic = min(i, T - 1);     // quad layout query
    const Slice qq = load_row(Q, ic, gq, stq);
    const Slice gqq = load_row(G, ic, gq, stg);
    // the same rows in the MFMA layout, by lane shuffles rather than a second read
    const Slice qm = slice_from_quad(qq, lane);
    const Slice gmm = slice_from_quad(gqq, lane);
    const Slice oq = load_row(o + head_at<STRIDED, kD>(lay.o, bh, hd.H, T), ic, gq, sto);
    const float lse2 = L[ic] * kLog2e;
    const float lse2_m = L[imc] * kLog2e;

    const int last = t0 + 15;
    int nact = 0;
#pragma unroll
    // (a device table is tested unconditionally: wide scalar loads, no chain of dependent ones)
    for (int r = 0; r < kMaxRungs; ++r)
        nact += (DEV ? ((r < rt.n) & (rt.d0[r] <= last)) : (r < rt.n && rt.d0[r] <= last)) ? 1 : 0;
    nact = __builtin_amdgcn_readfirstlane(nact);  // wave-uniform: scalar branches
    // rungs whose rows r0 and r1 for every query of the wave lie in the staged rows
    int nlds = 0;
#pragma unroll
    for (int r = 0; r < kMaxRungs; ++r)
        nlds += (INTERP && (DEV ? ((r < rt.n) & (rt.d0[r] + 1 <= kLeadQ + 16 * wv))
                                : (r < rt.n && rt.d0[r] + 1 <= kLeadQ + 16 * wv))) ? 1 : 0;
    nlds = __builtin_amdgcn_readfirstlane(nlds);
    // x = {k0, v0, k1, v1}: rows r0 and r1 = r0 - 1 of K and V (r1 is needed for
    // dalpha even when w == 0; then it is row r0 of the previous query, but loading it
    // costs less than moving it across lanes).  Rows of the first nlds rungs come from
    // LDS, the others from global memory; `which` selects 1 = global rungs only,
    // 2 = LDS rungs only, 3 = both.
    auto load_rung = [&](int r, Slice *x, int which) {
        if (r < nlds) {
            if (which & 2) {
                const int L0 = 16 * wv + nq + kLeadQ - rt.d0[r];
                x[0] = dma_slice(kr, L0, gq);
                x[1] = dma_slice(vr, L0, gq);
                x[2] = dma_slice(kr, L0 - 1, gq);
                x[3] = dma_slice(vr, L0 - 1, gq);
            }
        } else if (which & 1) {
            // rows of the clamped query ic (a query past T is masked)
            const int R0 = max(ic - rt.d0[r], 0);
            const int R1 = max(ic - rt.d0[r] - 1, 0);
            x[0] = load_row(K, R0, gq, stk);
            x[1] = load_row(V, R0, gq, stv);
            x[2] = load_row(K, R1, gq, stk);
            x[3] = load_row(V, R1, gq, stv);
        }
    };
    Slice xA[4], xB[4];
    if (0 < nact) load_rung(0, xA, 1);  // in flight during the band phase

    // rows [T0-kLeadQ, T0+64) of K and V, straight to LDS (rows outside [0, T) are
    // clamped copies: their keys are masked below)
    dma_rows<kStage>(kr, K, T0 - kLeadQ, T, stk);
    dma_rows<kStage>(vr, V, T0 - kLeadQ, T, stv);
    __builtin_amdgcn_s_setprio(0);
    stage_freq(sfreq, rf);
    // Delta_i = <dO_i, o_i>, once every load of the prologue is in flight
    const float delta = quad_sum(dot_slice(gqq, oq));
    const float delta_m = __shfl(delta, 4 * nm, 64);
    wait_vmem();
    __syncthreads();
    if (0 < nact) load_rung(0, xA, 2);

    // band (MFMA layout): keys [t0-16, t0+16)
    uint32_t cw[4];
    float pdp = 0.f;  // this lane's part of the band's sum of p dP (Delta from the entries)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        const int sr = kLeadQ - 16 + 16 * wv + 16 * b + nm;  // staged row
        const f32x4 s = mfma_dot64(dma_slice(kr, sr, gm), qm, f32x4{0.f, 0.f, 0.f, 0.f});
        const f32x4 dp = mfma_dot64(dma_slice(vr, sr, gm), gmm, f32x4{0.f, 0.f, 0.f, 0.f});
        float c[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int key = t0 - 16 + 16 * b + 4 * gm + e;
            const bool ok = key >= 0 && key <= im && im - key <= W;
            const float p = ok ? fast_exp2(s[e] * sl2 - lse2_m) : 0.f;
            c[e] = tau * p * (dp[e] - delta_m);
            pdp = fmaf(p, dp[e], pdp);
        }
        cw[2 * b] = pack_bf16(c[0], c[1]);
        cw[2 * b + 1] = pack_bf16(c[2], c[3]);
    }
    const bf16x8 C = as_bf8(make_uint4(cw[0], cw[1], cw[2], cw[3]));
    Acc16 acc;
#pragma unroll
    for (int c = 0; c < 4; ++c)
        acc.c[c] = mfma(dma_operand_t(kr, c, nm, kLeadQ - 16 + 16 * wv, gm), C, f32x4{0.f, 0.f, 0.f, 0.f});
    acc_to_quad(acc, lane);
    // the query's band sum of p dP, on each of its four quad lanes
    float dsum = to_quad(sum4(pdp), lane);

    // rungs (quad layout), two batches in flight; r1 = -1 is the zero row.
    // dalpha is a sum with heavy cancellation (|dalpha| is a small fraction of the sum
    // of its terms' magnitudes), so its Delta is not the one from the stored o (rounded
    // to bf16) but the entries' own Delta_i = sum_e p_e dP_e, known after the loop: the
    // lane accumulates xa = sum f p dP ds, xb = sum f p dv and y = sum f p ds over its
    // parts ds of <q, k[r1]-k[r0]> and dv of <dO, v[r1]-v[r0]>, and its dalpha terms are
    // tau (xa - Delta y) + xb (float32 per lane; float64 across lanes below).
    float xa = 0.f, xb = 0.f, y = 0.f;
    auto compute_rung = [&](int r, const Slice *x) {  // x = {k0, v0, k1, v1}
        const int d0 = rt.d0[r];
        const float w = rt.w[r];
        // with every w == 0 a rung is in the set of query i iff d0 <= i
        const bool incl = r < nact && i < T && (INTERP ? (d0 < i || (d0 == i && w == 0.f)) : d0 <= i);
        const bool has1 = i - d0 - 1 >= 0;  // row r1 exists (else the zero row)
        // this lane's parts of <q, k[r]>, <dO, v[r]> (four lanes per query)
        const float s0l = dot_slice(qq, x[0]), p0l = dot_slice(gqq, x[1]);
        const float s1a = dot_slice(qq, x[2]), p1a = dot_slice(gqq, x[3]);  // row r1 (or row 0)
        const float s1l = has1 ? s1a : 0.f, p1l = has1 ? p1a : 0.f;
        float sc, dP;
        if (INTERP) {
            sc = quad_sum((1.f - w) * s0l + w * s1l);
            dP = quad_sum((1.f - w) * p0l + w * p1l);
        } else {
            sc = quad_sum(s0l);
            dP = quad_sum(p0l);
        }
        const float p = incl ? fast_exp2(sc * sl2 - lse2) : 0.f;
        const float cc = tau * p * (dP - delta);
        // (tau dS, p) of this entry for the dk/dv kernel (zeros for an excluded entry)
        if (gq == 0) sterm[r * kBwdB + 16 * wave + nq] = pack_bf16(cc, p);
        if (INTERP)
            acc_axpy2(acc, cc * (1.f - w), x[0], cc * w, x[2]);
        else
            acc_axpy_bf(acc, cc, x[0]);
        // dalpha: f (tau dS <q, k[r1] - k[r0]> + p <dO, v[r1] - v[r0]>) from this lane's
        // parts (p = 0 for an excluded entry); the wave and workgroup sums below add the
        // four lanes of each query
        const float fp = (float)rt.f[r] * p, ds = s1l - s0l;
        xa = fmaf(fp * dP, ds, xa);
        xb = fmaf(fp, p1l - p0l, xb);
        y = fmaf(fp, ds, y);
        dsum = fmaf(p, dP, dsum);
    };
#pragma unroll
    for (int rb = 0; rb < kMaxRungs; rb += 2) {
        if (rb < nact) {
            if (rb + 1 < nact) load_rung(rb + 1, xB, 3);
            compute_rung(rb, xA);
            if (rb + 1 < nact) {
                if (rb + 2 < nact) load_rung(rb + 2, xA, 3);
                compute_rung(rb + 1, xB);
            }
        }
    }

    // this wave's rung terms, four rungs of its 16 queries per store (the entries were
    // written to LDS by lanes of this wave; LDS accesses of a wave complete in order)
    __builtin_amdgcn_wave_barrier();
    for (int r0 = 0; r0 < nact; r0 += 4) {
        const int r = r0 + (lane >> 4), qi = 16 * wv + (lane & 15);
        if (r < nact && T0 + qi < T)
            terms.p[((size_t)bh * terms.planes + r) * T + T0 + qi] = sterm[r * kBwdB + 16 * wave + (lane & 15)];
    }

    if (rf.on) acc_rope_t(acc, i, sfreq + 8 * gq);  // gradient w.r.t. the unrotated q
    if (i < T) {
        store_acc(dq + head_at<STRIDED, kD>(lay.dq, bh, hd.H, T) + (size_t)i * stdq, gq, acc, bad ? NAN : 1.f);
        if (gq == 0) delta_out[(size_t)bh * T + i] = bad ? NAN : delta;
    }
    float dal_q = fmaf(tau, fmaf(-dsum, y, xa), xb);
    if (bad) dal_q = NAN;
    // workgroup dalpha partial: wave sums, then the four waves in order
    double dal = (double)dal_q;
#pragma unroll
    for (int st = 32; st >= 1; st >>= 1) dal += __shfl_xor(dal, st, 64);
    if (lane == 0) red[wave] = dal;
    __syncthreads();
    if (threadIdx.x == 0) partials[blockIdx.x] = ((red[0] + red[1]) + red[2]) + red[3];
}

// ---------------------------------------------------------------------------
// NH: query heads of a group processed side by side.  The workgroup's four waves are
// kKG = 4 / NH key groups of 16 keys times NH head slots; a group of G query heads
// takes G / NH passes (ONE_PASS: G == NH, no pass loop), and the head slots' dk, dv
// are summed through LDS at the end.
template <bool INTERP, int NH, bool ONE_PASS, bool DEV, bool STRIDED>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void bwd_dkdv_bf16_d64_kernel(
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k, const uint16_t *__restrict__ v,
    const float *__restrict__ lse, const uint16_t *__restrict__ dO, const float *__restrict__ delta_in,
    RungTerms terms, uint16_t *__restrict__ dk, uint16_t *__restrict__ dv,
    const double *__restrict__ partials, int n_partials, float *__restrict__ dalpha,
    float *__restrict__ dtheta, int T, int W,
    RungTable rt_arg,
    const RungTable *__restrict__ rtp, RopeFreq rf, float tau, int tiles, Heads hd, Layouts lay) {
    const RungTable &rt = DEV ? *rtp : rt_arg;
    constexpr int kKG = 4 / NH;          // key groups of 16 per workgroup
    constexpr int kKeys = 16 * kKG;      // keys per workgroup
    constexpr int kSt = kKeys + 16;      // staged query rows per head slot
    // the tile's own K, V rows [T0, T0 + kOwn) (the band's keys)
    constexpr int kOwn = kKeys;
    __shared__ double sfreq[32];
    // q rows of every head slot, then their dO rows
    __shared__ __align__(16) uint16_t stage[2 * NH * kSt * kD];
    __shared__ __align__(16) uint16_t kown[kOwn * kD];
    __shared__ __align__(16) uint16_t vown[kOwn * kD];
    __shared__ float sl[NH * kSt], sd[NH * kSt];

    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int kg = wv / NH, hs = wv % NH;      // key group, head slot
    const int nm = lane & 15, gm = lane >> 4;  // MFMA layout
    const int nq = lane >> 2, gq = lane & 3;   // quad layout
    const int blk = xcd_remap(blockIdx.x, gridDim.x);
    const int bk = blk / tiles;                // batch * key/value heads + key/value head
    const int T0 = (blk % tiles) * kKeys;
    const uint16_t *K = k + head_at<STRIDED, kD>(lay.k, bk, hd.kv_heads(), T);
    const uint16_t *V = v + head_at<STRIDED, kD>(lay.v, bk, hd.kv_heads(), T);
    // row strides
    const int stq = STRIDED ? (int)lay.q.st : kD, stg = STRIDED ? (int)lay.g.st : kD;
    const int stk = STRIDED ? (int)lay.k.st : kD, stv = STRIDED ? (int)lay.v.st : kD;
    const int stdk = STRIDED ? (int)lay.dk.st : kD, stdv = STRIDED ? (int)lay.dv.st : kD;
    const float sl2 = tau * kLog2e;
    uint16_t *qr = stage + hs * kSt * kD;            // this wave's head slot
    uint16_t *gr = stage + (NH + hs) * kSt * kD;

    // final dalpha: the dq kernel has completed on this stream (the reduction borrows
    // kown before its rows are loaded)
    if (blockIdx.x == 0) {
        double *red = reinterpret_cast<double *>(kown);
        double s = 0.0;
        for (int t = threadIdx.x; t < n_partials; t += 256) s += partials[t];
        red[threadIdx.x] = s;
        __syncthreads();
        for (int st = 128; st >= 1; st >>= 1) {
            if ((int)threadIdx.x < st) red[threadIdx.x] += red[threadIdx.x + st];
            __syncthreads();
        }
        if (threadIdx.x == 0) {
            const float da = (float)red[0];
            *dalpha = da;
            // a table built from theta: d L / d theta = dalpha * d alpha / d theta
            if (DEV && dtheta) *dtheta = (float)((double)da * rt.dadtheta);
        }
        __syncthreads();
    }

    const int t0 = T0 + 16 * kg;
    const int jm = t0 + nm;      // MFMA layout key
    const int j_key = t0 + nq;   // quad layout key

    // rungs: some key of this wave has j + floor(d) < T for a prefix of the table
    int nact = 0;
#pragma unroll
    for (int r = 0; r < kMaxRungs; ++r)  // a device table: unconditional tests (wide scalar loads)
        nact += (DEV ? ((r < rt.n) & (t0 + rt.d0[r] < T)) : (r < rt.n && t0 + rt.d0[r] < T)) ? 1 : 0;
    nact = __builtin_amdgcn_readfirstlane(nact);  // wave-uniform: scalar branches

    // With several passes the table is staged before the pass loop: inside it the
    // compiler hoists the table's products out of the loop and keeps them in scratch
    // memory until the first pass stores them (behind a wait for every copy in flight).
    if constexpr (!ONE_PASS) stage_freq(sfreq, rf);
    Acc16 adk, adv;
    acc_zero(adk);
    acc_zero(adv);
    const int passes = ONE_PASS ? 1 : hd.G / NH;
    for (int pass = 0; pass < passes; ++pass) {
        // an opaque copy of the key index keeps the per-rung index arithmetic inside the
        // pass loop (hoisted for all rungs at once it would not fit the registers)
        int j = j_key;
        asm volatile("" : "+v"(j));
        const int bh = hd.q_of(bk, pass * NH + hs);  // this wave's query head
        const uint16_t *Q = q + head_at<STRIDED, kD>(lay.q, bh, hd.H, T);
        const uint16_t *Gd = dO + head_at<STRIDED, kD>(lay.g, bh, hd.H, T);
        const uint32_t *E = terms.p + (size_t)bh * terms.planes * T;  // this query head's terms
        // term of rung r, query ic: a 32-bit byte offset from the uniform base (planes * T
        // entries of one head stay far below 2^30)
        auto term = [&](int r, int ic) {
            return *reinterpret_cast<const uint32_t *>(reinterpret_cast<const char *>(E) +
                                                       4u * ((uint32_t)r * (uint32_t)T + (uint32_t)ic));
        };
        // Every rung entry's (tau dS, p) comes from the dq kernel, so a rung needs only the
        // q and dO rows of the queries that read this key (the entry of a query that
        // excludes the rung is zero).  The plane index is clamped to an active rung so a
        // batch's second slot past the last active rung reads written terms (masked below).
        // Integer offsets: query j + d0 of each of two rungs per batch.
        struct Pair {
            Slice x[4];     // q, dO of rung a's query; q, dO of rung b's query
            uint32_t e[2];  // their (tau dS, p)
        };
        auto load_pair = [&](int rb, Pair &pr) {
#pragma unroll
            for (int y = 0; y < 2; ++y) {
                const int r = min(rb + y, nact - 1);
                const int ic = min(j + rt.d0[r], T - 1);
                pr.x[2 * y] = load_row(Q, ic, gq, stq);
                pr.x[2 * y + 1] = load_row(Gd, ic, gq, stg);
                pr.e[y] = term(r, ic);
            }
        };
        // Interpolated offsets: query i0 = j + floor(d) reads this key as row r0 (weight
        // 1 - w) and query i0 + 1 reads it as row r1 (weight w).
        struct Rung {
            Slice x[4];     // q, dO of query i0; q, dO of query i0 + 1
            uint32_t e[2];  // their (tau dS, p)
        };
        auto load_rung = [&](int r0, Rung &ru) {
            const int r = min(r0, nact - 1);
#pragma unroll
            for (int y = 0; y < 2; ++y) {
                const int ic = min(j + rt.d0[r] + y, T - 1);
                ru.x[2 * y] = load_row(Q, ic, gq, stq);
                ru.x[2 * y + 1] = load_row(Gd, ic, gq, stg);
                ru.e[y] = term(r, ic);
            }
        };
        Pair pA, pB;
        Rung rA, rB;
        if (0 < nact) {  // in flight during the band phase
            if (INTERP) load_rung(0, rA);
            else load_pair(0, pA);
        }
        if (pass > 0) __syncthreads();  // every wave is done with the previous pass's rows
        // q and dO rows, lse and Delta of queries [T0, T0 + kSt) of every head slot (rows
        // past the end are clamped copies, masked below)
        // (every copy is issued before the lse / Delta loads, whose LDS stores wait for
        // all of this wave's loads)
#pragma unroll 1
        for (int u = 0; u < NH; ++u) {
            const int hu = hd.q_of(bk, pass * NH + u);
            dma_rows<kSt>(stage + u * kSt * kD, q + head_at<STRIDED, kD>(lay.q, hu, hd.H, T), T0, T, stq);
            dma_rows<kSt>(stage + (NH + u) * kSt * kD, dO + head_at<STRIDED, kD>(lay.g, hu, hd.H, T), T0, T, stg);
        }
        if (pass == 0) {
            dma_rows<kOwn>(kown, K, T0, T, stk);  // rows past the end: clamped copies
            dma_rows<kOwn>(vown, V, T0, T, stv);
            if constexpr (ONE_PASS) stage_freq(sfreq, rf);
        }
#pragma unroll 1
        for (int u = 0; u < NH; ++u) {
            const size_t ou = (size_t)hd.q_of(bk, pass * NH + u) * T;
            for (int c = threadIdx.x; c < kSt; c += 256) {
                const int row = T0 + c;
                sl[u * kSt + c] = row < T ? lse[ou + row] * kLog2e : 0.f;
                sd[u * kSt + c] = row < T ? delta_in[ou + row] : 0.f;
            }
        }
        wait_vmem();
        __syncthreads();

        // band (MFMA layout): queries [t0, t0 + 32) in two blocks
        {
            const Slice km = dma_slice(kown, 16 * kg + nm, gm);
            const Slice vm = dma_slice(vown, 16 * kg + nm, gm);
            uint32_t cw[4], pw[4];
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const int sq = 16 * kg + 16 * b + nm;  // staged query row of this lane's A operand
                const f32x4 s = mfma_dot64(dma_slice(qr, sq, gm), km, f32x4{0.f, 0.f, 0.f, 0.f});
                const f32x4 dp = mfma_dot64(dma_slice(gr, sq, gm), vm, f32x4{0.f, 0.f, 0.f, 0.f});
                float c[4], p[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int si = 16 * kg + 16 * b + 4 * gm + e;  // staged index of the query
                    const int qi = T0 + si;
                    const bool ok = qi < T && jm < T && qi >= jm && qi - jm <= W;
                    p[e] = ok ? fast_exp2(s[e] * sl2 - sl[hs * kSt + si]) : 0.f;
                    c[e] = tau * p[e] * (dp[e] - sd[hs * kSt + si]);
                }
                cw[2 * b] = pack_bf16(c[0], c[1]);
                cw[2 * b + 1] = pack_bf16(c[2], c[3]);
                pw[2 * b] = pack_bf16(p[0], p[1]);
                pw[2 * b + 1] = pack_bf16(p[2], p[3]);
            }
            const bf16x8 Cb = as_bf8(make_uint4(cw[0], cw[1], cw[2], cw[3]));
            const bf16x8 Pb = as_bf8(make_uint4(pw[0], pw[1], pw[2], pw[3]));
            Acc16 bk_, bv_;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                bk_.c[c] = mfma(dma_operand_t(qr, c, nm, 16 * kg, gm), Cb, f32x4{0.f, 0.f, 0.f, 0.f});
                bv_.c[c] = mfma(dma_operand_t(gr, c, nm, 16 * kg, gm), Pb, f32x4{0.f, 0.f, 0.f, 0.f});
            }
            acc_to_quad(bk_, lane);
            acc_to_quad(bv_, lane);
            if (ONE_PASS || pass == 0) {  // the accumulators are still zero: no adds
                adk = bk_;
                adv = bv_;
            } else {
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    adk.c[c] += bk_.c[c];
                    adv.c[c] += bv_.c[c];
                }
            }
        }

        if (!INTERP) {
            auto compute_pair = [&](int rb, const Pair &pr) {
                uint32_t e[2];
#pragma unroll
                for (int y = 0; y < 2; ++y) {
                    const bool in = rb + y < nact && j < T && j + rt.d0[rb + y] < T;
                    e[y] = in ? pr.e[y] : 0u;
                }
                // (tau dS_a, tau dS_b) and (p_a, p_b) as bfloat16 pairs
                acc_axpy2_bf(adk, __builtin_amdgcn_perm(e[1], e[0], 0x05040100u), pr.x[0], pr.x[2]);
                acc_axpy2_bf(adv, __builtin_amdgcn_perm(e[1], e[0], 0x07060302u), pr.x[1], pr.x[3]);
            };
            // two batches in flight: load the next while accumulating the current (one in
            // the instances that loop over head passes, whose registers hold more state)
            if constexpr (ONE_PASS) {
#pragma unroll
                for (int rb = 0; rb < kMaxRungs; rb += 4) {
                    if (rb < nact) {
                        if (rb + 2 < nact) load_pair(rb + 2, pB);
                        compute_pair(rb, pA);
                        if (rb + 2 < nact) {
                            if (rb + 4 < nact) load_pair(rb + 4, pA);
                            compute_pair(rb + 2, pB);
                        }
                    }
                }
            } else {
#pragma unroll
                for (int rb = 0; rb < kMaxRungs; rb += 2) {
                    if (rb < nact) {
                        if (rb > 0) load_pair(rb, pA);
                        compute_pair(rb, pA);
                    }
                }
            }
        } else {
            auto compute_rung = [&](int r, const Rung &ru) {
                const float w = rt.w[r];
                const int i0 = j + rt.d0[r];
                const bool in0 = r < nact && j < T && i0 < T;
                const bool in1 = r < nact && j < T && i0 + 1 < T && w != 0.f;
                const uint32_t ea = in0 ? ru.e[0] : 0u, eb = in1 ? ru.e[1] : 0u;
                const float ca = (1.f - w) * bf16_lo(ea), pa = (1.f - w) * bf16_hi(ea);
                const float cb = w * bf16_lo(eb), pb = w * bf16_hi(eb);
                acc_axpy2(adk, ca, ru.x[0], cb, ru.x[2]);
                acc_axpy2(adv, pa, ru.x[1], pb, ru.x[3]);
            };
            if constexpr (ONE_PASS) {
#pragma unroll
                for (int r = 0; r < kMaxRungs; r += 2) {
                    if (r < nact) {
                        if (r + 1 < nact) load_rung(r + 1, rB);
                        compute_rung(r, rA);
                        if (r + 1 < nact) {
                            if (r + 2 < nact) load_rung(r + 2, rA);
                            compute_rung(r + 1, rB);
                        }
                    }
                }
            } else {
#pragma unroll
                for (int r = 0; r < kMaxRungs; ++r) {
                    if (r < nact) {
                        if (r > 0) load_rung(r, rA);
                        compute_rung(r, rA);
                    }
                }
            }
        }
    }

    if constexpr (NH > 1) {
        // sum the head slots: slots 1.. hand their accumulators (quad layout, 32 floats
        // per lane) to slot 0 of the same key group through the staging LDS, as eight
        // 16-byte vectors per lane stored lane-minor (vector v of lane l at v * 64 + l),
        // so a wave's 16-byte accesses cover consecutive banks (lane-major 128-byte
        // blocks put every lane of an access on one bank: 6x the conflict cycles)
        static_assert(sizeof(stage) >= (size_t)(4 - kKG) * 64 * 32 * sizeof(float), "LDS for the sum");
        f32x4 *xfer = reinterpret_cast<f32x4 *>(stage);
        __syncthreads();  // every wave is done with the staged rows
        if (hs > 0) {
            f32x4 *dst = xfer + (size_t)(kg * (NH - 1) + hs - 1) * 8 * 64 + lane;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                dst[c * 64] = adk.c[c];
                dst[(4 + c) * 64] = adv.c[c];
            }
        }
        __syncthreads();
        if (hs == 0) {
#pragma unroll 1
            for (int u = 1; u < NH; ++u) {
                const f32x4 *src = xfer + (size_t)(kg * (NH - 1) + u - 1) * 8 * 64 + lane;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    adk.c[c] += src[c * 64];
                    adv.c[c] += src[(4 + c) * 64];
                }
            }
        }
    }

    if (hs == 0) {
        if (rf.on) acc_rope_t(adk, j_key, sfreq + 8 * gq);  // gradient w.r.t. the unrotated k
        if (j_key < T) {
            const float sc = DEV && table_unusable(rt, W) ? NAN : 1.f;  // bad device alpha, or another W
            store_acc(dk + head_at<STRIDED, kD>(lay.dk, bk, hd.kv_heads(), T) + (size_t)j_key * stdk, gq, adk, sc);
            store_acc(dv + head_at<STRIDED, kD>(lay.dv, bk, hd.kv_heads(), T) + (size_t)j_key * stdv, gq, adv, sc);
        }
    }
}

bool backward_mfma_supported(int dtype, int D, int W) { return dtype == 1 && D == 64 && W <= 16; }

// (with HS heads per workgroup the dq grid has ceil(T / (64 / HS)) * BH / HS <= this many)
size_t bwd_mfma_num_partials(int BH, int T) { return (size_t)((T + kBwdB - 1) / kBwdB) * (size_t)BH; }

template <int NH>
static hipError_t launch_dkdv(bool interp, const void *q, const void *k, const void *v,
                              const float *lse, const void *dO, const float *delta_ws,
                              const RungTerms &terms, void *dk, void *dv, const double *partials,
                              int n_partials, float *dalpha, float *dtheta,
                              int BH, const Heads &hd, int T, int W, const RungTable &rt,
                              const RungTable *rtp, const RopeFreq &rf, float tau,
                              const Layouts &lay, hipStream_t s) {
    constexpr int keys = 64 / NH;
    const int tiles = (T + keys - 1) / keys;
    const bool one = hd.G == NH;
    const int hk = hd.kv_heads();
    const bool strided = !is_packed(lay.q, hd.H, T, kD) || !is_packed(lay.k, hk, T, kD) ||
                         !is_packed(lay.v, hk, T, kD) || !is_packed(lay.g, hd.H, T, kD) ||
                         !is_packed(lay.dk, hk, T, kD) || !is_packed(lay.dv, hk, T, kD);
    if (rtp && strided) return hipErrorInvalidValue;  // device tables come with packed tensors
#define FIBATTN_DKDV(I, S)                                                                     \
    (one ? bwd_dkdv_bf16_d64_kernel<I, NH, true, false, S> : bwd_dkdv_bf16_d64_kernel<I, NH, false, false, S>)
    auto kern = rtp ? (one ? bwd_dkdv_bf16_d64_kernel<true, NH, true, true, false>
                           : bwd_dkdv_bf16_d64_kernel<true, NH, false, true, false>)
              : strided ? (interp ? FIBATTN_DKDV(true, true) : FIBATTN_DKDV(false, true))
                        : (interp ? FIBATTN_DKDV(true, false) : FIBATTN_DKDV(false, false));
#undef FIBATTN_DKDV
    return launch(kBwdDkDv, kern, dim3(tiles * (BH / hd.G)), dim3(256), 0, s, q, k, v, lse, dO,
                  delta_ws, terms, dk, dv, partials, n_partials, dalpha, dtheta, T, W, rt, rtp, rf, tau,
                  tiles, hd, lay);
}

hipError_t launch_backward_mfma(const void *q, const void *k, const void *v, const void *o,
                                const float *lse, const void *dO, void *dq, void *dk, void *dv,
                                float *dalpha, float *dtheta, float *delta_ws, double *partials,
                                const RungTerms &terms, int BH, const Heads &hd, int T, int W,
                                const RungTable &rt, const RungTable *rtp, const RopeFreq &rf,
                                const Layouts &lay, hipStream_t s) {
    const float tau = 1.f / sqrtf(64.f);
    bool interp = rtp != nullptr;  // a device table may hold any weights
    for (int r = 0; r < rt.n && !interp; ++r) interp = rt.w[r] != 0.f;
    const int hk = hd.kv_heads();
    const bool strided = !is_packed(lay.q, hd.H, T, kD) || !is_packed(lay.k, hk, T, kD) ||
                         !is_packed(lay.v, hk, T, kD) || !is_packed(lay.o, hd.H, T, kD) ||
                         !is_packed(lay.g, hd.H, T, kD) || !is_packed(lay.dq, hd.H, T, kD);
    if (rtp && strided) return hipErrorInvalidValue;  // device tables come with packed tensors
    // query heads per dq workgroup: the group's heads side by side for packed tensors with
    // a host table (as the forward)
    const int hs = (rtp || strided) ? 1 : hd.G % 4 == 0 ? 4 : hd.G % 2 == 0 ? 2 : 1;
    const int tiles = (T + kBwdB / hs - 1) / (kBwdB / hs);  // runs of 64 / hs queries
    const int nb = tiles * (BH / hs);                          // dq workgroups = dalpha partials
    auto dqk = rtp ? bwd_dq_bf16_d64_kernel<true, true, false, 1>
             : strided ? (interp ? bwd_dq_bf16_d64_kernel<true, false, true, 1> : bwd_dq_bf16_d64_kernel<false, false, true, 1>)
             : hs == 4 ? (interp ? bwd_dq_bf16_d64_kernel<true, false, false, 4> : bwd_dq_bf16_d64_kernel<false, false, false, 4>)
             : hs == 2 ? (interp ? bwd_dq_bf16_d64_kernel<true, false, false, 2> : bwd_dq_bf16_d64_kernel<false, false, false, 2>)
                       : (interp ? bwd_dq_bf16_d64_kernel<true, false, false, 1> : bwd_dq_bf16_d64_kernel<false, false, false, 1>);
    hipError_t e = launch(kBwdDq, dqk, dim3(nb), dim3(256), 0, s, q, k, v, o, lse, dO, dq, delta_ws,
                          partials, terms, T, W, rt, rtp, rf, tau, tiles, hd, lay);
    if (e != hipSuccess) return e;
    // query heads per key/value head processed side by side in a workgroup
    if (hd.G % 4 == 0)
        return launch_dkdv<4>(interp, q, k, v, lse, dO, delta_ws, terms, dk, dv, partials, nb, dalpha, dtheta, BH,
                              hd, T, W, rt, rtp, rf, tau, lay, s);
    if (hd.G % 2 == 0)
        return launch_dkdv<2>(interp, q, k, v, lse, dO, delta_ws, terms, dk, dv, partials, nb, dalpha, dtheta, BH,
                              hd, T, W, rt, rtp, rf, tau, lay, s);
    return launch_dkdv<1>(interp, q, k, v, lse, dO, delta_ws, terms, dk, dv, partials, nb, dalpha, dtheta, BH, hd,
                          T, W, rt, rtp, rf, tau, lay, s);
}

}  // namespace fibattn
