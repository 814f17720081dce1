// C ABI of libfibattn.so: argument validation, the host rung table, workspace
// layout and kernel timing.  The declarations and their contracts are in
// include/fibattn.h.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <vector>

#include "../../include/fibattn.h"
#include "launch.h"

using namespace fibattn;

namespace {

// The base table's own rules (Section 2): K <= FIBATTN_MAX_RUNGS, entries >= 1 and
// strictly increasing.
fibattn_status_t check_base(const int32_t *base, int K, BaseTable *b) {
    if (K < 0 || K > FIBATTN_MAX_RUNGS || (K > 0 && base == nullptr)) return FIBATTN_ERR_INVALID_ARG;
    b->K = K;
    for (int a = 0; a < kMaxRungs; ++a) b->f[a] = 0;
    for (int a = 0; a < K; ++a) {
        if (base[a] < 1) return FIBATTN_ERR_INVALID_ARG;
        if (a > 0 && base[a] <= base[a - 1]) return FIBATTN_ERR_INVALID_ARG;
        b->f[a] = base[a];
    }
    return FIBATTN_OK;
}

fibattn_status_t build_table(float alpha, const int32_t *base, int K, int W, RungTable *rt) {
    BaseTable b;
    fibattn_status_t st = check_base(base, K, &b);
    if (st != FIBATTN_OK) return st;
    return rung_table_fill(alpha, b, W, rt) ? FIBATTN_OK : FIBATTN_ERR_INVALID_ARG;
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

fibattn_status_t check_common(int B, int H, int T, int d_head, int W, int K, fibattn_dtype_t dtype) {
    if (B < 1 || H < 1 || T < 1 || W < 0 || K < 0) return FIBATTN_ERR_INVALID_ARG;
    if (dtype != FIBATTN_FP32 && dtype != FIBATTN_BF16) return FIBATTN_ERR_INVALID_ARG;
    if ((long long)B * H > 65535) return FIBATTN_ERR_UNSUPPORTED;
    if ((long long)B * H * T * d_head > (1ll << 40)) return FIBATTN_ERR_UNSUPPORTED;
    // one packed head's rows below 2^31 bytes: the kernels address rows (and the
    // backward's per-rung terms, 4 bytes per query and rung) with 32-bit offsets from
    // the head's first row
    const long long es = dtype == FIBATTN_BF16 ? 2 : 4;
    if ((long long)T * d_head * es >= (1ll << 31)) return FIBATTN_ERR_UNSUPPORTED;
    if (d_head != 32 && d_head != 64 && d_head != 128) return FIBATTN_ERR_UNSUPPORTED;
    if (W > FIBATTN_MAX_WINDOW || K > FIBATTN_MAX_RUNGS) return FIBATTN_ERR_UNSUPPORTED;
    return FIBATTN_OK;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Every tensor packed [B, heads, T, d].
Layouts packed_layouts(int H, int H_kv, int T, int D) {
    const Layout lq = Layout::packed(H, T, D), lk = Layout::packed(H_kv, T, D);
    return {lq, lk, lk, lq, lq, lq, lk, lk};
}

// A caller's placement of one tensor: non-negative strides that keep every row 16-byte
// aligned, and row offsets within a head below 2^31 bytes (the kernels address rows
// with 32-bit offsets from the head's first row).
fibattn_status_t check_layout(const fibattn_layout_t &l, int T, int d_head, fibattn_dtype_t dtype,
                              Layout *out) {
    const long long es = dtype == FIBATTN_BF16 ? 2 : 4;
    if (l.batch < 0 || l.head < 0 || l.pos < 0) return FIBATTN_ERR_INVALID_ARG;
    if ((l.batch * es) % 16 || (l.head * es) % 16 || (l.pos * es) % 16) return FIBATTN_ERR_INVALID_ARG;
    if (((long long)(T - 1) * l.pos + d_head) * es >= (1ll << 31)) return FIBATTN_ERR_UNSUPPORTED;
    *out = {l.batch, l.head, l.pos};
    return FIBATTN_OK;
}

// ---- kernel timing -------------------------------------------------------
// Per host thread: only launches made by the thread that began timing are timed, so
// calls from other threads never touch this state.
struct Timing {
    int id = -1;
    int capacity = 0;
    std::vector<hipEvent_t> ev;  // start/stop pairs
    int used = 0;
};
thread_local Timing g_timing;

// ---- static scratch of the allocation-free backward -------------------------
// One copy per GPU, created with the library's code object on that device.  Host code
// never uses this name as an address (on the host it is only a stand-in): kernels and
// copies get the device address resolved by scratch_on().
static __device__ __align__(256) unsigned char scratch[FIBATTN_SCRATCH_BYTES];

std::mutex g_scratch_mu;
std::vector<void *> g_scratch;  // per device ordinal; nullptr until resolved

// Device address of `dev`'s copy of the scratch array, looked up once per device with
// that device current (the caller's current device is restored).  nullptr on failure.
void *scratch_on(int dev) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (dev < 0) return nullptr;
    if ((size_t)dev < g_scratch.size() && g_scratch[dev]) return g_scratch[dev];
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return nullptr;
    if (cur != dev && hipSetDevice(dev) != hipSuccess) return nullptr;
    void *ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess || !ptr) {
        (void)hipGetLastError();  // leave no sticky error for the caller's next call
        return nullptr;
    }
    if ((size_t)dev >= g_scratch.size()) g_scratch.resize((size_t)dev + 1, nullptr);
    g_scratch[dev] = ptr;
    return ptr;
}

}  // namespace

namespace fibattn {

bool timing_events(int id, hipEvent_t *start, hipEvent_t *stop) {
    if (id != g_timing.id || g_timing.used >= g_timing.capacity) return false;
    *start = g_timing.ev[2 * g_timing.used];
    *stop = g_timing.ev[2 * g_timing.used + 1];
    ++g_timing.used;
    return true;
}

}  // namespace fibattn

extern "C" {

fibattn_status_t fibattn_rung_table(float alpha, const int32_t *base, int K, int W, int32_t *d0,
                                    float *w, int32_t *f, int *n) {
    if (!d0 || !w || !f || !n || W < 0) return FIBATTN_ERR_INVALID_ARG;
    RungTable rt;
    fibattn_status_t st = build_table(alpha, base, K, W, &rt);
    if (st != FIBATTN_OK) return st;
    for (int a = 0; a < rt.n; ++a) { d0[a] = rt.d0[a]; w[a] = rt.w[a]; f[a] = rt.f[a]; }
    *n = rt.n;
    return FIBATTN_OK;
}

static fibattn_status_t forward_impl(const void *q, const void *k, const void *v, void *o, float *lse,
                                     const Layouts &lay, int B, int H, int H_kv, int T, int d_head,
                                     int W, const int32_t *base, int K, float alpha,
                                     fibattn_dtype_t dtype, hipStream_t stream) {
    fibattn_status_t st = check_common(B, H, T, d_head, W, K, dtype);
    if (st != FIBATTN_OK) return st;
    if (H_kv < 1 || H_kv > H || H % H_kv != 0) return FIBATTN_ERR_INVALID_ARG;
    if (!q || !k || !v || !o || !lse) return FIBATTN_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(lse))
        return FIBATTN_ERR_INVALID_ARG;
    RungTable rt;
    st = build_table(alpha, base, K, W, &rt);
    if (st != FIBATTN_OK) return st;
    const Heads hd{H, H / H_kv};
    hipError_t e = launch_forward((int)dtype, d_head, q, k, v, o, lse, B * H, hd, T, W, rt, nullptr,
                                  lay, stream);
    return e == hipSuccess ? FIBATTN_OK : FIBATTN_ERR_HIP;
}

fibattn_status_t fibattn_forward_gqa(const void *q, const void *k, const void *v, void *o,
                                     float *lse, int B, int H, int H_kv, int T, int d_head, int W,
                                     const int32_t *base, int K, float alpha, fibattn_dtype_t dtype,
                                     hipStream_t stream) {
    if (H_kv < 1 || H_kv > H || H % H_kv != 0) return FIBATTN_ERR_INVALID_ARG;
    return forward_impl(q, k, v, o, lse, packed_layouts(H, H_kv, T, d_head), B, H, H_kv, T, d_head, W,
                        base, K, alpha, dtype, stream);
}

fibattn_status_t fibattn_forward_strided(const void *q, const void *k, const void *v, void *o,
                                         float *lse, const fibattn_layout_t *layouts, int B, int H,
                                         int H_kv, int T, int d_head, int W, const int32_t *base,
                                         int K, float alpha, fibattn_dtype_t dtype,
                                         hipStream_t stream) {
    if (!layouts || T < 1) return FIBATTN_ERR_INVALID_ARG;
    Layouts lay = packed_layouts(H, H_kv > 0 ? H_kv : 1, T, d_head);
    Layout *dst[4] = {&lay.q, &lay.k, &lay.v, &lay.o};
    for (int a = 0; a < 4; ++a) {
        const fibattn_status_t st = check_layout(layouts[a], T, d_head, dtype, dst[a]);
        if (st != FIBATTN_OK) return st;
    }
    return forward_impl(q, k, v, o, lse, lay, B, H, H_kv, T, d_head, W, base, K, alpha, dtype, stream);
}

fibattn_status_t fibattn_forward(const void *q, const void *k, const void *v, void *o, float *lse,
                                 int B, int H, int T, int d_head, int W, const int32_t *base,
                                 int K, float alpha, fibattn_dtype_t dtype, hipStream_t stream) {
    return fibattn_forward_gqa(q, k, v, o, lse, B, H, H, T, d_head, W, base, K, alpha, dtype, stream);
}

// The forward with q rotated on load, from a host table (rtp null) or a device table;
// lay.dq places q_out.
static fibattn_status_t forward_rope_q_impl(const void *q, const void *k, const void *v, void *o, float *lse,
                                            void *q_out, int B, int H, int H_kv, int T, int d_head, int W,
                                            const RungTable &rt, const RungTable *rtp, float rope_base,
                                            const Layouts &lay, fibattn_dtype_t dtype, hipStream_t stream) {
    if (H_kv < 1 || H_kv > H || H % H_kv != 0) return FIBATTN_ERR_INVALID_ARG;
    if (!q || !k || !v || !o || !lse) return FIBATTN_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(lse) ||
        !aligned16(q_out) || !aligned16(rtp))
        return FIBATTN_ERR_INVALID_ARG;
    if (!(rope_base > 1.f) || !isfinite(rope_base)) return FIBATTN_ERR_INVALID_ARG;
    const bool on_load = forward_mfma_supported((int)dtype, d_head, W);
    if (!on_load && !q_out) return FIBATTN_ERR_UNSUPPORTED;  // the rotated rows need a home
    const Heads hd{H, H / H_kv};
    hipError_t e;
    if (on_load) {
        // one launch: each query row is rotated where the forward loads it
        const RopeFreq rf = make_rope_freq((double)rope_base, d_head);
        e = launch_forward_mfma(q, k, v, o, lse, B * H, hd, T, W, rt, rtp, lay, stream, &rf, q_out);
    } else {
        // the RoPE launch on q into q_out, then the forward on it
        if ((long long)B * H > 65535ll * 16) return FIBATTN_ERR_UNSUPPORTED;
        e = launch_rope((int)dtype, d_head, q, q_out, lay.q, lay.dq, nullptr, nullptr, lay.q, lay.dq, B * H, H,
                        T, rope_base, 0, stream);
        Layouts lr = lay;
        lr.q = lay.dq;
        if (e == hipSuccess)
            e = launch_forward((int)dtype, d_head, q_out, k, v, o, lse, B * H, hd, T, W, rt, rtp, lr, stream);
    }
    return e == hipSuccess ? FIBATTN_OK : FIBATTN_ERR_HIP;
}

fibattn_status_t fibattn_forward_rope_q(const void *q, const void *k, const void *v, void *o,
                                        float *lse, void *q_out, int B, int H, int H_kv, int T,
                                        int d_head, int W, const int32_t *base, int K, float alpha,
                                        float rope_base, fibattn_dtype_t dtype, hipStream_t stream) {
    fibattn_status_t st = check_common(B, H, T, d_head, W, K, dtype);
    if (st != FIBATTN_OK) return st;
    if (H_kv < 1 || H_kv > H || H % H_kv != 0) return FIBATTN_ERR_INVALID_ARG;
    RungTable rt;
    st = build_table(alpha, base, K, W, &rt);
    if (st != FIBATTN_OK) return st;
    return forward_rope_q_impl(q, k, v, o, lse, q_out, B, H, H_kv, T, d_head, W, rt, nullptr, rope_base,
                               packed_layouts(H, H_kv, T, d_head), dtype, stream);
}

fibattn_status_t fibattn_forward_rope_q_strided(const void *q, const void *k, const void *v, void *o,
                                                float *lse, void *q_out, const fibattn_layout_t *layouts,
                                                int B, int H, int H_kv, int T, int d_head, int W,
                                                const int32_t *base, int K, float alpha, float rope_base,
                                                fibattn_dtype_t dtype, hipStream_t stream) {
    if (!layouts || T < 1) return FIBATTN_ERR_INVALID_ARG;
    fibattn_status_t st = check_common(B, H, T, d_head, W, K, dtype);
    if (st != FIBATTN_OK) return st;
    if (H_kv < 1 || H_kv > H || H % H_kv != 0) return FIBATTN_ERR_INVALID_ARG;
    Layouts lay = packed_layouts(H, H_kv, T, d_head);
    Layout *dst[5] = {&lay.q, &lay.k, &lay.v, &lay.o, &lay.dq};  // q_out is placed by the dq slot
    for (int a = 0; a < (q_out ? 5 : 4); ++a) {
        st = check_layout(layouts[a], T, d_head, dtype, dst[a]);
        if (st != FIBATTN_OK) return st;
    }
    RungTable rt;
    st = build_table(alpha, base, K, W, &rt);
    if (st != FIBATTN_OK) return st;
    return forward_rope_q_impl(q, k, v, o, lse, q_out, B, H, H_kv, T, d_head, W, rt, nullptr, rope_base, lay,
                               dtype, stream);
}

// Backward workspace: Delta (float32 [B,H,T]), then the per-workgroup dalpha partials
// (float64; sized for the larger of the two dtypes' partial counts), then, for shapes
// the matrix-core path may take (d_head 64, W <= 16), its per-(query, rung) terms:
// one bfloat16 pair per query and plane, K planes (kMaxRungs for a device-resident table,
// whose rung count the host does not know, passed as K = 0).
struct WorkspaceLayout {
    size_t partials, terms, total;
    int planes;
};

static WorkspaceLayout workspace_layout(int B, int H, int T, int d_head, int W, int K) {
    size_t np = bwd_num_partials(0, d_head, B * H, T);
    size_t np1 = bwd_num_partials(1, d_head, B * H, T);
    size_t np2 = bwd_mfma_num_partials(B * H, T);
    if (np1 > np) np = np1;
    if (np2 > np) np = np2;
    WorkspaceLayout l;
    l.partials = align256(sizeof(float) * (size_t)B * H * T);
    l.terms = l.partials + align256(sizeof(double) * np);
    l.planes = backward_mfma_supported(1, d_head, W) ? (K > 0 ? K : kMaxRungs) : 0;
    l.total = l.terms + align256(sizeof(uint32_t) * (size_t)l.planes * B * H * T);
    return l;
}

size_t fibattn_backward_workspace_bytes(int B, int H, int T, int d_head, int W, int K) {
    // the workspace does not depend on the storage type: checked here under the looser
    // (bfloat16) size limits, the call itself then checks those of its own type
    if (check_common(B, H, T, d_head, W, K, FIBATTN_BF16) != FIBATTN_OK) return 0;
    return workspace_layout(B, H, T, d_head, W, K).total;
}

static fibattn_status_t backward_impl(const void *q, const void *k, const void *v, const void *o,
                                      const float *lse, const void *dO, void *dq, void *dk,
                                      void *dv, float *dalpha, void *workspace,
                                      size_t workspace_bytes, const Layouts &lay, int B, int H,
                                      int H_kv, int T, int d_head, int W, const int32_t *base,
                                      int K, float alpha, float rope_base, fibattn_dtype_t dtype,
                                      hipStream_t stream) {
    fibattn_status_t st = check_common(B, H, T, d_head, W, K, dtype);
    if (st != FIBATTN_OK) return st;
    if (H_kv < 1 || H_kv > H || H % H_kv != 0) return FIBATTN_ERR_INVALID_ARG;
    if (!q || !k || !v || !o || !lse || !dO || !dq || !dk || !dv || !dalpha)
        return FIBATTN_ERR_INVALID_ARG;
    const void *ptrs[] = {q, k, v, o, lse, dO, dq, dk, dv};
    for (const void *p : ptrs)
        if (!aligned16(p)) return FIBATTN_ERR_INVALID_ARG;
    if (!(rope_base == 0.f || (rope_base > 1.f && isfinite(rope_base)))) return FIBATTN_ERR_INVALID_ARG;
    const WorkspaceLayout wl = workspace_layout(B, H, T, d_head, W, K);
    if (!workspace || !aligned16(workspace) || workspace_bytes < wl.total) return FIBATTN_ERR_WORKSPACE;
    RungTable rt;
    st = build_table(alpha, base, K, W, &rt);
    if (st != FIBATTN_OK) return st;
    float *delta_ws = (float *)workspace;
    double *partials = (double *)((char *)workspace + wl.partials);
    const RungTerms terms{(uint32_t *)((char *)workspace + wl.terms), wl.planes};
    const RopeFreq rf = make_rope_freq((double)rope_base, d_head);
    const Heads hd{H, H / H_kv};
    hipError_t e = launch_backward((int)dtype, d_head, q, k, v, o, lse, dO, dq, dk, dv, dalpha, nullptr,
                                   delta_ws, partials, terms, B * H, hd, T, W, rt, nullptr, rf,
                                   rope_base, lay, stream);
    return e == hipSuccess ? FIBATTN_OK : FIBATTN_ERR_HIP;
}

fibattn_status_t fibattn_backward_gqa(const void *q, const void *k, const void *v, const void *o,
                                      const float *lse, const void *dO, void *dq, void *dk,
                                      void *dv, float *dalpha, void *workspace,
                                      size_t workspace_bytes, int B, int H, int H_kv, int T,
                                      int d_head, int W, const int32_t *base, int K, float alpha,
                                      float rope_base, fibattn_dtype_t dtype, hipStream_t stream) {
    if (H_kv < 1 || H_kv > H || H % H_kv != 0) return FIBATTN_ERR_INVALID_ARG;
    return backward_impl(q, k, v, o, lse, dO, dq, dk, dv, dalpha, workspace, workspace_bytes,
                         packed_layouts(H, H_kv, T, d_head), B, H, H_kv, T, d_head, W, base, K, alpha,
                         rope_base, dtype, stream);
}

fibattn_status_t fibattn_backward_strided(const void *q, const void *k, const void *v, const void *o,
                                          const float *lse, const void *dO, void *dq, void *dk,
                                          void *dv, float *dalpha, void *workspace,
                                          size_t workspace_bytes, const fibattn_layout_t *layouts,
                                          int B, int H, int H_kv, int T, int d_head, int W,
                                          const int32_t *base, int K, float alpha, float rope_base,
                                          fibattn_dtype_t dtype, hipStream_t stream) {
    if (!layouts || T < 1) return FIBATTN_ERR_INVALID_ARG;
    Layouts lay = packed_layouts(H, H_kv > 0 ? H_kv : 1, T, d_head);
    Layout *dst[8] = {&lay.q, &lay.k, &lay.v, &lay.o, &lay.g, &lay.dq, &lay.dk, &lay.dv};
    for (int a = 0; a < 8; ++a) {
        const fibattn_status_t st = check_layout(layouts[a], T, d_head, dtype, dst[a]);
        if (st != FIBATTN_OK) return st;
    }
    return backward_impl(q, k, v, o, lse, dO, dq, dk, dv, dalpha, workspace, workspace_bytes, lay, B, H,
                         H_kv, T, d_head, W, base, K, alpha, rope_base, dtype, stream);
}

fibattn_status_t fibattn_backward(const void *q, const void *k, const void *v, const void *o,
                                  const float *lse, const void *dO, void *dq, void *dk, void *dv,
                                  float *dalpha, void *workspace, size_t workspace_bytes, int B,
                                  int H, int T, int d_head, int W, const int32_t *base, int K,
                                  float alpha, float rope_base, fibattn_dtype_t dtype,
                                  hipStream_t stream) {
    return fibattn_backward_gqa(q, k, v, o, lse, dO, dq, dk, dv, dalpha, workspace, workspace_bytes,
                                B, H, H, T, d_head, W, base, K, alpha, rope_base, dtype, stream);
}

fibattn_status_t fibattn_backward_noalloc(const void *q, const void *k, const void *v,
                                          const void *o, const float *lse, const void *dO,
                                          void *dq, void *dk, void *dv, float *dalpha, int B, int H,
                                          int H_kv, int T, int d_head, int W, const int32_t *base,
                                          int K, float alpha, float rope_base, fibattn_dtype_t dtype,
                                          hipStream_t stream) {
    // the size checks come first, so a problem too large for the scratch enqueues nothing
    fibattn_status_t st = check_common(B, H, T, d_head, W, K, dtype);
    if (st != FIBATTN_OK) return st;
    if (H_kv < 1 || H_kv > H || H % H_kv != 0) return FIBATTN_ERR_INVALID_ARG;
    const size_t need = workspace_layout(B, H, T, d_head, W, K).total;
    if (need > FIBATTN_SCRATCH_BYTES) return FIBATTN_ERR_SCRATCH;
    int dev = -1;
    if (stream ? hipStreamGetDevice(stream, &dev) != hipSuccess : hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return FIBATTN_ERR_HIP;
    }
    void *ws = scratch_on(dev);
    if (!ws) return FIBATTN_ERR_HIP;
    return backward_impl(q, k, v, o, lse, dO, dq, dk, dv, dalpha, ws, FIBATTN_SCRATCH_BYTES,
                         packed_layouts(H, H_kv, T, d_head), B, H, H_kv, T, d_head, W, base, K, alpha,
                         rope_base, dtype, stream);
}

// ---- device-resident alpha -------------------------------------------------------

size_t fibattn_device_table_bytes(void) { return align256(sizeof(RungTable)); }

fibattn_status_t fibattn_device_table(const float *alpha, const int32_t *base, int K, int W,
                                      void *table, hipStream_t stream) {
    if (!alpha || !table || !aligned16(table) || W < 0 || W > FIBATTN_MAX_WINDOW)
        return FIBATTN_ERR_INVALID_ARG;
    BaseTable b;
    fibattn_status_t st = check_base(base, K, &b);
    if (st != FIBATTN_OK) return st;
    hipError_t e = launch_rung_table(alpha, b, W, (RungTable *)table, stream);
    return e == hipSuccess ? FIBATTN_OK : FIBATTN_ERR_HIP;
}

fibattn_status_t fibattn_device_table_theta(const float *theta, float *alpha, const int32_t *base, int K,
                                            int W, void *table, hipStream_t stream) {
    if (!theta || !table || !aligned16(table) || W < 0 || W > FIBATTN_MAX_WINDOW)
        return FIBATTN_ERR_INVALID_ARG;
    BaseTable b;
    fibattn_status_t st = check_base(base, K, &b);
    if (st != FIBATTN_OK) return st;
    hipError_t e = launch_rung_table_theta(theta, alpha, b, W, (RungTable *)table, stream);
    return e == hipSuccess ? FIBATTN_OK : FIBATTN_ERR_HIP;
}

fibattn_status_t fibattn_forward_dt(const void *q, const void *k, const void *v, void *o, float *lse,
                                    int B, int H, int H_kv, int T, int d_head, int W,
                                    const void *table, fibattn_dtype_t dtype, hipStream_t stream) {
    fibattn_status_t st = check_common(B, H, T, d_head, W, 0, dtype);
    if (st != FIBATTN_OK) return st;
    if (H_kv < 1 || H_kv > H || H % H_kv != 0) return FIBATTN_ERR_INVALID_ARG;
    if (!q || !k || !v || !o || !lse || !table) return FIBATTN_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(lse) ||
        !aligned16(table))
        return FIBATTN_ERR_INVALID_ARG;
    RungTable unused;
    memset(&unused, 0, sizeof(unused));
    const Heads hd{H, H / H_kv};
    hipError_t e = launch_forward((int)dtype, d_head, q, k, v, o, lse, B * H, hd, T, W, unused,
                                  (const RungTable *)table, packed_layouts(H, H_kv, T, d_head), stream);
    return e == hipSuccess ? FIBATTN_OK : FIBATTN_ERR_HIP;
}

fibattn_status_t fibattn_forward_rope_q_dt(const void *q, const void *k, const void *v, void *o,
                                           float *lse, void *q_out, int B, int H, int H_kv, int T,
                                           int d_head, int W, const void *table, float rope_base,
                                           fibattn_dtype_t dtype, hipStream_t stream) {
    fibattn_status_t st = check_common(B, H, T, d_head, W, 0, dtype);
    if (st != FIBATTN_OK) return st;
    if (!table) return FIBATTN_ERR_INVALID_ARG;
    RungTable unused;
    memset(&unused, 0, sizeof(unused));
    return forward_rope_q_impl(q, k, v, o, lse, q_out, B, H, H_kv, T, d_head, W, unused,
                               (const RungTable *)table, rope_base, packed_layouts(H, H_kv, T, d_head), dtype,
                               stream);
}

fibattn_status_t fibattn_backward_dt(const void *q, const void *k, const void *v, const void *o,
                                     const float *lse, const void *dO, void *dq, void *dk, void *dv,
                                     float *dalpha, float *dtheta, void *workspace, size_t workspace_bytes, int B,
                                     int H, int H_kv, int T, int d_head, int W, const void *table,
                                     float rope_base, fibattn_dtype_t dtype, hipStream_t stream) {
    fibattn_status_t st = check_common(B, H, T, d_head, W, 0, dtype);
    if (st != FIBATTN_OK) return st;
    if (H_kv < 1 || H_kv > H || H % H_kv != 0) return FIBATTN_ERR_INVALID_ARG;
    if (!q || !k || !v || !o || !lse || !dO || !dq || !dk || !dv || !dalpha || !table)
        return FIBATTN_ERR_INVALID_ARG;
    const void *ptrs[] = {q, k, v, o, lse, dO, dq, dk, dv, table};
    for (const void *p : ptrs)
        if (!aligned16(p)) return FIBATTN_ERR_INVALID_ARG;
    if (!(rope_base == 0.f || (rope_base > 1.f && isfinite(rope_base)))) return FIBATTN_ERR_INVALID_ARG;
    const WorkspaceLayout wl = workspace_layout(B, H, T, d_head, W, 0);
    if (!workspace || !aligned16(workspace) || workspace_bytes < wl.total) return FIBATTN_ERR_WORKSPACE;
    RungTable unused;
    memset(&unused, 0, sizeof(unused));
    float *delta_ws = (float *)workspace;
    double *partials = (double *)((char *)workspace + wl.partials);
    const RungTerms terms{(uint32_t *)((char *)workspace + wl.terms), wl.planes};
    const RopeFreq rf = make_rope_freq((double)rope_base, d_head);
    const Heads hd{H, H / H_kv};
    hipError_t e = launch_backward((int)dtype, d_head, q, k, v, o, lse, dO, dq, dk, dv, dalpha, dtheta,
                                   delta_ws, partials, terms, B * H, hd, T, W, unused,
                                   (const RungTable *)table, rf, rope_base,
                                   packed_layouts(H, H_kv, T, d_head), stream);
    return e == hipSuccess ? FIBATTN_OK : FIBATTN_ERR_HIP;
}

fibattn_status_t fibattn_alpha_from_theta(const float *theta, float *alpha, int n, hipStream_t stream) {
    if (!theta || !alpha || n < 1) return FIBATTN_ERR_INVALID_ARG;
    hipError_t e = launch_alpha_from_theta(theta, alpha, n, stream);
    return e == hipSuccess ? FIBATTN_OK : FIBATTN_ERR_HIP;
}

fibattn_status_t fibattn_dtheta(const float *theta, const float *dalpha, float *dtheta, int n,
                                hipStream_t stream) {
    if (!theta || !dalpha || !dtheta || n < 1) return FIBATTN_ERR_INVALID_ARG;
    hipError_t e = launch_dtheta(theta, dalpha, dtheta, n, stream);
    return e == hipSuccess ? FIBATTN_OK : FIBATTN_ERR_HIP;
}

fibattn_status_t fibattn_rope(const void *x, void *y, int B, int H, int T, int d_head,
                              float rope_base, int transpose, fibattn_dtype_t dtype,
                              hipStream_t stream) {
    if (B < 1 || H < 1 || T < 1 || !x || !y) return FIBATTN_ERR_INVALID_ARG;
    if (!aligned16(x) || !aligned16(y)) return FIBATTN_ERR_INVALID_ARG;
    if (dtype != FIBATTN_FP32 && dtype != FIBATTN_BF16) return FIBATTN_ERR_INVALID_ARG;
    if (!(rope_base > 1.f) || !isfinite(rope_base)) return FIBATTN_ERR_INVALID_ARG;
    if (d_head != 32 && d_head != 64 && d_head != 128) return FIBATTN_ERR_UNSUPPORTED;
    if ((long long)B * H > 65535ll * 16) return FIBATTN_ERR_UNSUPPORTED;
    const Layout l = Layout::packed(H, T, d_head);
    hipError_t e = launch_rope((int)dtype, d_head, x, y, l, l, nullptr, nullptr, l, l, B * H, H, T,
                               rope_base, transpose, stream);
    return e == hipSuccess ? FIBATTN_OK : FIBATTN_ERR_HIP;
}

fibattn_status_t fibattn_rope_qk(const void *q, const void *k, void *q_out, void *k_out, int B, int H,
                                 int T, int d_head, float rope_base, fibattn_dtype_t dtype,
                                 hipStream_t stream) {
    if (B < 1 || H < 1 || T < 1 || !q || !k || !q_out || !k_out) return FIBATTN_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(q_out) || !aligned16(k_out))
        return FIBATTN_ERR_INVALID_ARG;
    if (dtype != FIBATTN_FP32 && dtype != FIBATTN_BF16) return FIBATTN_ERR_INVALID_ARG;
    if (!(rope_base > 1.f) || !isfinite(rope_base)) return FIBATTN_ERR_INVALID_ARG;
    if (d_head != 32 && d_head != 64 && d_head != 128) return FIBATTN_ERR_UNSUPPORTED;
    if ((long long)B * H > 65535ll * 16) return FIBATTN_ERR_UNSUPPORTED;
    const Layout l = Layout::packed(H, T, d_head);
    hipError_t e = launch_rope((int)dtype, d_head, q, q_out, l, l, k, k_out, l, l, B * H, H, T, rope_base,
                               0, stream);
    return e == hipSuccess ? FIBATTN_OK : FIBATTN_ERR_HIP;
}

fibattn_status_t fibattn_rope_qk_table(const void *q, const void *k, void *q_out, void *k_out, int B, int H,
                                       int H_kv, int T, int d_head, float rope_base, const float *theta,
                                       float *alpha, const int32_t *base, int K, int W, void *table,
                                       fibattn_dtype_t dtype, hipStream_t stream) {
    // q and q_out both null: k alone (its launch carries the table job)
    if (B < 1 || H < 1 || T < 1 || !k || !k_out || !q != !q_out) return FIBATTN_ERR_INVALID_ARG;
    if (H_kv < 1 || H_kv > H || H % H_kv != 0) return FIBATTN_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(q_out) || !aligned16(k_out))
        return FIBATTN_ERR_INVALID_ARG;
    if (dtype != FIBATTN_FP32 && dtype != FIBATTN_BF16) return FIBATTN_ERR_INVALID_ARG;
    if (!(rope_base > 1.f) || !isfinite(rope_base)) return FIBATTN_ERR_INVALID_ARG;
    if (d_head != 32 && d_head != 64 && d_head != 128) return FIBATTN_ERR_UNSUPPORTED;
    if ((long long)B * H > 65535ll * 16) return FIBATTN_ERR_UNSUPPORTED;
    TableJob job{};
    if (theta) {
        if (!table || !aligned16(table) || W < 0 || W > FIBATTN_MAX_WINDOW) return FIBATTN_ERR_INVALID_ARG;
        const fibattn_status_t st = check_base(base, K, &job.b);
        if (st != FIBATTN_OK) return st;
        job.theta = theta;
        job.alpha = alpha;
        job.out = (RungTable *)table;
        job.W = W;
    }
    const Layout lq = Layout::packed(H, T, d_head), lk = Layout::packed(H_kv, T, d_head);
    hipError_t e = q ? launch_rope((int)dtype, d_head, q, q_out, lq, lq, k, k_out, lk, lk, B * H, H, T, rope_base,
                                   0, stream, B * H_kv, H_kv, theta ? &job : nullptr)
                     : launch_rope((int)dtype, d_head, k, k_out, lk, lk, nullptr, nullptr, lk, lk, B * H_kv, H_kv, T,
                                   rope_base, 0, stream, 0, 0, theta ? &job : nullptr);
    return e == hipSuccess ? FIBATTN_OK : FIBATTN_ERR_HIP;
}

const char *fibattn_status_string(fibattn_status_t s) {
    switch (s) {
        case FIBATTN_OK: return "ok";
        case FIBATTN_ERR_INVALID_ARG: return "invalid argument";
        case FIBATTN_ERR_UNSUPPORTED: return "unsupported size or configuration";
        case FIBATTN_ERR_WORKSPACE: return "workspace missing or too small";
        case FIBATTN_ERR_HIP: return "HIP launch error";
        case FIBATTN_ERR_SCRATCH:
            return "problem needs more scratch than the allocation-free backward's static buffer "
                   "(FIBATTN_SCRATCH_BYTES = 64 MiB)";
        default: break;
    }
    return "unknown status";
}

fibattn_status_t fibattn_timing_begin(int kernel_id, int capacity) {
    if (kernel_id < 0 || kernel_id >= kNumKernels || capacity < 1 || capacity > 1 << 16)
        return FIBATTN_ERR_INVALID_ARG;
    for (hipEvent_t e : g_timing.ev) (void)hipEventDestroy(e);
    g_timing.ev.assign(2 * (size_t)capacity, nullptr);
    for (auto &e : g_timing.ev)
        if (hipEventCreate(&e) != hipSuccess) return FIBATTN_ERR_HIP;
    g_timing.id = kernel_id;
    g_timing.capacity = capacity;
    g_timing.used = 0;
    return FIBATTN_OK;
}

fibattn_status_t fibattn_timing_end(float *avg_ms, int *count) {
    if (!avg_ms || !count) return FIBATTN_ERR_INVALID_ARG;
    *avg_ms = 0.f;
    *count = g_timing.used;
    fibattn_status_t st = FIBATTN_OK;
    if (g_timing.used > 0) {
        if (hipEventSynchronize(g_timing.ev[2 * g_timing.used - 1]) != hipSuccess) st = FIBATTN_ERR_HIP;
        double tot = 0.0;
        for (int a = 0; a < g_timing.used && st == FIBATTN_OK; ++a) {
            float ms = 0.f;
            if (hipEventElapsedTime(&ms, g_timing.ev[2 * a], g_timing.ev[2 * a + 1]) != hipSuccess)
                st = FIBATTN_ERR_HIP;
            tot += ms;
        }
        *avg_ms = (float)(tot / g_timing.used);
    }
    for (hipEvent_t e : g_timing.ev) (void)hipEventDestroy(e);
    g_timing.ev.clear();
    g_timing.id = -1;
    g_timing.capacity = 0;
    g_timing.used = 0;
    return st;
}

}  // extern "C"
