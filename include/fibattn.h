/*
 * fibattn.h - C ABI of libfibattn.so: Fibonacci-offset sparse attention on AMD
 * Instinct MI355X (gfx950).
 *
 * Operation (Section 2 of "Depth-Staggered Fibonacci Spacing for Sparse Attention",
 * paragraphs "Attended set" and "Implementation note"):
 *   query i of each (batch b, head h) attends to
 *     - the dense local window, distances delta = 0..W (truncated at position 0);
 *     - K rung distances d_k = alpha * f_k shared by every query, f being an offset
 *       base table (the Fibonacci base 1,2,3,5,...,987 or a power-of-2 control).
 *   A rung is read at the continuous position i - d_k: its key and value are the
 *   linear blend (1 - w_k) * row[i - floor(d_k)] + w_k * row[i - floor(d_k) - 1],
 *   w_k = d_k - floor(d_k).  Logits are tau * <q_i, key>, tau = 1/sqrt(d_head);
 *   the output is the softmax-weighted sum of the (blended) values.
 *   RoPE is applied to q and k at their true positions before the gather
 *   (fibattn_rope; Section 2 "Attended set", Section 3 "Model and training").
 *
 * Conventions where the paper is silent (the oracle follows the same ones):
 *   - d_k = fl32(alpha * f_k): one IEEE float32 multiply, round to nearest even;
 *   - rungs with d_k <= W coincide with window distances (the attended set is a
 *     union) and are dropped; equal rung distances are kept once;
 *   - a rung with d_k > i reaches before position 0 and is masked for query i;
 *   - the rows are i - floor(d) and i - floor(d) - 1; row -1 (reached only when
 *     w == 0) is a zero vector, which matters only for dalpha.
 *
 * Memory and ownership:
 *   - every tensor pointer is DEVICE memory owned by the caller, contiguous,
 *     16-byte aligned, layout [B, H, T, d_head] (row = one position of one head);
 *   - lse is float32 [B, H, T]; dalpha is one float32 on the device;
 *   - `base` is a HOST array of K strictly increasing int32 values >= 1; it is
 *     read during the call and not retained;
 *   - the library allocates no device memory; the backward's scratch space is the
 *     caller's `workspace` buffer.
 *
 * Execution: each call validates its arguments on the host, then enqueues kernels
 * on `stream` (0 = the null stream) and returns without synchronising.  Faults
 * inside kernels surface at the caller's next synchronisation.  Results are
 * bitwise deterministic from run to run (no atomics; fixed-order reductions).
 *
 * Errors: a call with invalid arguments returns a status code and enqueues
 * nothing; it never aborts or throws.
 */
#ifndef FIBATTN_H
#define FIBATTN_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    FIBATTN_OK = 0,
    FIBATTN_ERR_INVALID_ARG = 1,  /* null/misaligned pointer, bad size, bad base table, bad alpha */
    FIBATTN_ERR_UNSUPPORTED = 2,  /* valid but not implemented: d_head, W or K beyond the limits */
    FIBATTN_ERR_WORKSPACE = 3,    /* backward workspace missing or too small */
    FIBATTN_ERR_HIP = 4,          /* a kernel launch failed (hipGetLastError) */
    FIBATTN_ERR_SCRATCH = 5,      /* the problem needs more than FIBATTN_SCRATCH_BYTES of scratch */
    /* not statuses: they give the type the range of int, so that any int a caller
     * passes (fibattn_status_string) is a valid value of it */
    FIBATTN_STATUS_MIN_ = -0x7fffffff - 1,
    FIBATTN_STATUS_MAX_ = 0x7fffffff
} fibattn_status_t;

typedef enum {
    FIBATTN_FP32 = 0,             /* float32 storage and arithmetic */
    FIBATTN_BF16 = 1,             /* bfloat16 storage, float32 arithmetic, one rounding per output */
    /* not dtypes: any int passed as a dtype is a valid value of the type, and every
     * value other than the two above is refused with FIBATTN_ERR_INVALID_ARG */
    FIBATTN_DTYPE_MIN_ = -0x7fffffff - 1,
    FIBATTN_DTYPE_MAX_ = 0x7fffffff
} fibattn_dtype_t;

#define FIBATTN_MAX_RUNGS 32      /* K <= 32 */
#define FIBATTN_MAX_WINDOW 128    /* W <= 128 */

/*
 * Rung table (host only, no GPU needed): the offsets every query shares.
 * Writes, in increasing distance, floor(d_k) to d0[], w_k to w[] and f_k to f[]
 * for the rungs kept after the inclusion and dedupe rules above, and their count
 * to *n.  Arrays must hold FIBATTN_MAX_RUNGS entries.
 * Returns FIBATTN_ERR_INVALID_ARG for a bad base table, K or alpha.
 */
fibattn_status_t fibattn_rung_table(float alpha, const int32_t *base, int K, int W,
                                    int32_t *d0, float *w, int32_t *f, int *n);

/*
 * Forward (Section 2 "Attended set").
 *   q, k : post-RoPE queries and keys, dtype, [B,H,T,d_head]
 *   v    : values, dtype, [B,H,T,d_head]
 *   o    : output, dtype, [B,H,T,d_head] (written)
 *   lse  : float32 [B,H,T] (written): natural-log log-sum-exp of the tau-scaled
 *          logits of each query, saved for the backward
 * Limits: d_head in {32, 64, 128}; 0 <= W <= FIBATTN_MAX_WINDOW; 0 <= K <= FIBATTN_MAX_RUNGS;
 * alpha finite and > 0; B*H <= 65535; B*H*T*d_head <= 2^40; one head's rows,
 * T*d_head elements, under 2^31 bytes (T < 2^24 for bfloat16 with d_head 64): else
 * FIBATTN_ERR_UNSUPPORTED.  bfloat16 with d_head 64 and W <= 16 runs the
 * matrix-core kernels; every other supported shape runs the generic kernels.
 */
fibattn_status_t fibattn_forward(const void *q, const void *k, const void *v,
                                 void *o, float *lse,
                                 int B, int H, int T, int d_head, int W,
                                 const int32_t *base, int K, float alpha,
                                 fibattn_dtype_t dtype, hipStream_t stream);

/* Bytes of device workspace fibattn_backward needs for these sizes (0 for bad sizes):
 * Delta (float32 [B,H,T]), the float64 dalpha partials and, when d_head = 64 and
 * W <= 16, one 4-byte term per query and rung (K of them; pass K = 0 for a device
 * table, whose rung count can be up to 32).  Its contents on entry are ignored. */
size_t fibattn_backward_workspace_bytes(int B, int H, int T, int d_head, int W, int K);

/*
 * Backward: exact gradient of the forward, the inclusion masks held constant
 * (a hard mask carries no gradient to alpha; Section 2 "Implementation note").
 *   q, k, v, o, lse : as passed to / returned by fibattn_forward
 *   dO   : upstream gradient of o, dtype, [B,H,T,d_head]
 *   dq, dk, dv : gradients (written), dtype; accumulated in float32, rounded once
 *   dalpha : device float32 (overwritten): sum over b, h, i and rung entries of
 *            f_k * dL/dw_k (dw_k/dalpha = f_k); reduced in float64 in fixed order
 *   workspace : device buffer of at least fibattn_backward_workspace_bytes(...)
 *   rope_base : 0 -> dq, dk are gradients w.r.t. the rotated q, k passed in;
 *               > 1 -> the inverse rotation R^T at true positions (same pairing and
 *               angles as fibattn_rope) is applied before the single rounding, so
 *               dq, dk are gradients w.r.t. the unrotated inputs of the RoPE step.
 * Same limits as the forward.
 */
fibattn_status_t fibattn_backward(const void *q, const void *k, const void *v,
                                  const void *o, const float *lse, const void *dO,
                                  void *dq, void *dk, void *dv, float *dalpha,
                                  void *workspace, size_t workspace_bytes,
                                  int B, int H, int T, int d_head, int W,
                                  const int32_t *base, int K, float alpha, float rope_base,
                                  fibattn_dtype_t dtype, hipStream_t stream);

/*
 * Grouped key/value heads (Section 3 "Model and training": the model's 8 query heads
 * share 2 key/value heads).  As fibattn_forward / fibattn_backward, with
 *   q, o, dO, dq : [B,H,T,d_head];  lse : [B,H,T]
 *   k, v, dk, dv : [B,H_kv,T,d_head], H_kv >= 1 dividing H
 * Query head h of batch b reads key/value head h / (H / H_kv) of batch b; dk, dv are
 * the sums over the H / H_kv query heads of each group (reduced inside the library
 * in a fixed order; no atomics).  The workspace is fibattn_backward_workspace_bytes
 * with the query head count H.  H_kv == H is exactly fibattn_forward /
 * fibattn_backward.  Returns FIBATTN_ERR_INVALID_ARG when H_kv does not divide H.
 */
fibattn_status_t fibattn_forward_gqa(const void *q, const void *k, const void *v,
                                     void *o, float *lse,
                                     int B, int H, int H_kv, int T, int d_head, int W,
                                     const int32_t *base, int K, float alpha,
                                     fibattn_dtype_t dtype, hipStream_t stream);

fibattn_status_t fibattn_backward_gqa(const void *q, const void *k, const void *v,
                                      const void *o, const float *lse, const void *dO,
                                      void *dq, void *dk, void *dv, float *dalpha,
                                      void *workspace, size_t workspace_bytes,
                                      int B, int H, int H_kv, int T, int d_head, int W,
                                      const int32_t *base, int K, float alpha, float rope_base,
                                      fibattn_dtype_t dtype, hipStream_t stream);

/*
 * The forward with RoPE applied to the queries where they are loaded (Section 2
 * "Attended set": rotary embeddings at the true positions, before the gather).  As
 * fibattn_forward_gqa, except that
 *   q     : the UNROTATED queries, dtype, [B,H,T,d_head] (read)
 *   k     : the keys already rotated (fibattn_rope, same rope_base), [B,H_kv,T,d_head]
 *   q_out : nullable; R q, dtype, [B,H,T,d_head] (written; may be q itself), the rotated
 *           queries a later fibattn_backward_gqa(..., rope_base) takes as q.  NULL
 *           (forward-only callers) writes nothing beyond o and lse.
 *   rope_base : > 1 and finite (else FIBATTN_ERR_INVALID_ARG); pairing and angles as
 *           fibattn_rope
 * A query row is read by its own query only, so it is rotated inside the forward at no
 * extra row traffic; a key row is read by up to 1 + W + K queries and is rotated once,
 * by the RoPE launch.  o and lse are those of fibattn_forward_gqa on (R q, k, v).
 * bfloat16 with d_head 64 and W <= 16 is one launch; its cos and sin come from the
 * hardware units (absolute error <= 2.3e-7 with the angle's float32 rounding, against
 * ~1e-7 for fibattn_rope), so an element of q_out can differ from fibattn_rope's by one
 * bfloat16 rounding step where the exact value lies that close to a rounding midpoint.
 * Other shapes run the RoPE launch on q into q_out, then the forward (q_out NULL:
 * FIBATTN_ERR_UNSUPPORTED).
 */
fibattn_status_t fibattn_forward_rope_q(const void *q, const void *k, const void *v,
                                        void *o, float *lse, void *q_out,
                                        int B, int H, int H_kv, int T, int d_head, int W,
                                        const int32_t *base, int K, float alpha, float rope_base,
                                        fibattn_dtype_t dtype, hipStream_t stream);

/*
 * Tensors in any placement whose rows are contiguous, e.g. q, k, v taken straight out
 * of a [B, T, H, d_head] or a packed [B, T, 3, H, d_head] projection output, without a
 * copy.  A layout gives element strides: element (b, h, t, c) of a [B, heads, T,
 * d_head] tensor is at  b*batch + h*head + t*pos + c  elements from its pointer.
 *   layouts (host array, read during the call):
 *     fibattn_forward_strided : 4 entries, for q, k, v, o
 *     fibattn_backward_strided: 8 entries, for q, k, v, o, dO, dq, dk, dv
 *   Requirements (else FIBATTN_ERR_INVALID_ARG): batch, head, pos >= 0 and multiples of
 *   16 bytes (8 bf16 or 4 float32 elements), so that every row is 16-byte aligned.
 *   FIBATTN_ERR_UNSUPPORTED when a row of a head starts 2^31 bytes or more after the
 *   head's first row.  lse and the workspace stay packed ([B,H,T] float32).  The caller
 *   guarantees that no two output rows overlap each other or an input row (not
 *   checked).  Otherwise exactly fibattn_forward_gqa / fibattn_backward_gqa; the
 *   packed entry points are these with layouts (H*T*d, T*d, d) (heads H or H_kv).
 */
typedef struct {
    int64_t batch, head, pos;
} fibattn_layout_t;

fibattn_status_t fibattn_forward_strided(const void *q, const void *k, const void *v,
                                         void *o, float *lse, const fibattn_layout_t *layouts,
                                         int B, int H, int H_kv, int T, int d_head, int W,
                                         const int32_t *base, int K, float alpha,
                                         fibattn_dtype_t dtype, hipStream_t stream);

fibattn_status_t fibattn_backward_strided(const void *q, const void *k, const void *v,
                                          const void *o, const float *lse, const void *dO,
                                          void *dq, void *dk, void *dv, float *dalpha,
                                          void *workspace, size_t workspace_bytes,
                                          const fibattn_layout_t *layouts,
                                          int B, int H, int H_kv, int T, int d_head, int W,
                                          const int32_t *base, int K, float alpha, float rope_base,
                                          fibattn_dtype_t dtype, hipStream_t stream);

/* fibattn_forward_rope_q with per-tensor placements (the fibattn_layout_t rules above):
 * layouts holds 5 entries, for q, k, v, o and q_out (the last ignored when q_out is
 * NULL), e.g. q, k, v as slices of a fused [B,T,3,H,d] projection output. */
fibattn_status_t fibattn_forward_rope_q_strided(const void *q, const void *k, const void *v,
                                                void *o, float *lse, void *q_out,
                                                const fibattn_layout_t *layouts,
                                                int B, int H, int H_kv, int T, int d_head, int W,
                                                const int32_t *base, int K, float alpha,
                                                float rope_base, fibattn_dtype_t dtype,
                                                hipStream_t stream);

/*
 * Device-resident alpha (Section 2, "The per-layer scalar": alpha = 0.5 + sigmoid(theta)
 * with theta learned per layer), so that a training step never reads alpha on the host.
 *
 * fibattn_device_table builds, on the stream, the rung table of *alpha (a device
 * float) for a host base table (same rules and errors as fibattn_rung_table, checked
 * on the host) and window W into `table`, a caller-owned device buffer of
 * fibattn_device_table_bytes() bytes, 16-byte aligned.  The table is read by
 * fibattn_forward_dt / fibattn_backward_dt, which take it in place of (base, K, alpha)
 * and otherwise behave as fibattn_forward_gqa / fibattn_backward_gqa; W must be the
 * one the table was built with (the table records it: called with another W, every
 * output is NaN, as for a bad alpha), and the backward's workspace is
 * fibattn_backward_workspace_bytes(B, H, T, d_head, W, 0).  A table may hold any weights, so these calls always
 * run the interpolating kernels.  An alpha that is not finite and positive yields a
 * table that makes every output (o, lse, dq, dk, dv, dalpha) NaN.
 *
 * fibattn_alpha_from_theta: alpha[l] = 0.5 + sigmoid(theta[l]), l < n (sigmoid in
 * float64, rounded once to float32).  fibattn_dtheta: dtheta[l] = dalpha[l] *
 * sigmoid(theta[l]) (1 - sigmoid(theta[l])).  All pointers are device float32 arrays.
 *
 * fibattn_device_table_theta: the layer's step in one launch instead of two: from one
 * device float theta it writes alpha = 0.5 + sigmoid(theta) to *alpha (skipped when
 * alpha is NULL; the same value as fibattn_alpha_from_theta) and builds that alpha's
 * table (as fibattn_device_table), which also records d alpha / d theta.  Given such a
 * table, fibattn_backward_dt writes dL/dtheta = dalpha * sigmoid (1 - sigmoid) to its
 * `dtheta` argument (the value fibattn_dtheta computes from the stored dalpha), so the
 * learned-alpha step needs no launch of its own besides the table.  dtheta may be NULL;
 * with a table built from alpha (fibattn_device_table) it receives NaN.
 */
size_t fibattn_device_table_bytes(void);

fibattn_status_t fibattn_device_table(const float *alpha, const int32_t *base, int K, int W,
                                      void *table, hipStream_t stream);

fibattn_status_t fibattn_forward_dt(const void *q, const void *k, const void *v,
                                    void *o, float *lse,
                                    int B, int H, int H_kv, int T, int d_head, int W,
                                    const void *table, fibattn_dtype_t dtype, hipStream_t stream);

/* fibattn_forward_rope_q with the rung table in device memory (as fibattn_forward_dt):
 * q unrotated, k rotated, q_out nullable; the same limits and errors as both. */
fibattn_status_t fibattn_forward_rope_q_dt(const void *q, const void *k, const void *v,
                                           void *o, float *lse, void *q_out,
                                           int B, int H, int H_kv, int T, int d_head, int W,
                                           const void *table, float rope_base,
                                           fibattn_dtype_t dtype, hipStream_t stream);

fibattn_status_t fibattn_backward_dt(const void *q, const void *k, const void *v,
                                     const void *o, const float *lse, const void *dO,
                                     void *dq, void *dk, void *dv, float *dalpha, float *dtheta,
                                     void *workspace, size_t workspace_bytes,
                                     int B, int H, int H_kv, int T, int d_head, int W,
                                     const void *table, float rope_base,
                                     fibattn_dtype_t dtype, hipStream_t stream);

fibattn_status_t fibattn_device_table_theta(const float *theta, float *alpha,
                                            const int32_t *base, int K, int W,
                                            void *table, hipStream_t stream);

fibattn_status_t fibattn_alpha_from_theta(const float *theta, float *alpha, int n,
                                          hipStream_t stream);

fibattn_status_t fibattn_dtheta(const float *theta, const float *dalpha, float *dtheta, int n,
                                hipStream_t stream);

/*
 * RoPE at the true positions t = 0..T-1 (Section 2 "Attended set"; base 1e4 in
 * Section 3).  Rotate-half pairing: (x_j, x_{j+D/2}) rotates by the angle
 * t * rope_base^(-2j/D), j < D/2; angles are evaluated in float64 and their cosine
 * and sine rounded to float32.  transpose != 0 applies the inverse rotation R^T,
 * which carries gradients of rotated tensors back to the unrotated ones.
 *   x : input, dtype, [B,H,T,d_head];  y : output (may equal x), same layout.
 * Limits: d_head in {32, 64, 128}; rope_base finite and > 1.
 */
fibattn_status_t fibattn_rope(const void *x, void *y, int B, int H, int T, int d_head,
                              float rope_base, int transpose,
                              fibattn_dtype_t dtype, hipStream_t stream);

/*
 * RoPE of q and k in one launch: q_out = R q, k_out = R k (same rotation as
 * fibattn_rope with transpose = 0; outputs may alias their inputs).
 */
fibattn_status_t fibattn_rope_qk(const void *q, const void *k, void *q_out, void *k_out,
                                 int B, int H, int T, int d_head, float rope_base,
                                 fibattn_dtype_t dtype, hipStream_t stream);

/*
 * Backward that allocates nothing and takes no workspace: for callers that cannot
 * allocate device memory during the call (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc).  Arguments, semantics and results are those
 * of fibattn_backward_gqa (bitwise the same outputs, same kernels), without
 * `workspace` / `workspace_bytes`: the scratch (Delta, the dalpha partials and the
 * per-(query, rung) terms) lives in a static device array of FIBATTN_SCRATCH_BYTES
 * that the library holds on every GPU it runs on until the process ends.  Its address
 * on a device is looked up once (on the first call whose stream is on that device).
 *   Returns FIBATTN_ERR_SCRATCH, enqueueing nothing, when
 *   fibattn_backward_workspace_bytes(B, H, T, d_head, W, K) exceeds
 *   FIBATTN_SCRATCH_BYTES (e.g. B*H*T above ~1e6 query-heads at K = 15, d_head 64).
 *   Every call on one GPU shares that GPU's array and leaves its contents behind:
 *   calls that overlap on one GPU (concurrent streams, or host threads whose calls'
 *   kernels can run at the same time) race on it and must be serialised by the caller.
 *   Nothing in the array needs to start at zero.
 */
#define FIBATTN_SCRATCH_BYTES ((size_t)64 << 20)

fibattn_status_t fibattn_backward_noalloc(const void *q, const void *k, const void *v,
                                          const void *o, const float *lse, const void *dO,
                                          void *dq, void *dk, void *dv, float *dalpha,
                                          int B, int H, int H_kv, int T, int d_head, int W,
                                          const int32_t *base, int K, float alpha, float rope_base,
                                          fibattn_dtype_t dtype, hipStream_t stream);

/*
 * A layer's prologue in one launch: RoPE of q [B,H,T,d_head] and k [B,H_kv,T,d_head]
 * (H_kv dividing H: grouped heads) as fibattn_rope_qk, and, when theta is not NULL, the
 * layer's rung table from theta (as fibattn_device_table_theta: alpha = 0.5 +
 * sigmoid(theta) written to *alpha unless alpha is NULL, the table of that alpha for
 * (base, K, W) written to `table`, which also records d alpha / d theta).  So the step
 * of a layer with a learned alpha launches as many kernels as one with a host alpha:
 * this, fibattn_forward_dt and fibattn_backward_dt (which then also returns dtheta).
 * With theta NULL, base, K, W and table are ignored.  q and q_out both NULL rotate k
 * alone (the launch still carries the table job): the prologue of a step whose forward
 * rotates q on load (fibattn_forward_rope_q_dt).  Same limits and errors as
 * fibattn_rope_qk and fibattn_device_table_theta.
 */
fibattn_status_t fibattn_rope_qk_table(const void *q, const void *k, void *q_out, void *k_out,
                                       int B, int H, int H_kv, int T, int d_head, float rope_base,
                                       const float *theta, float *alpha, const int32_t *base, int K,
                                       int W, void *table, fibattn_dtype_t dtype, hipStream_t stream);

/* Human-readable name of a status code (static storage). */
const char *fibattn_status_string(fibattn_status_t status);

/*
 * Kernel timing (instrumentation for benchmarks).  The state is per host thread:
 * fibattn_timing_begin(id, capacity) makes the library launch each of the next
 * `capacity` launches of kernel `id` made by the calling thread with a HIP event
 * pair that takes the dispatch's
 * own start and end timestamps on the launch stream (0 rope, 1 forward, 2 backward
 * dq+dalpha, 3 backward dk/dv, 4 dalpha reduce, 5 device-alpha kernels).
 * fibattn_timing_end(&avg_ms, &count) synchronises on the last event, returns
 * the mean launch duration and the number of launches timed, and stops timing.
 */
fibattn_status_t fibattn_timing_begin(int kernel_id, int capacity);
fibattn_status_t fibattn_timing_end(float *avg_ms, int *count);

#ifdef __cplusplus
}
#endif

#endif /* FIBATTN_H */
