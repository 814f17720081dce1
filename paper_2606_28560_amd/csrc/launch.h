// Host-side launchers of the fibattn kernels (internal to libfibattn.so).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace fibattn {

enum KernelId { kRope = 0, kForward = 1, kBwdDq = 2, kBwdDkDv = 3, kDalphaReduce = 4, kAlpha = 5,
                kNumKernels = 6 };

// The start/stop event pair for the next launch of kernel `id` while kernel timing is
// active for it; false otherwise.
bool timing_events(int id, hipEvent_t *start, hipEvent_t *stop);

// Launches `kernel`; while timing is active for `id` the launch carries an event pair that
// takes the dispatch's own start and end timestamps (hipExtLaunchKernel), so the pair
// measures this kernel alone, free of marker packets and launch gaps.
template <typename... P, typename... A>
hipError_t launch(int id, void (*kernel)(P...), dim3 grid, dim3 block, unsigned lds, hipStream_t s,
                  A... args) {
    hipEvent_t e0, e1;
    if (timing_events(id, &e0, &e1))
        hipExtLaunchKernelGGL(kernel, grid, block, lds, s, e0, e1, 0u, static_cast<P>(args)...);
    else
        hipLaunchKernelGGL(kernel, grid, block, lds, s, static_cast<P>(args)...);
    return hipGetLastError();
}

// dtype: 0 float32, 1 bfloat16.  All launchers return hipGetLastError() of their launches.
// BH = batch * query heads; k, v (and dk, dv) hold BH / hd.G heads.  rtp != nullptr:
// the rung table is the device-resident one at rtp (rt unused).
hipError_t launch_forward(int dtype, int D, const void *q, const void *k, const void *v, void *o,
                          float *lse, int BH, const Heads &hd, int T, int W, const RungTable &rt,
                          const RungTable *rtp, const Layouts &lay, hipStream_t s);

// Number of dalpha partials the dq kernel writes (one per workgroup).
size_t bwd_num_partials(int dtype, int D, int BH, int T);

// dtheta (nullable, device tables only): also writes dalpha * rtp->dadtheta there.
hipError_t launch_backward(int dtype, int D, const void *q, const void *k, const void *v,
                           const void *o, const float *lse, const void *dO, void *dq, void *dk,
                           void *dv, float *dalpha, float *dtheta, float *delta_ws, double *partials,
                           const RungTerms &terms, int BH, const Heads &hd, int T, int W,
                           const RungTable &rt, const RungTable *rtp, const RopeFreq &rf,
                           float rope_base, const Layouts &lay, hipStream_t s);

// bfloat16, d_head = 64, W <= 16: matrix-core band + VALU rungs (fwd_mfma.hip, bwd_mfma.hip).
bool forward_mfma_supported(int dtype, int D, int W);
// rq: q is unrotated and each query row is rotated with these frequencies where the
// forward loads it; the rotated rows go to q_rot, placed by lay.dq, unless it is null.
hipError_t launch_forward_mfma(const void *q, const void *k, const void *v, void *o, float *lse,
                               int BH, const Heads &hd, int T, int W, const RungTable &rt,
                               const RungTable *rtp, const Layouts &lay, hipStream_t s,
                               const RopeFreq *rq = nullptr, void *q_rot = nullptr);
bool backward_mfma_supported(int dtype, int D, int W);
size_t bwd_mfma_num_partials(int BH, int T);
hipError_t launch_backward_mfma(const void *q, const void *k, const void *v, const void *o,
                                const float *lse, const void *dO, void *dq, void *dk, void *dv,
                                float *dalpha, float *dtheta, float *delta_ws, double *partials,
                                const RungTerms &terms, int BH, const Heads &hd, int T, int W,
                                const RungTable &rt, const RungTable *rtp, const RopeFreq &rf,
                                const Layouts &lay, hipStream_t s);

RopeFreq make_rope_freq(double rope_base, int D);  // on = 0 when rope_base <= 0

// Device-resident alpha: builds the rung table from *alpha (one thread) into *out.
hipError_t launch_rung_table(const float *alpha, const BaseTable &b, int W, RungTable *out,
                             hipStream_t s);
// The same from *theta: alpha = 0.5 + sigmoid(theta) (written to *alpha_out when not null)
// and the table, which also records d alpha / d theta, in one launch.
hipError_t launch_rung_table_theta(const float *theta, float *alpha_out, const BaseTable &b, int W,
                                   RungTable *out, hipStream_t s);
// alpha_l = 0.5 + sigmoid(theta_l); dtheta_l = dalpha_l sigmoid(theta_l) (1 - sigmoid(theta_l)).
hipError_t launch_alpha_from_theta(const float *theta, float *alpha, int n, hipStream_t s);
hipError_t launch_dtheta(const float *theta, const float *dalpha, float *dtheta, int n, hipStream_t s);

// RoPE of one tensor (x1 == nullptr) or of two tensors in one launch: BH = batch * heads
// rows of the first, BH1 rows of heads1 heads of the second (BH1 <= 0: same as the first);
// inputs and outputs placed by their layouts.  A table job (may be null) is carried by
// the first launch.
hipError_t launch_rope(int dtype, int D, const void *x0, void *y0, const Layout &lx0, const Layout &ly0,
                       const void *x1, void *y1, const Layout &lx1, const Layout &ly1, int BH, int heads,
                       int T, float rope_base, int transpose, hipStream_t s, int BH1 = 0, int heads1 = 0,
                       const TableJob *job = nullptr);

}  // namespace fibattn
