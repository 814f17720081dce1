// Host-side launchers of the fibattn kernels (internal to libfibattn.so).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace fibattn {

enum KernelId { kRope = 0, kForward = 1, kBwdDq = 2, kBwdDkDv = 3, kDalphaReduce = 4, kNumKernels = 5 };

// Records a HIP event before / after a launch when kernel timing is active for `id`.
void timing_before(int id, hipStream_t s);
void timing_after(int id, hipStream_t s);

// dtype: 0 float32, 1 bfloat16.  All launchers return hipGetLastError() of their launches.
hipError_t launch_forward(int dtype, int D, const void *q, const void *k, const void *v, void *o,
                          float *lse, int BH, int T, int W, const RungTable &rt, hipStream_t s);

// Number of dalpha partials the dq kernel writes (one per workgroup).
size_t bwd_num_partials(int dtype, int D, int BH, int T);

hipError_t launch_backward(int dtype, int D, const void *q, const void *k, const void *v,
                           const void *o, const float *lse, const void *dO, void *dq, void *dk,
                           void *dv, float *dalpha, float *delta_ws, double *partials, int BH,
                           int T, int W, const RungTable &rt, const RopeFreq &rf, float rope_base,
                           hipStream_t s);

// bfloat16, d_head = 64, W <= 16: matrix-core band + VALU rungs (fwd_mfma.hip, bwd_mfma.hip).
bool forward_mfma_supported(int dtype, int D, int W);
hipError_t launch_forward_mfma(const void *q, const void *k, const void *v, void *o, float *lse,
                               int BH, int T, int W, const RungTable &rt, hipStream_t s);
bool backward_mfma_supported(int dtype, int D, int W);
size_t bwd_mfma_num_partials(int BH, int T);
hipError_t launch_backward_mfma(const void *q, const void *k, const void *v, const void *o,
                                const float *lse, const void *dO, void *dq, void *dk, void *dv,
                                float *dalpha, float *delta_ws, double *partials, int BH, int T,
                                int W, const RungTable &rt, const RopeFreq &rf, hipStream_t s);

RopeFreq make_rope_freq(double rope_base, int D);  // on = 0 when rope_base <= 0

// RoPE of one tensor (x1 == nullptr) or of two same-shaped tensors in one launch.
hipError_t launch_rope(int dtype, int D, const void *x0, void *y0, const void *x1, void *y1, int BH,
                       int T, float rope_base, int transpose, hipStream_t s);

}  // namespace fibattn
