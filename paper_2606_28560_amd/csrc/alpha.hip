// Device-resident alpha (Section 2, "The per-layer scalar"): alpha_l = 0.5 +
// sigmoid(theta_l) with theta a learned parameter, so that a training step can run
// without reading theta back to the host.  The rung table is then built on the
// device with the same rules as the host table (rung_table_fill), and the gradient
// dL/dalpha that the backward produces is carried to theta.
#include "launch.h"

namespace fibattn {

__global__ void rung_table_kernel(const float *__restrict__ alpha, BaseTable b, int W,
                                  RungTable *__restrict__ out) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    RungTable t;
    rung_table_fill(*alpha, b, W, &t);  // n = -1 when alpha is not finite and positive
    *out = t;
}

__global__ void rung_table_theta_kernel(const float *__restrict__ theta, float *__restrict__ alpha_out,
                                        BaseTable b, int W, RungTable *__restrict__ out) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    table_from_theta(theta, alpha_out, b, W, out);  // alpha as alpha_from_theta_kernel
}

// sigmoid in float64, rounded once to float32 (the host schedules round the same way)
__global__ __launch_bounds__(256) void alpha_from_theta_kernel(const float *__restrict__ theta,
                                                               float *__restrict__ alpha, int n) {
    const int l = blockIdx.x * 256 + threadIdx.x;
    if (l < n) alpha[l] = (float)(0.5 + 1.0 / (1.0 + exp(-(double)theta[l])));
}

// d alpha / d theta = sigmoid(theta) (1 - sigmoid(theta))
__global__ __launch_bounds__(256) void dtheta_kernel(const float *__restrict__ theta,
                                                     const float *__restrict__ dalpha,
                                                     float *__restrict__ dtheta, int n) {
    const int l = blockIdx.x * 256 + threadIdx.x;
    if (l < n) {
        const double sg = 1.0 / (1.0 + exp(-(double)theta[l]));
        dtheta[l] = (float)((double)dalpha[l] * sg * (1.0 - sg));
    }
}

hipError_t launch_rung_table(const float *alpha, const BaseTable &b, int W, RungTable *out,
                             hipStream_t s) {
    return launch(kAlpha, rung_table_kernel, dim3(1), dim3(64), 0, s, alpha, b, W, out);
}

hipError_t launch_rung_table_theta(const float *theta, float *alpha_out, const BaseTable &b, int W,
                                   RungTable *out, hipStream_t s) {
    return launch(kAlpha, rung_table_theta_kernel, dim3(1), dim3(64), 0, s, theta, alpha_out, b, W, out);
}

hipError_t launch_alpha_from_theta(const float *theta, float *alpha, int n, hipStream_t s) {
    return launch(kAlpha, alpha_from_theta_kernel, dim3((n + 255) / 256), dim3(256), 0, s, theta,
                  alpha, n);
}

hipError_t launch_dtheta(const float *theta, const float *dalpha, float *dtheta, int n,
                         hipStream_t s) {
    return launch(kAlpha, dtheta_kernel, dim3((n + 255) / 256), dim3(256), 0, s, theta, dalpha,
                  dtheta, n);
}

}  // namespace fibattn
