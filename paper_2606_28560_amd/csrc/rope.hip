// RoPE at true positions (Section 2 "Attended set": rotary embeddings are applied
// at the true positions before gathering; Section 3: base 1e4).
//
// Rotate-half pairing: for j < D/2 the pair (x_j, x_{j+D/2}) of the row at position t
// rotates by theta = t * base^(-2j/D).  A workgroup owns TP consecutive positions and
// RB rows (b, h) at those positions; it evaluates cos/sin of its TP * D/2 angles once,
// in float64, rounds them to float32 in LDS, and rotates every row with them.
#include "launch.h"

namespace fibattn {

constexpr int kRopeTP = 8;   // positions per workgroup
constexpr int kRopeRB = 16;  // (b, h) rows per workgroup

template <typename S> __device__ __forceinline__ float ld1(const S *p);
template <> __device__ __forceinline__ float ld1<float>(const float *p) { return *p; }
template <> __device__ __forceinline__ float ld1<uint16_t>(const uint16_t *p) {
    return __uint_as_float((uint32_t)(*p) << 16);
}
template <typename S> __device__ __forceinline__ void st1(S *p, float x);
template <> __device__ __forceinline__ void st1<float>(float *p, float x) { *p = x; }
template <> __device__ __forceinline__ void st1<uint16_t>(uint16_t *p, float x) {
    *p = (uint16_t)f32_to_bf16(x);
}

template <typename S, int D>
__global__ __launch_bounds__(256) void rope_kernel(const S *x, S *y,
                                                   int BH, int T, double rope_base,
                                                   int transpose) {
    constexpr int HALF = D / 2;
    __shared__ float cs[kRopeTP * HALF], sn[kRopeTP * HALF];
    const int t0 = blockIdx.x * kRopeTP;
    for (int a = threadIdx.x; a < kRopeTP * HALF; a += 256) {
        const int t = t0 + a / HALF;
        const int jj = a % HALF;
        const double inv_freq = pow(rope_base, -2.0 * (double)jj / (double)D);
        const double ang = (double)t * inv_freq;
        double sv, cv;
        sincos(ang, &sv, &cv);
        cs[a] = (float)cv;
        sn[a] = transpose ? -(float)sv : (float)sv;
    }
    __syncthreads();
    const int bh0 = blockIdx.y * kRopeRB;
    for (int a = threadIdx.x; a < kRopeRB * kRopeTP * HALF; a += 256) {
        const int jj = a % HALF;
        const int tt = (a / HALF) % kRopeTP;
        const int rr = a / (HALF * kRopeTP);
        const int t = t0 + tt;
        const int bh = bh0 + rr;
        if (t >= T || bh >= BH) continue;
        const size_t row = ((size_t)bh * T + t) * D;
        const float c = cs[tt * HALF + jj], s = sn[tt * HALF + jj];
        const float u = ld1<S>(x + row + jj);
        const float w = ld1<S>(x + row + jj + HALF);
        st1<S>(y + row + jj, u * c - w * s);
        st1<S>(y + row + jj + HALF, w * c + u * s);
    }
}

hipError_t launch_rope(int dtype, int D, const void *x, void *y, int BH, int T, float rope_base,
                       int transpose, hipStream_t s) {
    dim3 grid((T + kRopeTP - 1) / kRopeTP, (BH + kRopeRB - 1) / kRopeRB);
    const double lb = (double)rope_base;
    timing_before(kRope, s);
    if (dtype == 0 && D == 32)
        hipLaunchKernelGGL((rope_kernel<float, 32>), grid, dim3(256), 0, s, (const float *)x,
                           (float *)y, BH, T, lb, transpose);
    else if (dtype == 0 && D == 64)
        hipLaunchKernelGGL((rope_kernel<float, 64>), grid, dim3(256), 0, s, (const float *)x,
                           (float *)y, BH, T, lb, transpose);
    else if (dtype == 1 && D == 32)
        hipLaunchKernelGGL((rope_kernel<uint16_t, 32>), grid, dim3(256), 0, s,
                           (const uint16_t *)x, (uint16_t *)y, BH, T, lb, transpose);
    else if (dtype == 1 && D == 64)
        hipLaunchKernelGGL((rope_kernel<uint16_t, 64>), grid, dim3(256), 0, s,
                           (const uint16_t *)x, (uint16_t *)y, BH, T, lb, transpose);
    else
        return hipErrorInvalidValue;
    timing_after(kRope, s);
    return hipGetLastError();
}

}  // namespace fibattn
