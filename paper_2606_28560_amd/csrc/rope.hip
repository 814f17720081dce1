// RoPE at true positions (Section 2 "Attended set": rotary embeddings are applied
// at the true positions before gathering; Section 3: base 1e4).
//
// Rotate-half pairing: for j < D/2 the pair (x_j, x_{j+D/2}) of the row at position t
// rotates by theta = t * base^(-2j/D).  A workgroup owns a few consecutive positions
// and a group of (b, h) rows at those positions; it evaluates cos/sin of its angles
// once, in float64, rounds them to float32 in LDS, and rotates every row with them.
#include "launch.h"

namespace fibattn {

constexpr int kRopeTP = 8;   // positions per workgroup (generic kernel)
constexpr int kRopeRB = 16;  // (b, h) rows per workgroup (generic kernel)

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

// Generic kernel (any storage type and head size): one element pair per thread.
// BH = batch * heads rows of positions [0, T); x and y placed by lx and ly.
template <typename S, int D>
__global__ __launch_bounds__(256) void rope_kernel(const S *x, S *y, int BH, int T, double rope_base,
                                                   int transpose, int heads, Layout lx, Layout ly,
                                                   TableJob job) {
    constexpr int HALF = D / 2;
    __shared__ float cs[kRopeTP * HALF], sn[kRopeTP * HALF];
    if (job.out && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0)
        table_from_theta(job.theta, job.alpha, job.b, job.W, job.out);
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
        const S *xr = x + lx.head(bh, heads) + (long long)t * lx.st;
        S *yr = y + ly.head(bh, heads) + (long long)t * ly.st;
        const float c = cs[tt * HALF + jj], s = sn[tt * HALF + jj];
        const float u = ld1<S>(xr + jj);
        const float w = ld1<S>(xr + jj + HALF);
        st1<S>(yr + jj, u * c - w * s);
        st1<S>(yr + jj + HALF, w * c + u * s);
    }
}

// bfloat16, d_head 64: a workgroup owns 4 NP positions of 16 (b, h) rows; each lane group
// of four handles NP positions (t, t + 4) of one head.  NP = 2 (two rows' loads in flight
// per lane) for two tensors (10.7 -> 10.2 us for q and k of the 60M layer) and for one
// tensor of at least 2^17 rows (k of the T = 4096 layer: 11.4 -> 10.1 us); NP = 1 for a
// smaller single tensor, which doubles its workgroup count (k of the T = 1024 layer keeps
// 1024 workgroups).
// Lane group g of a row's four lanes holds dims [8g, 8g+8) and [32+8g, 32+8g+8),
// i.e. the eight rotate-half pairs (j, j+32), j in [8g, 8g+8): two 16-byte loads
// and stores per lane and row, reading 64 contiguous bytes per row per instruction.
// The loads are issued before the angles are evaluated.
constexpr int kRope64RB = 16;

// two float32 -> bfloat16 (round to nearest even) in one conversion instruction
typedef __bf16 rope_bf16x2 __attribute__((ext_vector_type(2)));
typedef float rope_f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((rope_f32x2){lo, hi}, rope_bf16x2));
}

// blockIdx.z selects the tensor: (x0 -> y0) or (x1 -> y1), each with its own row count
// (batch * heads) and head count (k may have fewer heads than q) and placed by its io
// (STRIDED; else every tensor is packed [BH, T, 64]).
struct RopeIO {
    Layout x, y;
    int BH, heads;
};
template <bool STRIDED, int NP>
__global__ __launch_bounds__(256) void rope_bf16_d64_kernel(const uint16_t *x0, uint16_t *y0,
                                                            const uint16_t *x1, uint16_t *y1,
                                                            int T, RopeFreq rf, int transpose,
                                                            RopeIO io0, RopeIO io1, TableJob job) {
    constexpr int kRope64TP = 4 * NP;  // positions per workgroup
    __shared__ float cs[kRope64TP * 32], sn[kRope64TP * 32];
    const uint16_t *x = blockIdx.z ? x1 : x0;
    uint16_t *y = blockIdx.z ? y1 : y0;
    const RopeIO &io = blockIdx.z ? io1 : io0;
    const int BH = io.BH, heads = io.heads;
    if (job.out && blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0 && threadIdx.x == 0)
        table_from_theta(job.theta, job.alpha, job.b, job.W, job.out);
    if (blockIdx.y * kRope64RB >= BH) return;  // the tensor with fewer heads
    const int t0 = blockIdx.x * kRope64TP;
    const int g = threadIdx.x & 3;
    const int rr = threadIdx.x >> 2;  // 0..63
    const int bh = blockIdx.y * kRope64RB + (rr >> 2);
    const int bhc = min(bh, BH - 1);
    uint4 a[NP], b[NP];
    const uint16_t *xr[NP];
    uint16_t *yr[NP];
#pragma unroll
    for (int h = 0; h < NP; ++h) {  // positions t0 + (rr & 3) (and t0 + (rr & 3) + 4)
        const int tc = min(t0 + (rr & 3) + 4 * h, T - 1);
        const size_t packed = ((size_t)bhc * T + tc) * 64;
        xr[h] = x + (STRIDED ? io.x.head(bhc, heads) + (long long)tc * io.x.st : packed);
        yr[h] = y + (STRIDED ? io.y.head(bhc, heads) + (long long)tc * io.y.st : packed);
        a[h] = *reinterpret_cast<const uint4 *>(xr[h] + 8 * g);
        b[h] = *reinterpret_cast<const uint4 *>(xr[h] + 32 + 8 * g);
    }
    if (threadIdx.x < kRope64TP * 32) {
        float c, sv;
        rope_cs(t0 + (threadIdx.x >> 5), rf.inv[threadIdx.x & 31], c, sv);
        cs[threadIdx.x] = c;
        sn[threadIdx.x] = transpose ? -sv : sv;
    }
    __syncthreads();
    if (bh >= BH) return;
#pragma unroll
    for (int h = 0; h < NP; ++h) {
        const int tt = (rr & 3) + 4 * h;
        if (t0 + tt >= T) continue;
        const uint32_t aw[4] = {a[h].x, a[h].y, a[h].z, a[h].w}, bw[4] = {b[h].x, b[h].y, b[h].z, b[h].w};
        uint32_t ow[4], pw[4];
        const float *C = cs + tt * 32 + 8 * g;
        const float *Sn = sn + tt * 32 + 8 * g;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const float u0 = bf16_lo(aw[w]), u1 = bf16_hi(aw[w]);
            const float v0 = bf16_lo(bw[w]), v1 = bf16_hi(bw[w]);
            const float c0 = C[2 * w], c1 = C[2 * w + 1], s0 = Sn[2 * w], s1 = Sn[2 * w + 1];
            ow[w] = pack2_bf16(u0 * c0 - v0 * s0, u1 * c1 - v1 * s1);
            pw[w] = pack2_bf16(v0 * c0 + u0 * s0, v1 * c1 + u1 * s1);
        }
        *reinterpret_cast<uint4 *>(yr[h] + 8 * g) = make_uint4(ow[0], ow[1], ow[2], ow[3]);
        *reinterpret_cast<uint4 *>(yr[h] + 32 + 8 * g) = make_uint4(pw[0], pw[1], pw[2], pw[3]);
    }
}

RopeFreq make_rope_freq(double rope_base, int D) {
    RopeFreq rf;
    rf.on = rope_base > 0.0;
    for (int j = 0; j < 32; ++j) rf.inv[j] = (j < D / 2 && rf.on) ? pow(rope_base, -2.0 * (double)j / (double)D) : 0.0;
    return rf;
}

static hipError_t launch_rope_generic(int dtype, int D, const void *x, void *y, int BH, int T,
                                      double lb, int transpose, int heads, const Layout &lx,
                                      const Layout &ly, const TableJob &job, hipStream_t s) {
    dim3 grid((T + kRopeTP - 1) / kRopeTP, (BH + kRopeRB - 1) / kRopeRB);
#define FIBATTN_ROPE(S, DD)                                                                          \
    if ((dtype == 0) == (sizeof(S) == 4) && D == DD)                                                  \
        return launch(kRope, rope_kernel<S, DD>, grid, dim3(256), 0, s, x, y, BH, T, lb, transpose, \
                      heads, lx, ly, job);
    FIBATTN_ROPE(float, 32)
    FIBATTN_ROPE(float, 64)
    FIBATTN_ROPE(float, 128)
    FIBATTN_ROPE(uint16_t, 32)
    FIBATTN_ROPE(uint16_t, 64)
    FIBATTN_ROPE(uint16_t, 128)
#undef FIBATTN_ROPE
    return hipErrorInvalidValue;
}

// One launch for one tensor (x1 == nullptr) or two tensors (BH1 rows of heads1 heads for
// the second); BH = batch * heads rows; each input and output placed by its layout.  The
// table job (job.out set) rides on the first launch.
hipError_t launch_rope(int dtype, int D, const void *x0, void *y0, const Layout &lx0, const Layout &ly0,
                       const void *x1, void *y1, const Layout &lx1, const Layout &ly1, int BH, int heads,
                       int T, float rope_base, int transpose, hipStream_t s, int BH1, int heads1,
                       const TableJob *job) {
    const double lb = (double)rope_base;
    TableJob nojob{};
    const TableJob &tj = job ? *job : nojob;
    if (BH1 <= 0) { BH1 = BH; heads1 = heads; }
    if (dtype == 1 && D == 64) {
        const RopeFreq rf = make_rope_freq(lb, 64);
        auto same = [&](const Layout &l, int hs) {
            const Layout p = Layout::packed(hs, T, 64);
            return l.sb == p.sb && l.sh == p.sh && l.st == p.st;
        };
        const bool strided = !same(lx0, heads) || !same(ly0, heads) ||
                             (x1 && (!same(lx1, heads1) || !same(ly1, heads1)));
        const int rows = x1 ? max(BH, BH1) : BH;
        const bool np2 = x1 || (long long)BH * T >= (1ll << 17);
        const int tp = np2 ? 8 : 4;  // positions per workgroup
        auto kern = np2 ? (strided ? rope_bf16_d64_kernel<true, 2> : rope_bf16_d64_kernel<false, 2>)
                        : (strided ? rope_bf16_d64_kernel<true, 1> : rope_bf16_d64_kernel<false, 1>);
        return launch(kRope, kern,
                      dim3((T + tp - 1) / tp, (rows + kRope64RB - 1) / kRope64RB, x1 ? 2 : 1),
                      dim3(256), 0, s, x0, y0, x1, y1, T, rf, transpose, RopeIO{lx0, ly0, BH, heads},
                      RopeIO{lx1, ly1, BH1, heads1}, tj);
    }
    hipError_t e = launch_rope_generic(dtype, D, x0, y0, BH, T, lb, transpose, heads, lx0, ly0, tj, s);
    if (e == hipSuccess && x1)
        e = launch_rope_generic(dtype, D, x1, y1, BH1, T, lb, transpose, heads1, lx1, ly1, nojob, s);
    return e;
}

}  // namespace fibattn
