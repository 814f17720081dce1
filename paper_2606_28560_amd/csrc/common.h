// Device-side helpers shared by the fibattn kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fibattn {

constexpr int kMaxRungs = 32;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Rung table: the offsets every query of a launch shares (floor of the distance,
// blend weight, base value), increasing d, for the window W it was built with.  Passed
// by value in the kernel arguments, or built on the device from a device-resident alpha
// (rung_table_fill).  n < 0 marks a table built from an alpha that is not finite and
// positive; kernels reading a device table write NaN for such a table and for one
// built with another W (table_unusable).
struct RungTable {
    int n;
    int W;
    int d0[kMaxRungs];
    float w[kMaxRungs];
    int f[kMaxRungs];
    // d alpha / d theta = sigmoid(theta) (1 - sigmoid(theta)) for a table built from theta
    // (alpha = 0.5 + sigmoid(theta)); NaN for a table built from alpha itself
    double dadtheta;
};

// A device-built table that must not be used for a launch with window W: its alpha
// was not finite and positive, or it was built for another window (its in-window rule
// then dropped or kept the wrong rungs).
__host__ __device__ inline bool table_unusable(const RungTable &rt, int W) { return rt.n < 0 || rt.W != W; }

// A validated base table (strictly increasing, >= 1, K <= kMaxRungs) by value.
struct BaseTable {
    int K;
    int f[kMaxRungs];
};

// Section 2 rung rules for a validated base: d_k = fl32(alpha * f_k) (one float32
// multiply), a rung with d_k <= W coincides with the window and is dropped (the
// attended set is a union), equal distances are one entry; w = d - floor(d) is exact.
// Returns false (and an empty table with n = -1) when alpha is not finite and
// positive or a distance overflows int.
__host__ __device__ inline bool rung_table_fill(float alpha, const BaseTable &b, int W, RungTable *rt) {
    for (int a = 0; a < kMaxRungs; ++a) { rt->d0[a] = 0; rt->w[a] = 0.f; rt->f[a] = 0; }
    rt->n = -1;
    rt->W = W;
    rt->dadtheta = __builtin_nan("");
    if (!(alpha > 0.f) || !(alpha < INFINITY)) return false;
    int n = 0;
    float last = -1.f;
    for (int a = 0; a < b.K; ++a) {
        const float d = alpha * (float)b.f[a];
        if (!(d <= 2147483520.f)) { rt->n = -1; return false; }
        if (!(d > (float)W)) continue;     // coincides with the window
        if (n > 0 && d == last) continue;  // equal distances are one entry
        const float fl = floorf(d);
        rt->d0[n] = (int)fl;
        rt->w[n] = d - fl;
        rt->f[n] = b.f[a];
        last = d;
        ++n;
    }
    rt->n = n;
    return true;
}

// The table of a layer whose alpha is learned (Section 2, "The per-layer scalar"):
// alpha = 0.5 + sigmoid(theta) with the sigmoid in float64 and one rounding to float32
// (as the host schedules), the table of that alpha, and d alpha / d theta.  One thread.
__device__ inline void table_from_theta(const float *theta, float *alpha_out, const BaseTable &b, int W,
                                        RungTable *out) {
    const double sg = 1.0 / (1.0 + exp(-(double)*theta));
    const float alpha = (float)(0.5 + sg);
    RungTable t;
    rung_table_fill(alpha, b, W, &t);
    t.dadtheta = sg * (1.0 - sg);
    *out = t;
    if (alpha_out) *alpha_out = alpha;
}

// A table build carried by another launch (the RoPE of a learned-alpha layer): done by
// thread 0 of block 0 when `out` is set.
struct TableJob {
    const float *theta;
    float *alpha;
    RungTable *out;
    BaseTable b;
    int W;
};

// Per-(query, rung) terms of the backward that the dq kernel of the matrix-core path
// hands to its dk/dv kernel: for query i of flat head bh and rung r of the table, the
// bfloat16 pair (tau dS, p) (tau dS in the low half) at index (bh * planes + r) * T + i
// (planes >= the table's n).  The dk/dv accumulation rounds these weights to bfloat16
// anyway.
struct RungTerms {
    uint32_t *p;
    int planes;
};

// Grouped key/value heads (Section 3 "Model and training": 8 query heads share 2
// key/value heads): query head h of batch b reads key/value head h / G of that batch.
struct Heads {
    int H;  // query heads per batch
    int G;  // query heads per key/value head (1: one key/value head per query head)
    __host__ __device__ int kv_heads() const { return H / G; }
    // (batch * H + h) -> (batch * H/G + h/G)
    __host__ __device__ int kv_of(int bh) const { return (bh / H) * (H / G) + (bh % H) / G; }
    // (batch * H/G + hk), group member g -> batch * H + hk * G + g
    __host__ __device__ int q_of(int bk, int g) const { return (bk / (H / G)) * H + (bk % (H / G)) * G + g; }
};

// Placement of a [B, heads, T, d] tensor whose rows (the d elements of one position
// of one head) are contiguous: element (b, h, t, c) at b*sb + h*sh + t*st + c, in
// elements.  The packed layout is (heads*T*d, T*d, d).
struct Layout {
    long long sb, sh, st;
    __host__ __device__ static Layout packed(int heads, int T, int D) {
        return {(long long)heads * T * D, (long long)T * D, (long long)D};
    }
    // element offset of row 0 of the flat head index bh = b * heads + h
    __host__ __device__ long long head(int bh, int heads) const {
        return (long long)(bh / heads) * sb + (long long)(bh % heads) * sh;
    }
};
// Element offset of row 0 of head bh: from the layout when STRIDED, else packed
// [*, T, D] (the layout is then not read, keeping its fields out of registers).
template <bool STRIDED, int D>
__device__ __forceinline__ long long head_at(const Layout &l, int bh, int heads, int T) {
    return STRIDED ? l.head(bh, heads) : (long long)bh * T * D;
}
// The tensors of a launch: q, k, v, o, and for the backward dO, dq, dk, dv.  k, v,
// dk, dv have the key/value head count.
struct Layouts {
    Layout q, k, v, o, g, dq, dk, dv;
};
// Whether a placement is exactly the packed one, the only one the kernels' packed
// (STRIDED = false) instances address: equal row strides alone do not make it so (a
// slice of a longer sequence has packed rows but a larger head stride).
inline bool is_packed(const Layout &l, int heads, int T, int D) {
    const Layout p = Layout::packed(heads, T, D);
    return l.sb == p.sb && l.sh == p.sh && l.st == p.st;
}

// RoPE inverse frequencies base^(-2j/D) for j < D/2 <= 32, evaluated in float64 on
// the host; `on` = 0 when no rotation is requested.
struct RopeFreq {
    double inv[32];
    int on;
};

// cos/sin of t * inv_freq: the angle and its reduction to [-pi, pi] are float64, the
// reduced angle is evaluated with float32 sincosf (error ~1e-7 absolute).
__device__ __forceinline__ void rope_cs(int t, double inv_freq, float &c, float &s) {
    const double a = (double)t * inv_freq;
    const double two_pi = 6.283185307179586476925286766559;
    const double r = a - two_pi * rint(a * (1.0 / two_pi));
    sincosf((float)r, &s, &c);
}

// cos and sin of the angle 2 pi t fr (fr: revolutions per position): t fr is reduced to
// [-1/2, 1/2] in float64, rounded to float32 (angle error <= 2 pi 2^-26) and evaluated on
// the hardware sine and cosine units, whose inputs are in revolutions (max absolute error
// 1.3e-7, measured over 2^24 points of [-1/2, 1/2]).
__device__ __forceinline__ void rope_cs_rev(int t, double fr, float &c, float &s) {
    const double a = (double)t * fr;
    const float r = (float)(a - rint(a));
    s = __builtin_amdgcn_sinf(r);
    c = __builtin_amdgcn_cosf(r);
}

// RoPE rotation of the rotate-half pair (u, v) = (x_j, x_{j + D/2}) by the angle with
// cosine c and sine s, with explicit fused multiply-adds.
__device__ __forceinline__ void rope_rotate(float u, float v, float c, float s, float &x, float &y) {
    x = fmaf(u, c, -(v * s));
    y = fmaf(v, c, u * s);
}

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
// 16-byte store that does not allocate in the caches (the outputs are not read again
// by this kernel)
__device__ __forceinline__ void nt_store16(void *p, uint4 x) {
    __builtin_nontemporal_store(u32x4{x.x, x.y, x.z, x.w}, reinterpret_cast<u32x4 *>(p));
}

// ---- storage types -------------------------------------------------------
// A lane moves 16 bytes of a row at a time: 4 float32 or 8 bfloat16 values.
__device__ __forceinline__ float bf16_lo(uint32_t x) { return __uint_as_float(x << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t x) { return __uint_as_float(x & 0xffff0000u); }

// float32 -> bfloat16 bits, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

template <typename S> struct Vec;

template <> struct Vec<float> {
    static constexpr int N = 4;
    __device__ __forceinline__ static void load(const float *p, float *x) {
        float4 t = *reinterpret_cast<const float4 *>(p);
        x[0] = t.x; x[1] = t.y; x[2] = t.z; x[3] = t.w;
    }
    __device__ __forceinline__ static void store(float *p, const float *x) {
        *reinterpret_cast<float4 *>(p) = make_float4(x[0], x[1], x[2], x[3]);
    }
};

template <> struct Vec<uint16_t> {
    static constexpr int N = 8;
    __device__ __forceinline__ static void load(const uint16_t *p, float *x) {
        uint4 t = *reinterpret_cast<const uint4 *>(p);
        x[0] = bf16_lo(t.x); x[1] = bf16_hi(t.x);
        x[2] = bf16_lo(t.y); x[3] = bf16_hi(t.y);
        x[4] = bf16_lo(t.z); x[5] = bf16_hi(t.z);
        x[6] = bf16_lo(t.w); x[7] = bf16_hi(t.w);
    }
    __device__ __forceinline__ static void store(uint16_t *p, const float *x) {
        uint4 t;
        t.x = f32_to_bf16(x[0]) | (f32_to_bf16(x[1]) << 16);
        t.y = f32_to_bf16(x[2]) | (f32_to_bf16(x[3]) << 16);
        t.z = f32_to_bf16(x[4]) | (f32_to_bf16(x[5]) << 16);
        t.w = f32_to_bf16(x[6]) | (f32_to_bf16(x[7]) << 16);
        *reinterpret_cast<uint4 *>(p) = t;
    }
};

// Sum over the G lanes of an aligned lane group (G a power of two, G <= 64).
template <int G>
__device__ __forceinline__ float group_sum(float x) {
#pragma unroll
    for (int m = G / 2; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
    return x;
}

template <int N>
__device__ __forceinline__ float dot(const float *a, const float *b) {
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < N; ++c) s = fmaf(a[c], b[c], s);
    return s;
}

}  // namespace fibattn
