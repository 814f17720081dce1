// Helpers for the bfloat16, d_head = 64 kernels built on gfx950 matrix cores.
//
// Lane layout shared by these kernels: a wave owns 16 consecutive rows (queries in
// the forward and dq kernels, keys in the dk/dv kernel).  Lane l serves row
// n = l % 16 and, with g = l / 16, the head dims [8g, 8g+8) and [32+8g, 32+8g+8)
// (its "slice"), so a row is spread over the four lanes n, n+16, n+32, n+48 and
// each 16-byte load instruction reads 64 contiguous bytes of each of 16 rows.
//
// This is also the layout of v_mfma_f32_16x16x32_bf16 (A: lane -> row l%16,
// k = 8(l/16)+j; B: lane -> column l%16, same k; C: lane -> column l%16, rows
// 4(l/16)+i).  The head-dim contraction of Q.K^T is two MFMAs whose k index 8g+j
// stands for dim 32s + 8g + j (s = 0, 1): each operand is half of the lane's slice.
// For products that sum over key/query rows, the output row m = 4g+i of dim block c
// stands for slice position 4c + i of lane group g (out_dim below), so lane (n, g)
// ends up holding exactly its own slice of the output row.
#pragma once

#include "common.h"

namespace fibattn {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef short v4i16 __attribute__((ext_vector_type(4)));

constexpr int kD = 64;

// 16 bfloat16 values of one row slice: a = dims [8g, 8g+8), b = [32+8g, 32+8g+8).
// Slice position d (0..15) is word d/2, low half for even d; positions 0..7 are in
// a, 8..15 in b.
struct Slice {
    uint4 a, b;
};

// Slice g of row `row` of rows `st` elements apart (64 contiguous bf16 each) at a
// uniform base address: a 32-bit byte offset from the base lets the loads use
// scalar-base addressing (the host keeps every row offset below 2^31 bytes).
__device__ __forceinline__ Slice load_row(const uint16_t *base, int row, int g, int st) {
    const uint32_t off = (uint32_t)row * (uint32_t)(2 * st) + (uint32_t)g * 16u;
    const char *p = reinterpret_cast<const char *>(base);
    Slice s;
    s.a = *reinterpret_cast<const uint4 *>(p + off);
    s.b = *reinterpret_cast<const uint4 *>(p + off + 64);
    return s;
}

// 2^x with the hardware instruction (no denormal rescaling; here x <= 8, and results
// below the float32 normal range are negligible weights).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ uint32_t word(const Slice &s, int w) {
    switch (w) {
        case 0: return s.a.x; case 1: return s.a.y; case 2: return s.a.z; case 3: return s.a.w;
        case 4: return s.b.x; case 5: return s.b.y; case 6: return s.b.z; default: return s.b.w;
    }
}

__device__ __forceinline__ bf16x2 as_bf2(uint32_t x) { return __builtin_bit_cast(bf16x2, x); }
__device__ __forceinline__ bf16x8 as_bf8(uint4 x) { return __builtin_bit_cast(bf16x8, x); }

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    f32x2 v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// <x, y> over the 16 dims of the slice (float32 accumulation of exact bf16 products).
__device__ __forceinline__ float dot_slice(const Slice &x, const Slice &y) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < 8; ++w) s = __builtin_amdgcn_fdot2_f32_bf16(as_bf2(word(x, w)), as_bf2(word(y, w)), s, false);
    return s;
}

// Sum / max over the four lanes that share a row in the MFMA layout (n, n+16, n+32, n+48).
__device__ __forceinline__ float sum4(float x) {
    x += __shfl_xor(x, 16, 64);
    x += __shfl_xor(x, 32, 64);
    return x;
}
__device__ __forceinline__ float max4(float x) {
    x = fmaxf(x, __shfl_xor(x, 16, 64));
    x = fmaxf(x, __shfl_xor(x, 32, 64));
    return x;
}

// Quad layout (used where rows are read from global memory one per lane group):
// lanes 4n .. 4n+3 share row n, lane 4n+g holding slice g of it, so the four lanes
// of a row read 64 contiguous bytes per load instruction.  Sums over a quad use DPP
// lane swaps (quad_perm [1,0,3,2] then [2,3,0,1]); every lane must be active.
__device__ __forceinline__ float quad_sum(float x) {  // folds into two v_add_f32_dpp
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, true));
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, true));
    return x;
}

// acc.c[c][i] holds slice position 4c + i of the lane's row.
struct Acc16 {
    f32x4 c[4];
};

__device__ __forceinline__ void acc_zero(Acc16 &a) {
#pragma unroll
    for (int c = 0; c < 4; ++c) a.c[c] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// acc += a * x with bf16 dot2 products, no unpacking: the weight pairs (a, 0) and
// (0, a) pick the low and the high element of each word (a rounded to bf16).
__device__ __forceinline__ void acc_axpy_bf(Acc16 &acc, float a, const Slice &x) {
    const uint32_t alo = pack_bf16(a, 0.f), ahi = alo << 16;
#pragma unroll
    for (int w = 0; w < 8; ++w) {
        const uint32_t u = word(x, w);
        const int d = 2 * w;
        acc.c[d >> 2][d & 3] = __builtin_amdgcn_fdot2_f32_bf16(as_bf2(u), as_bf2(alo), acc.c[d >> 2][d & 3], false);
        acc.c[(d + 1) >> 2][(d + 1) & 3] =
            __builtin_amdgcn_fdot2_f32_bf16(as_bf2(u), as_bf2(ahi), acc.c[(d + 1) >> 2][(d + 1) & 3], false);
    }
}

// acc += a * x + b * y with one bf16 dot2 per dim: the pair (x_d, y_d) is packed
// with v_perm; ab holds the bfloat16 weights (a in the low half).
__device__ __forceinline__ void acc_axpy2_bf(Acc16 &acc, uint32_t abits, const Slice &x, const Slice &y) {
    const bf16x2 ab = as_bf2(abits);
#pragma unroll
    for (int w = 0; w < 8; ++w) {
        const uint32_t xu = word(x, w), yu = word(y, w);
        const uint32_t lo = __builtin_amdgcn_perm(yu, xu, 0x05040100u);  // (x_lo, y_lo)
        const uint32_t hi = __builtin_amdgcn_perm(yu, xu, 0x07060302u);  // (x_hi, y_hi)
        const int d = 2 * w;
        acc.c[d >> 2][d & 3] = __builtin_amdgcn_fdot2_f32_bf16(as_bf2(lo), ab, acc.c[d >> 2][d & 3], false);
        acc.c[(d + 1) >> 2][(d + 1) & 3] =
            __builtin_amdgcn_fdot2_f32_bf16(as_bf2(hi), ab, acc.c[(d + 1) >> 2][(d + 1) & 3], false);
    }
}
// The same with float32 weights, rounded to bfloat16.
__device__ __forceinline__ void acc_axpy2(Acc16 &acc, float a, const Slice &x, float b, const Slice &y) {
    acc_axpy2_bf(acc, pack_bf16(a, b), x, y);
}

// Scaled store of the lane's slice as bf16 (two 16-byte stores).
__device__ __forceinline__ void store_acc(uint16_t *row, int g, const Acc16 &acc, float scale) {
    uint4 a, b;
    a.x = pack_bf16(acc.c[0][0] * scale, acc.c[0][1] * scale);
    a.y = pack_bf16(acc.c[0][2] * scale, acc.c[0][3] * scale);
    a.z = pack_bf16(acc.c[1][0] * scale, acc.c[1][1] * scale);
    a.w = pack_bf16(acc.c[1][2] * scale, acc.c[1][3] * scale);
    b.x = pack_bf16(acc.c[2][0] * scale, acc.c[2][1] * scale);
    b.y = pack_bf16(acc.c[2][2] * scale, acc.c[2][3] * scale);
    b.z = pack_bf16(acc.c[3][0] * scale, acc.c[3][1] * scale);
    b.w = pack_bf16(acc.c[3][2] * scale, acc.c[3][3] * scale);
    nt_store16(row + 8 * g, a);
    nt_store16(row + 32 + 8 * g, b);
}

// R^T (the inverse RoPE rotation) at position t on the lane's slice: slice positions
// d and d + 8 hold the rotate-half pair (8g + d, 32 + 8g + d); rev8 points at the
// eight frequencies (in revolutions per position) of lane group g.
__device__ __forceinline__ void acc_rope_t(Acc16 &a, int t, const double *rev8) {
#pragma unroll
    for (int d = 0; d < 8; ++d) {
        float c, s;
        rope_cs_rev(t, rev8[d], c, s);
        const float x = a.c[d >> 2][d & 3];
        const float y = a.c[2 + (d >> 2)][d & 3];
        a.c[d >> 2][d & 3] = x * c + y * s;
        a.c[2 + (d >> 2)][d & 3] = y * c - x * s;
    }
}

// Stage the RoPE frequencies in LDS as revolutions per position (inverse frequency /
// 2 pi; read by acc_rope_t after a barrier).
__device__ __forceinline__ void stage_freq(double *dst, const RopeFreq &rf) {
    if (threadIdx.x == 0) {
#pragma unroll
        for (int j = 0; j < 32; ++j) dst[j] = rf.inv[j] * 0.15915494309189533576888376337251;
    }
}

// Moves a value from the MFMA layout (row n on lanes n + 16g) to the quad layout
// (row n on lanes 4n + g): lane 4n + g takes the value of lane n + 16g.
__device__ __forceinline__ float to_quad(float x, int lane) {
    return __shfl(x, (lane >> 2) + 16 * (lane & 3), 64);
}
// A row slice held in the quad layout, moved to the MFMA layout (lane l serves row
// l % 16 with slice l / 16; quad lanes 4n..4n+3 hold the slices of row n).
__device__ __forceinline__ Slice slice_from_quad(const Slice &x, int lane) {
    const int src = 4 * (lane & 15) + (lane >> 4);
    Slice y;
    y.a.x = __shfl(x.a.x, src, 64); y.a.y = __shfl(x.a.y, src, 64);
    y.a.z = __shfl(x.a.z, src, 64); y.a.w = __shfl(x.a.w, src, 64);
    y.b.x = __shfl(x.b.x, src, 64); y.b.y = __shfl(x.b.y, src, 64);
    y.b.z = __shfl(x.b.z, src, 64); y.b.w = __shfl(x.b.w, src, 64);
    return y;
}
__device__ __forceinline__ void acc_to_quad(Acc16 &a, int lane) {
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int e = 0; e < 4; ++e) a.c[c][e] = to_quad(a.c[c][e], lane);
}

__device__ __forceinline__ f32x4 mfma(const bf16x8 &a, const bf16x8 &b, const f32x4 &c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// <row slices> over all 64 dims for 16 rows x 16 columns: A rows from `ar`, B
// columns from `bc` (both the lane's own slices).
__device__ __forceinline__ f32x4 mfma_dot64(const Slice &ar, const Slice &bc, f32x4 c) {
    c = mfma(as_bf8(ar.a), as_bf8(bc.a), c);
    c = mfma(as_bf8(ar.b), as_bf8(bc.b), c);
    return c;
}

// Output dim of row m in dim block c of a transposed-operand MFMA: slice position
// 4c + (m & 3) of lane group m / 4 (see top).
__device__ __forceinline__ int out_dim(int c, int m) {
    return (c < 2 ? 0 : 32) + 8 * (m >> 2) + 4 * (c & 1) + (m & 3);
}

// Rows [r_begin, r_begin + NROWS) of rows `st` elements apart (64 contiguous bf16
// each) copied to LDS with direct-to-LDS loads (no registers; completion counts in
// vmcnt): row-major, 128-byte
// rows whose 16-byte chunks are XOR-swizzled by the row (chunk c of band row r sits in
// slot c ^ (r & 7)), so that lanes reading one chunk of consecutive rows spread over
// the banks.  Rows outside [0, T) are clamped to a valid row: callers mask them.
// Each wave moves 1 KB (8 rows) per instruction.  256 threads.
template <int NROWS>
__device__ __forceinline__ void dma_rows(uint16_t *dst, const uint16_t *X, int r_begin, int T, int st) {
    static_assert(NROWS % 8 == 0, "whole 1 KB blocks");
    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
    for (int blk = wv; blk < NROWS / 8; blk += 4) {
        const int rr = 8 * blk + (lane >> 3);
        const int ch = (lane & 7) ^ (rr & 7);
        const int row = min(max(r_begin + rr, 0), T - 1);
        __builtin_amdgcn_global_load_lds(X + (size_t)row * st + 8 * ch, dst + 512 * blk, 16, 0, 0);
    }
}
// Chunk c (dims 8c..8c+7) of band row rr staged by dma_rows.
__device__ __forceinline__ uint4 dma_chunk(const uint16_t *src, int rr, int c) {
    return *reinterpret_cast<const uint4 *>(src + rr * kD + 8 * (c ^ (rr & 7)));
}
__device__ __forceinline__ Slice dma_slice(const uint16_t *src, int rr, int g) {
    Slice s;
    s.a = dma_chunk(src, rr, g);
    s.b = dma_chunk(src, rr, 4 + g);
    return s;
}
// A operand of a transposed-operand MFMA from rows staged by dma_rows: output dim
// out_dim(c, n) for lane n of each 16-lane group g; k index 8g + j is staged row
// base + 4g + (j & 3) + 16 (j >> 2).  Two gfx950 LDS transpose reads
// (ds_read_b64_tr_b16): in each 16-lane group, lane m points at 4 dims
// (8 bytes) of one row, and lane n receives element n % 4 of the blocks read by
// lanes n / 4, n / 4 + 4, n / 4 + 8 and n / 4 + 12.  So lane m reads row
// k0 + m / 4, dims B + 8 (m % 4) .. + 3, and lane n gets dim B + 8 (n / 4) + n % 4 of
// rows k0 .. k0 + 3: out_dim(c, n) with B = 32 [c >= 2] + 4 (c & 1).
__device__ __forceinline__ bf16x8 dma_operand_t(const uint16_t *src, int c, int /*n*/, int base, int g) {
    const int m = threadIdx.x & 15;
    const int ch = (c < 2 ? 0 : 4) + (m & 3);  // 16-byte chunk holding the lane's 4 dims
    const int off = 4 * (c & 1);
    v4i16 t[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int r = base + 16 * h + 4 * g + (m >> 2);
        t[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) v4i16 *)(src + r * kD + 8 * (ch ^ (r & 7)) + off));
    }
    return __builtin_bit_cast(bf16x8, t);
}
// Waits for this wave's outstanding vector-memory loads, direct-to-LDS ones included.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Block index -> work item, keeping consecutive work items (the tiles of one
// (batch, head)) on one XCD: workgroups are dispatched round-robin over 8 XCDs.
// Within an XCD the first round places dispatch positions j, j + 32, j + 64, ...
// on one CU (32 CUs per XCD).  Later tiles of a sequence carry more rungs (and
// early key tiles more rung queries), so every other run of 32 positions is
// reversed: a CU then holds tiles from both ends of the sequence rather than
// four tiles at the same position.
__device__ __forceinline__ int xcd_remap(int b, int nblocks) {
    if (nblocks & 7) return b;
    const int per = nblocks >> 3;
    int j = b >> 3;
    const int lo = j & ~31, hi = min(lo + 32, per);
    if ((j >> 5) & 1) j = lo + hi - 1 - j;
    return (b & 7) * per + j;
}

}  // namespace fibattn
