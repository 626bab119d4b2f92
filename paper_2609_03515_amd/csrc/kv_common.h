// Device helpers shared by the eviction-path kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace ikv {

constexpr int kWave = 64;

typedef __bf16 __attribute__((ext_vector_type(2))) bf16x2;
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Cross-lane exchange inside a 16-lane DPP row.  Controls used here:
//   0xB1 quad_perm [1,0,3,2] (lane ^ 1)     0x4E quad_perm [2,3,0,1] (lane ^ 2)
//   0x141 row_half_mirror (lane ^ 7 inside each 8-lane half)      0x128 row_ror:8 (lane ^ 8 inside 16)
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
    return __builtin_amdgcn_update_dpp(0.0f, x, CTRL, 0xF, 0xF, true);
}
constexpr int kXor1 = 0xB1;
constexpr int kXor2 = 0x4E;
constexpr int kMirror8 = 0x141;
constexpr int kRor8 = 0x128;

// Partner control for the butterfly step that separates lanes by bit `mask` (1, 2, 4, 8) of the lane
// index inside its aligned group; the partner differs in that bit and agrees on all higher bits.
template <int MASK>
struct StepCtrl;
template <> struct StepCtrl<1> { static constexpr int v = kXor1; };
template <> struct StepCtrl<2> { static constexpr int v = kXor2; };
template <> struct StepCtrl<4> { static constexpr int v = kMirror8; };
template <> struct StepCtrl<8> { static constexpr int v = kRor8; };

// Sum over the aligned group of W lanes (W in 1, 2, 4, 8, 16); every lane of the group gets the total.
template <int W>
__device__ __forceinline__ float group_allsum(float x) {
    if constexpr (W >= 2) x += dpp<kXor1>(x);
    if constexpr (W >= 4) x += dpp<kXor2>(x);
    if constexpr (W >= 8) x += dpp<kMirror8>(x);
    if constexpr (W >= 16) x += dpp<kRor8>(x);
    return x;
}

// Reduce-scatter of V = W values over an aligned group of W lanes: afterwards v[0] of the lane with in-group
// index p holds the group total of value index p.  At each step the lane keeps the half of the remaining
// indices selected by its own bit and adds the partner's copy of the same indices.
template <int W, int HALF>
__device__ __forceinline__ void scatter_step(float (&v)[W], int p) {
    const bool upper = (p & HALF) != 0;
#pragma unroll
    for (int i = 0; i < HALF; ++i) {
        const float lo = v[i], hi = v[i + HALF];
        const float keep = upper ? hi : lo;
        const float send = upper ? lo : hi;
        v[i] = keep + dpp<StepCtrl<HALF>::v>(send);
    }
}
template <int W>
__device__ __forceinline__ float reduce_scatter(float (&v)[W], int p) {
    if constexpr (W >= 16) scatter_step<W, 8>(v, p);
    if constexpr (W >= 8) scatter_step<W, 4>(v, p);
    if constexpr (W >= 4) scatter_step<W, 2>(v, p);
    if constexpr (W >= 2) scatter_step<W, 1>(v, p);
    return v[0];
}

// Exchanges between the four 16-lane rows of a wave with gfx950's row swaps, which run on the vector ALU
// instead of the LDS crossbar that a cross-row shuffle (ds_bpermute) goes through:
//   v_permlane16_swap a, b: row 1 of a <-> row 0 of b, row 3 of a <-> row 2 of b;
//   v_permlane32_swap a, b: rows 2, 3 of a <-> rows 0, 1 of b.
// They are issued from inline assembly with two wait states before (a vector ALU write of an operand just
// before the swap) and after: the compiler's builtins for these instructions return a wrong second result
// after its instruction combining (seen in its output: the second half of the swap replaced by the first).
__device__ __forceinline__ void swap_rows16(float& a, float& b) {
    asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ void swap_rows32(float& a, float& b) {
    asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
}

// Sum over the four rows at the lane's position, (row0 + row1) + (row2 + row3) in every lane: the order of a
// xor-16-then-xor-32 butterfly, so the result is bit-identical to it.
__device__ __forceinline__ float rows_allsum(float x) {
    float a = x, b = x;
    swap_rows16(a, b);  // a = [x0 x0 x2 x2], b = [x1 x1 x3 x3]
    float c = a + b, d = c;
    swap_rows32(c, d);  // c = [x01 x01 x01 x01], d = [x23 x23 x23 x23]
    return c + d;
}
__device__ __forceinline__ float rows_allmax(float x) {
    float a = x, b = x;
    swap_rows16(a, b);
    float c = fmaxf(a, b), d = c;
    swap_rows32(c, d);
    return fmaxf(c, d);
}
// Four values reduced over the rows at once: row r of the result holds the sum of value r (a, b, e, f for
// r = 0..3) at the lane's position, again (row0 + row1) + (row2 + row3).
__device__ __forceinline__ float rows_sum4(float a, float b, float e, float f) {
    swap_rows16(a, b);  // a = [a0 b0 a2 b2], b = [a1 b1 a3 b3]
    swap_rows16(e, f);
    float ab = a + b, ef = e + f;  // [a01 b01 a23 b23], [e01 f01 e23 f23]
    swap_rows32(ab, ef);           // [a01 b01 e01 f01], [a23 b23 e23 f23]
    return ab + ef;
}

// Online-softmax pair (running max, sum of exp(z - max)).
struct MaxSum {
    float m, s;
};
__device__ __forceinline__ MaxSum ms_combine(MaxSum a, MaxSum b) {
    const float m = fmaxf(a.m, b.m);
    if (m == -INFINITY) return {m, 0.0f};
    return {m, a.s * __expf(a.m - m) + b.s * __expf(b.m - m)};
}
// (a.m and b.m are finite or -inf; a pair whose max is the finite floor used by the scorer has sum 0.)

// Order-preserving map of a float onto uint32 (larger float -> larger key; -0 < +0).
__device__ __forceinline__ uint32_t float_key(float x) {
    const uint32_t b = __float_as_uint(x);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Eviction order of single-eviction steps: a leaves before b when its utility key is lower, or equal with a
// higher position (ties keep the lower position); a candidate with idx < 0 is none.
__device__ __forceinline__ bool evicts_before(const EvictCand& a, const EvictCand& b) {
    return b.idx < 0 || (a.idx >= 0 && (a.key < b.key || (a.key == b.key && a.pos > b.pos)));
}
__device__ __forceinline__ EvictCand shfl_xor_cand(const EvictCand& c, int o) {
    return EvictCand{(uint32_t)__shfl_xor((int)c.key, o, 64), __shfl_xor(c.pos, o, 64), __shfl_xor(c.idx, o, 64)};
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, kWave));
    return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, kWave);
    return x;
}

// Element traits: 16-byte chunk of a K row and of a query, and the dot product of two chunks.
template <typename T>
struct Elem;

template <>
struct Elem<float> {
    static constexpr int kPerChunk = 4;
    typedef f32x4 chunk_t;
    __device__ __forceinline__ static float dot(const chunk_t& k, const chunk_t& q, float acc) {
        acc = fmaf(k.x, q.x, acc);
        acc = fmaf(k.y, q.y, acc);
        acc = fmaf(k.z, q.z, acc);
        acc = fmaf(k.w, q.w, acc);
        return acc;
    }
    __device__ __forceinline__ static void unpack(const chunk_t& c, float (&f)[kPerChunk]) {
        f[0] = c.x;
        f[1] = c.y;
        f[2] = c.z;
        f[3] = c.w;
    }
    __device__ __forceinline__ static void store(float* dst, float x) { *dst = x; }
};

struct bf16_t {
    uint16_t bits;
};

template <>
struct Elem<bf16_t> {
    static constexpr int kPerChunk = 8;
    typedef u32x4 chunk_t;  // 8 bf16 as 4 packed pairs
    __device__ __forceinline__ static float dot2(uint32_t a, uint32_t b, float acc) {
        return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b),
                                               acc, false);
    }
    __device__ __forceinline__ static float dot(const chunk_t& k, const chunk_t& q, float acc) {
        acc = dot2(k.x, q.x, acc);
        acc = dot2(k.y, q.y, acc);
        acc = dot2(k.z, q.z, acc);
        acc = dot2(k.w, q.w, acc);
        return acc;
    }
    // bf16 -> f32 is exact: the bf16 bits are the high half of the f32 bits
    __device__ __forceinline__ static void unpack(const chunk_t& c, float (&f)[kPerChunk]) {
        const uint32_t w[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            f[2 * i] = __uint_as_float(w[i] << 16);
            f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    }
    // f32 -> bf16 rounding to nearest, ties to even (inputs are finite)
    __device__ __forceinline__ static void store(bf16_t* dst, float x) {
        const uint32_t b = __float_as_uint(x);
        dst->bits = (uint16_t)((b + 0x7fffu + ((b >> 16) & 1u)) >> 16);
    }
};

// l2 norm of one value row, as every producer of VNorm's norms computes it: an aligned group of LPR lanes
// (LPR = min(16, the row's 16-byte chunks)), lane p squaring and adding the elements of its chunks p, p + LPR,
// ... in order, then a DPP sum over the group.  The same arithmetic at append time and in a pass over V gives
// bit-identical norms.  Every lane of the group must call it (the sum crosses lanes).
template <typename T, int LPR, int CPL>
__device__ __forceinline__ float row_norm_lanes(const typename Elem<T>::chunk_t (&c)[CPL]) {
    float ss = 0.0f;
#pragma unroll
    for (int cc = 0; cc < CPL; ++cc) {
        float f[Elem<T>::kPerChunk];
        Elem<T>::unpack(c[cc], f);
#pragma unroll
        for (int x = 0; x < Elem<T>::kPerChunk; ++x) ss = fmaf(f[x], f[x], ss);
    }
    return sqrtf(group_allsum<LPR>(ss));
}

// Lanes per row of row_norm (the group size): min(16, row_bytes / 16).
__device__ __forceinline__ int norm_lanes(int row_bytes) { return row_bytes >= 256 ? 16 : row_bytes / 16; }

// row_norm_lanes for a row of `row_bytes` bytes (64 or 128 elements of bf16 or f32) at `row`, 16-byte aligned;
// p = the lane's index in its group of norm_lanes(row_bytes) lanes.
__device__ __forceinline__ float row_norm(const void* row, int row_bytes, bool bf16, int p) {
    const u32x4* rp = static_cast<const u32x4*>(row);
    if (bf16) {
        const u32x4 c[1] = {rp[p]};
        return row_bytes == 256 ? row_norm_lanes<bf16_t, 16, 1>(c) : row_norm_lanes<bf16_t, 8, 1>(c);
    }
    if (row_bytes == 512) {
        const f32x4 c[2] = {__builtin_bit_cast(f32x4, rp[p]), __builtin_bit_cast(f32x4, rp[p + 16])};
        return row_norm_lanes<float, 16, 2>(c);
    }
    const f32x4 c[1] = {__builtin_bit_cast(f32x4, rp[p])};
    return row_norm_lanes<float, 16, 1>(c);
}

__host__ __device__ constexpr int ilog2(int x) { return x <= 1 ? 0 : 1 + ilog2(x >> 1); }
__host__ __device__ constexpr size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

}  // namespace ikv
