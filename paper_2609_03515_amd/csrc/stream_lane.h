// Streaming machinery shared by the scorer and the fused decode-attention kernels: one workgroup of 8 waves
// streams rows of a (layer, sequence, KV head) slab with raw buffer loads; a K row is split into 16-byte
// chunks over an aligned group of LPR lanes, each lane accumulates the partial dot products of RPG rows with
// the GP (padded) query heads of its group, and a DPP reduce-scatter leaves each lane with one full
// (row, head) logit.
#pragma once

#include "kernels.h"
#include "kv_common.h"

namespace ikv {
namespace {

#ifndef IKV_SCORE_WAVES
#define IKV_SCORE_WAVES 8
#endif
#ifndef IKV_NT_LOADS
#define IKV_NT_LOADS 1
#endif
#ifndef IKV_NBUF
#define IKV_NBUF 0
#endif
#ifndef IKV_LPR
#define IKV_LPR 16
#endif

constexpr size_t kFastLdsMax = 80 * 1024;  // keep >= 2 workgroups per CU (160 KiB LDS)
constexpr int kWaves = IKV_SCORE_WAVES;
constexpr int kThreads = kWaves * kWave;
constexpr float kFloor = -1.0e30f;  // finite start of running maxima: exp(-inf - floor) = 0, no NaN
constexpr int kNonTemporal = 2;     // buffer-load cache policy: K is streamed once, no reuse to cache for
constexpr int kRsrcConfig = 0x00020000;  // raw (unformatted, stride 0) buffer resource, gfx9 family

// Cache policy of the results written while K is still streaming (group sums, logits): device scope (sc1).
// Writes interleaved with the saturated read stream cost far more than their bytes; measured at the 8B shape,
// the 27 MB of group sums cost ~40 us of a 290 us launch with the default policy, ~24 us with this one
// (non-temporal: ~30 us).
constexpr int kStoreStream = 16;

// Raw buffer resource over `bytes` bytes at `base` (reads at offsets >= bytes return zero).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_rsrc(const void* base, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, kRsrcConfig);
}

// 16- and 4-byte stores at byte offset `off` of a raw buffer resource, with the streaming-result cache policy.
__device__ __forceinline__ void store_stream(__amdgpu_buffer_rsrc_t rs, int off, const f32x4& v) {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), rs, off, 0, kStoreStream);
}
__device__ __forceinline__ void store_stream(__amdgpu_buffer_rsrc_t rs, int off, float v) {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), rs, off, 0, kStoreStream);
}

template <typename T, int D, int GP>
struct Geometry {
    using E = Elem<T>;
    static constexpr int kEpc = E::kPerChunk;
    static constexpr int kChunks = D / kEpc;
    // Lanes per K row: IKV_LPR (16: one 16-byte chunk each for d = 128 bf16, a wave load covers 1 KiB of
    // consecutive rows), at least the padded group (the reduce-scatter leaves one (row, head) per lane), at
    // most the row's chunks.  A padded group of 8 over rows of at most 16 chunks takes 8 lanes instead: there
    // the dot products cost two instructions per byte of K and dominate the issue slots, and 8 lanes (two
    // chunks each, every load still on whole 128-byte lines) need a 3-step reduce-scatter of 8 values per
    // lane instead of a 4-step one of 16 (the Qwen-shaped steady step: 347 -> 320 us with the scorer's
    // schedule).  Group 4 gains nothing from it and the attention's V pass (two chunks of accumulators per
    // lane) loses 5-13%.
    static constexpr int kLprWide = (GP > IKV_LPR ? GP : IKV_LPR) < kChunks ? (GP > IKV_LPR ? GP : IKV_LPR) : kChunks;
    static constexpr int kLpr = (GP == 8 && kChunks <= 16) ? 8 : kLprWide;
    static constexpr int kCpl = kChunks / kLpr;
    static constexpr int kNg = kWave / kLpr;
    static constexpr int kRpg = kLpr / GP;
    static constexpr int kRpw = kNg * kRpg;
    static constexpr int kRpi = kWaves * kRpw;
    static_assert(kRpg * GP == kLpr, "group must not exceed the lanes of a row");
    // K loads of this many units are in flight per lane.  Rows are claimed dynamically and 2 measured best
    // (more buffers cost occupancy without raising the stream rate).
    static constexpr int kNbufLds = IKV_NBUF > 0 ? IKV_NBUF : 2;
    // Registers of the streaming loop: the K buffers in flight, the queries, the partial dot products and
    // bookkeeping.  LDS holds about 3 workgroups per CU at the graded shapes, so ask the compiler for the
    // matching waves per SIMD when the loop fits that register budget; otherwise leave it unconstrained
    // rather than spill.
    static constexpr int kWantWaves = (3 * kWaves + 3) / 4;
    static constexpr int min_waves(int nbuf) {
#ifdef IKV_MIN_WAVES
        return IKV_MIN_WAVES;
#else
        return nbuf * kRpg * kCpl * 4 + GP * kCpl * 4 + kLpr + 16 <= (512 / kWantWaves) / 8 * 8 ? kWantWaves : 1;
#endif
    }
    static constexpr int kMinWavesLds = min_waves(kNbufLds);
};

// Per-lane streaming machinery shared by both paths.
template <typename T, int D, int GP>
struct Lane {
    using Gm = Geometry<T, D, GP>;
    using E = Elem<T>;
    using chunk_t = typename E::chunk_t;
    static constexpr int LPR = Gm::kLpr, CPL = Gm::kCpl, NG = Gm::kNg, RPG = Gm::kRpg, RPW = Gm::kRpw;
    static constexpr int RPI = Gm::kRpi, EPC = Gm::kEpc;

    int lane, wave, grp, p, hh, kk;

    __device__ Lane() {
        lane = threadIdx.x & (kWave - 1);
        wave = threadIdx.x / kWave;
        grp = lane / LPR;
        p = lane % LPR;
        hh = p % GP;  // head owned after the reduce-scatter
        kk = p / GP;  // row slot owned after the reduce-scatter
    }

    // Row of iteration `it` owned by this lane after the reduce-scatter.
    __device__ int owned_row(int row0, int it) const { return row0 + it * RPI + wave * RPW + kk * NG + grp; }

    __device__ void load_q(const ScoreArgs& a, size_t lb, int g, chunk_t (&qv)[GP][CPL]) const {
        const T* qg = static_cast<const T*>(a.q) + (lb * a.hq + (size_t)g * a.group) * D;
#pragma unroll
        for (int h = 0; h < GP; ++h)
#pragma unroll
            for (int c = 0; c < CPL; ++c) {
                if (h < a.group)
                    qv[h][c] = *reinterpret_cast<const chunk_t*>(qg + h * D + (p + c * LPR) * EPC);
                else
                    qv[h][c] = chunk_t{};
            }
    }

    // K rows and positions are read with raw buffer loads over the range's rows: 32-bit lane offsets with
    // immediate row/chunk offsets, and reads past the range return zero instead of needing a clamp (those
    // logits are masked).  Loads are unconditional, so the compiler keeps the next iterations' loads in flight
    // while the current one is reduced.  The position of the row this lane will own comes with the same batch
    // (it decides the recency bias).
    static constexpr int kRowBytes = D * (int)sizeof(T);
    __device__ void load(__amdgpu_buffer_rsrc_t krs, __amdgpu_buffer_rsrc_t prs, int row0, int it,
                         chunk_t (&dst)[RPG][CPL], int& pdst) const {
        const int base = row0 + it * RPI + wave * RPW + grp;
        const int off = base * kRowBytes + p * 16;
#pragma unroll
        for (int k = 0; k < RPG; ++k)
#pragma unroll
            for (int c = 0; c < CPL; ++c)
                dst[k][c] = __builtin_bit_cast(
                    chunk_t, __builtin_amdgcn_raw_buffer_load_b128(krs, off + k * NG * kRowBytes + c * LPR * 16, 0,
                                                                   IKV_NT_LOADS ? kNonTemporal : 0));
        pdst = (int)__builtin_amdgcn_raw_buffer_load_b32(prs, (base + kk * NG) * 4, 0, 0);
    }

    // Unit u = the RPW consecutive rows [u * RPW, (u + 1) * RPW) one wave covers in one step.
    __device__ int unit_row(int u) const { return u * RPW + kk * NG + grp; }
    // This lane's chunks of the unit's rows: row u * RPW + k * NG + grp for k < RPG, chunks p + c * LPR.
    __device__ void load_rows(__amdgpu_buffer_rsrc_t rs, int u, chunk_t (&dst)[RPG][CPL]) const {
        const int off = (u * RPW + grp) * kRowBytes + p * 16;
#pragma unroll
        for (int k = 0; k < RPG; ++k)
#pragma unroll
            for (int c = 0; c < CPL; ++c)
                dst[k][c] = __builtin_bit_cast(
                    chunk_t, __builtin_amdgcn_raw_buffer_load_b128(rs, off + k * NG * kRowBytes + c * LPR * 16, 0,
                                                                   IKV_NT_LOADS ? kNonTemporal : 0));
    }
    __device__ void load_unit(__amdgpu_buffer_rsrc_t krs, __amdgpu_buffer_rsrc_t prs, int u, chunk_t (&dst)[RPG][CPL],
                              int& pdst) const {
        load_rows(krs, u, dst);
        pdst = (int)__builtin_amdgcn_raw_buffer_load_b32(prs, unit_row(u) * 4, 0, 0);
    }

    // This lane's chunks of one row (the row's 16-byte chunks p + c * LPR), e.g. the step's newcomer.
    __device__ void load_row(const T* row, chunk_t (&dst)[CPL]) const {
#pragma unroll
        for (int c = 0; c < CPL; ++c) dst[c] = *reinterpret_cast<const chunk_t*>(row + (p + c * LPR) * EPC);
    }
    // Replaces row `row` of unit u in this lane's buffers by `src` (the lanes that hold chunks of it) and its
    // position by posv (the lanes that own it after the reduce-scatter).
    __device__ void put_row(chunk_t (&dst)[RPG][CPL], int& pdst, const chunk_t (&src)[CPL], int posv, int u,
                            int row) const {
#pragma unroll
        for (int k = 0; k < RPG; ++k) {
            const bool here = u * RPW + k * NG + grp == row;
#pragma unroll
            for (int c = 0; c < CPL; ++c) dst[k][c] = here ? src[c] : dst[k][c];
        }
        if (unit_row(u) == row) pdst = posv;
    }

    // Logit of the (row, head) this lane owns for one iteration; -inf when masked (a padded head, or a row
    // past the end of the range).
    __device__ float logit(const ScoreArgs& a, const chunk_t (&kb)[RPG][CPL], const chunk_t (&qv)[GP][CPL],
                           int posv, int row, int row_end) const {
        float v[LPR];
#pragma unroll
        for (int k = 0; k < RPG; ++k)
#pragma unroll
            for (int h = 0; h < GP; ++h) {
                float acc = 0.0f;
#pragma unroll
                for (int c = 0; c < CPL; ++c) acc = E::dot(kb[k][c], qv[h][c], acc);
                v[k * GP + h] = acc;
            }
        const float dotv = reduce_scatter<LPR>(v, p);
        const float z = fmaf(dotv, a.scale, posv >= a.recent_from ? a.bias : 0.0f);
        return (row < row_end && hh < a.group) ? z : -INFINITY;
    }
};

#ifndef IKV_EPI_UNROLL
#define IKV_EPI_UNROLL 8
#endif
constexpr int kEpi = IKV_EPI_UNROLL;  // epilogue LDS reads kept in flight per lane

}  // namespace
}  // namespace ikv
