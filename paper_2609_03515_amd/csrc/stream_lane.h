// Streaming machinery shared by the scorer and the fused decode-attention kernels: one workgroup of 8 waves
// streams rows of a (layer, sequence, KV head) slab with raw buffer loads; a K row is split into 16-byte
// chunks over an aligned group of LPR lanes, each lane accumulates the partial dot products of RPG rows with
// the GP (padded) query heads of its group, and a DPP reduce-scatter leaves each lane with one full
// (row, head) logit.
#pragma once

#include <atomic>
#include <type_traits>

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

// Host side: raises a kernel's dynamic-LDS limit to kFastLdsMax once per device.  `done` is the kernel's own
// flag array; concurrent first calls may both set the (idempotent) attribute, and the flags are atomics.
constexpr int kMaxDevices = 64;
inline hipError_t raise_lds_limit(const void* kern, std::atomic<bool> (&done)[kMaxDevices]) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) dev = -1;
    if (dev >= 0 && done[dev].load(std::memory_order_acquire)) return hipSuccess;
    const hipError_t e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kFastLdsMax);
    if (e == hipSuccess && dev >= 0) done[dev].store(true, std::memory_order_release);
    return e;
}

// Raw buffer resource over `bytes` bytes at `base` (reads at offsets >= bytes return zero).  A resource is
// wave-uniform: base and size are taken from the wave's first active lane, so every caller passes the same
// values in all lanes (per-lane differences go into the offsets).  Without the explicit broadcast a value the
// compiler happens to compute in vector registers (e.g. a size derived from a uniform boolean) makes it wrap
// every buffer access in a loop over the distinct resources of the wave.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_rsrc(const void* base, int bytes) {
    const uint64_t p = reinterpret_cast<uint64_t>(base);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)p);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(p >> 32));
    void* b = reinterpret_cast<void*>(((uint64_t)hi << 32) | lo);
    return __builtin_amdgcn_make_buffer_rsrc(b, (short)0, __builtin_amdgcn_readfirstlane(bytes), kRsrcConfig);
}

// 16- and 4-byte stores at byte offset `off` of a raw buffer resource, with the streaming-result cache policy.
__device__ __forceinline__ void store_stream(__amdgpu_buffer_rsrc_t rs, int off, const f32x4& v) {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), rs, off, 0, kStoreStream);
}
__device__ __forceinline__ void store_stream(__amdgpu_buffer_rsrc_t rs, int off, float v) {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), rs, off, 0, kStoreStream);
}
// The same 4-byte store by address, for destinations that differ between the lanes of a wave (a resource must
// be wave-uniform): a relaxed device-scope store, which carries the same device-scope cache policy.
__device__ __forceinline__ void store_stream_at(float* p, float v) {
    __hip_atomic_store(reinterpret_cast<uint32_t*>(p), __builtin_bit_cast(uint32_t, v), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}

template <typename T, int D, int GP>
struct Geometry {
    using E = Elem<T>;
    static constexpr int kEpc = E::kPerChunk;
    static constexpr int kChunks = D / kEpc;
    // Lanes per K row: IKV_LPR (16: one 16-byte chunk each for d = 128 bf16, a wave load covers 1 KiB of
    // consecutive rows), at least the padded group (the reduce-scatter leaves one (row, head) per lane), at
    // most the row's chunks.  A padded group of 8 over rows of at most 16 chunks takes 8 lanes instead (two
    // chunks each, every load still on whole 128-byte lines): with vector dot products the 3-step
    // reduce-scatter of 8 values took the Qwen-shaped steady step from 347 to 320 us, and with the matrix-core
    // logits (which keep this layout) the step is still ~0.4% and step 1 ~3% faster than with 16 lanes.
    // Group 4 gains nothing from it and the attention's V pass (two chunks of accumulators per lane) loses
    // 5-13%.
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

typedef __bf16 __attribute__((ext_vector_type(8))) bf16x8;

// Logits of the K pass, one claimed unit of rows at a time, for the G heads that share a KV head.  Two forms
// leave the same LDS layout (block u of 64 words holds the logits of rows [u RPW, (u + 1) RPW) in the word of
// the lane that owns each (row, head) after the reduce-scatter), so the kernels' epilogues and V passes do not
// depend on which one ran:
//  * the vector-ALU lane machinery above (units of RPW rows, one logit per lane);
//  * matrix cores, for bf16 keys with a padded group of 8 or 16: the group's query heads against 16 key rows
//    are a 16 x 16 x d product (heads past G are zero rows), D / 32 v_mfma_f32_16x16x32_bf16 per unit.  With
//    G = 7 the vector dot products cost two instructions per byte of K and left the Qwen-shaped scorer
//    partly ALU-bound (removing them saved 24 of 323 us per launch); with G = 4 they are hidden behind the
//    stream (the matrix-core form measured no faster there), so group 4 keeps the vector form.
template <typename T, int D, int GP>
constexpr bool use_mfma() {
    return std::is_same<T, bf16_t>::value && (GP == 8 || GP == 16) &&
           Geometry<T, D, 1>::kChunks >= GP;
}

template <typename T, int D, int GP, bool kMfma = use_mfma<T, D, GP>()>
struct KUnit {
    using L = Lane<T, D, GP>;
    using chunk_t = typename L::chunk_t;
    static constexpr int kRows = L::RPW;  // rows per claimed unit
    typedef chunk_t q_t[GP][L::CPL];
    typedef chunk_t buf_t[L::RPG][L::CPL];
    typedef chunk_t row_t[L::CPL];
    typedef float max_t;

    L ln;

    __device__ void load_q(const ScoreArgs& a, size_t lb, int g, q_t& qv) const { ln.load_q(a, lb, g, qv); }
    __device__ void load(__amdgpu_buffer_rsrc_t krs, __amdgpu_buffer_rsrc_t prs, int u, buf_t& dst, int& pdst) const {
        ln.load_unit(krs, prs, u, dst, pdst);
    }
    __device__ void load_row(const T* row, row_t& dst) const { ln.load_row(row, dst); }
    __device__ void put_row(buf_t& dst, int& pdst, const row_t& src, int posv, int u, int row) const {
        ln.put_row(dst, pdst, src, posv, u, row);
    }
    __device__ max_t max_init() const { return kFloor; }
    // logits of unit u (rows past row_end masked to -inf) into LDS, and the running maximum
    __device__ void logits(const ScoreArgs& a, const buf_t& kb, const q_t& qv, int posv, int u, int row_end,
                           float* zs, max_t& m) const {
        const float z = ln.logit(a, kb, qv, posv, ln.unit_row(u), row_end);
        m = fmaxf(m, z);
        zs[u * kWave + ln.lane] = z;
    }
    // the wave's per-head maxima into red[0, GP) (lanes of one head: equal lane index mod GP; steps below 16
    // stay inside a 16-lane row, the rows are combined with row swaps)
    __device__ void publish_max(max_t m, float* red) const {
#pragma unroll
        for (int o = GP; o < 16; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, kWave));
        m = rows_allmax(m);
        if (ln.lane < GP) red[ln.lane] = m;
    }
};

// Matrix-core form.  v_mfma_f32_16x16x32_bf16 operand layout (checked on the device): lane l supplies row
// l % 16 of A (a query head) and column l % 16 of B (a key row), each as 8 elements (slice l / 16) of the
// 32-element k block, and receives D[4 (l / 16) + i][l % 16] for i < 4: four heads of one row, which go to
// LDS as one 16-byte store.  MFMA kb covers the elements [32 kb, 32 kb + 32) of every row.
//
// Loading those operands directly would have every load instruction read 64 bytes of 16 rows, half of each
// 128-byte line, and the other half one instruction later: measured 14% slower than the vector form on the
// Qwen shape.  So the loads stay whole-line: load (c, v) gives lane l = 16 kq + 8 w + r (r < 8, w < 2) the
// 16 bytes 128 c + 64 w + 16 kq of row 8 v + r of the unit; the 8 lanes with equal r cover line c of that
// row.  Lane l then needs, for MFMA 2 c + w, what it loaded itself at v = w, and for MFMA 2 c + (1 - w) what
// lane l ^ 8 loaded at v = w: one DPP row_ror:8 move per dword, restricted by the bank mask to the lanes
// that take it (banks 2, 3 are the lanes with w = 1).
template <typename T, int D, int GP>
struct KUnit<T, D, GP, true> {
    using L = Lane<T, D, GP>;
    typedef u32x4 chunk_t;
    static constexpr int kLines = D * (int)sizeof(T) / 128;  // 128-byte lines per row
    static constexpr int kRows = 16;
    static_assert(L::RPW * GP == kWave && kRows % L::RPW == 0 && GP % 4 == 0, "whole LDS blocks, 4 heads per store");
    typedef chunk_t q_t[2 * kLines];
    typedef chunk_t buf_t[kLines][2];
    typedef chunk_t row_t[kLines];
    typedef f32x4 max_t;

    int col, kq, w, r;  // D column (row of the unit) / A row (head); k slice; half-line and row of the loads

    __device__ KUnit() {
        const int lane = threadIdx.x & (kWave - 1);
        col = lane % 16;
        kq = lane / 16;
        w = (lane / 8) % 2;
        r = lane % 8;
    }

    __device__ void load_q(const ScoreArgs& a, size_t lb, int g, q_t& qv) const {
        const T* qh = static_cast<const T*>(a.q) + (lb * a.hq + (size_t)g * a.group + col) * D + kq * 8;
#pragma unroll
        for (int kb = 0; kb < 2 * kLines; ++kb)
            qv[kb] = col < a.group ? *reinterpret_cast<const chunk_t*>(qh + kb * 32) : chunk_t{};
    }
    static constexpr int kRowBytes = D * (int)sizeof(T);
    __device__ void load(__amdgpu_buffer_rsrc_t krs, __amdgpu_buffer_rsrc_t prs, int u, buf_t& dst, int& pdst) const {
        const int off = (u * kRows + r) * kRowBytes + w * 64 + kq * 16;
#pragma unroll
        for (int c = 0; c < kLines; ++c)
#pragma unroll
            for (int v = 0; v < 2; ++v)
                dst[c][v] = __builtin_amdgcn_raw_buffer_load_b128(krs, off + v * 8 * kRowBytes + c * 128, 0,
                                                                  IKV_NT_LOADS ? kNonTemporal : 0);
        pdst = (int)__builtin_amdgcn_raw_buffer_load_b32(prs, (u * kRows + col) * 4, 0, 0);
    }
    // this lane's pieces of one row as the loads above would give them (the newcomer)
    __device__ void load_row(const T* row, row_t& dst) const {
#pragma unroll
        for (int c = 0; c < kLines; ++c)
            dst[c] = *reinterpret_cast<const chunk_t*>(row + c * 64 + w * 32 + kq * 8);
    }
    __device__ void put_row(buf_t& dst, int& pdst, const row_t& src, int posv, int u, int row) const {
#pragma unroll
        for (int v = 0; v < 2; ++v) {
            const bool here = u * kRows + 8 * v + r == row;
#pragma unroll
            for (int c = 0; c < kLines; ++c) dst[c][v] = here ? src[c] : dst[c][v];
        }
        pdst = u * kRows + col == row ? posv : pdst;
    }
    __device__ max_t max_init() const { return max_t{kFloor, kFloor, kFloor, kFloor}; }

    // B operand of MFMA 2 c + h from the whole-line loads of line c
    template <int BANKS>
    __device__ static chunk_t take(const chunk_t& own, const chunk_t& other) {
        chunk_t x;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            x[j] = (uint32_t)__builtin_amdgcn_update_dpp((int)own[j], (int)other[j], kRor8, 0xF, BANKS, false);
        return x;
    }
    __device__ void logits(const ScoreArgs& a, const buf_t& kb, const q_t& qv, int posv, int u, int row_end,
                           float* zs, max_t& m) const {
        f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int c = 0; c < kLines; ++c) {
            const chunk_t b0 = take<0xC>(kb[c][0], kb[c][1]);  // w = 1 lanes: lane l ^ 8's load of rows 8..15
            const chunk_t b1 = take<0x3>(kb[c][1], kb[c][0]);  // w = 0 lanes: lane l ^ 8's load of rows 0..7
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, qv[2 * c]),
                                                          __builtin_bit_cast(bf16x8, b0), acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, qv[2 * c + 1]),
                                                          __builtin_bit_cast(bf16x8, b1), acc, 0, 0, 0);
        }
        const int row = u * kRows + col;
        const int h0 = kq * 4;
        const float bias = posv >= a.recent_from ? a.bias : 0.0f;
        f32x4 z;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            z[i] = (row < row_end && h0 + i < a.group) ? fmaf(acc[i], a.scale, bias) : -INFINITY;
            m[i] = fmaxf(m[i], z[i]);
        }
        // the word of (row, head) is the one the lane that owns it in the vector form writes: block row / RPW,
        // lane (row_in_block % NG) * LPR + (row_in_block / NG) * GP + head.  Rows of the last block past row_end
        // still get their -inf; nothing past that block is written.
        const int rib = row % L::RPW;
        const int word = row / L::RPW * kWave + rib % L::NG * L::LPR + rib / L::NG * GP + h0;
        const int pad_end = (row_end + L::RPW - 1) / L::RPW * L::RPW;
        if (h0 < GP && row < pad_end) *reinterpret_cast<f32x4*>(zs + word) = z;
    }
    __device__ void publish_max(max_t m, float* red) const {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int o = 1; o < 16; o <<= 1) m[i] = fmaxf(m[i], __shfl_xor(m[i], o, kWave));
        if (col == 0 && kq * 4 < GP)
#pragma unroll
            for (int i = 0; i < 4; ++i) red[kq * 4 + i] = m[i];
    }
};

// Streams the units [0, n) a wave claims (claim() returns the next unclaimed unit, wave-uniform) with NB = 1 or
// 2 units' loads in flight: load(slot, u) issues the loads of unit u into buffer `slot` (a compile-time
// std::integral_constant), proc(slot, u) consumes them.  The loop is left as soon as a claim runs past the end,
// before any load for it is issued, so no load is still in flight when the wave moves on (a load past the
// end would return zeros, but only after the loads queued ahead of it, and the registers it writes are
// reused after the loop).  `first`: a unit claimed and, if below n, loaded into slot 0 before the call
// (NB = 2), or -1.
template <int NB, class ClaimF, class LoadF, class ProcF>
__device__ __forceinline__ void claimed_units(int n, int first, ClaimF claim, LoadF load, ProcF proc) {
    static_assert(NB == 1 || NB == 2, "one or two units in flight");
    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    if constexpr (NB == 1) {
        for (;;) {
            const int u = claim();
            if (u >= n) break;
            load(S0{}, u);
            proc(S0{}, u);
        }
    } else {
        int ua = first;
        if (ua < 0) {
            ua = claim();
            if (ua < n) load(S0{}, ua);
        }
        while (ua < n) {
            const int ub = claim();
            if (ub >= n) {
                proc(S0{}, ua);
                break;
            }
            load(S1{}, ub);
            proc(S0{}, ua);
            ua = claim();
            if (ua >= n) {
                proc(S1{}, ub);
                break;
            }
            load(S0{}, ua);
            proc(S1{}, ub);
        }
    }
}

#ifndef IKV_EPI_UNROLL
#define IKV_EPI_UNROLL 8
#endif
constexpr int kEpi = IKV_EPI_UNROLL;  // epilogue LDS reads kept in flight per lane

}  // namespace
}  // namespace ikv
