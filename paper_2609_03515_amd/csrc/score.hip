// Last-query attention scoring (Eq. 1 with GQA-shared KV heads) for gfx950.
//
// The work is a matrix-vector product per (layer, sequence, KV head) slab: every cached key row meets the G
// query heads of its group.  It is bound by the HBM stream of K (2G flop per 2-byte element), so it runs on
// the vector ALUs with packed bf16 dot products, not on MFMA.
//
// Lane layout: a K row of d elements is LPR 16-byte chunks, one per lane of an aligned LPR-lane group (16 for
// d = 128 bf16 / d = 64 f32, 8 for d = 64 bf16); a wave load instruction therefore covers 64/LPR consecutive
// rows, 1 KiB contiguous.  Each lane handles RPG = LPR / GP rows per iteration (GP = group size rounded up to
// a power of two), producing RPG * GP = LPR partial dot products; a DPP reduce-scatter over the group leaves
// each lane with one complete (row, head) logit.  Per-lane online max/sum gives the softmax statistics.
//
// Fast path (whole slab fits in LDS): logits stay in LDS; after the per-head (max, sum) reduction the kernel
// writes r(row) = sum over the group's heads of exp(z - max) / sum.  Split path: several workgroups per slab
// write their logits and per-head partial (max, sum); a finish kernel combines them.
#include "kernels.h"
#include "kv_common.h"

namespace ikv {
namespace {

constexpr size_t kFastLdsMax = 80 * 1024;  // keep >= 2 workgroups per CU (160 KiB LDS)
constexpr int kWaves = 8;
constexpr int kSplitIters = 16;

template <typename T, int D, int GP>
struct Geometry {
    using E = Elem<T>;
    static constexpr int kEpc = E::kPerChunk;
    static constexpr int kChunks = D / kEpc;
    static constexpr int kLpr = kChunks >= 16 ? 16 : kChunks;
    static constexpr int kCpl = kChunks / kLpr;
    static constexpr int kNg = kWave / kLpr;
    static constexpr int kRpg = kLpr / GP;
    static constexpr int kRpw = kNg * kRpg;
    static constexpr int kRpi = kWaves * kRpw;
    static_assert(kRpg * GP == kLpr, "group must not exceed the lanes of a row");
};

template <typename T, int D, int GP, bool SPLIT>
__global__ __launch_bounds__(kWaves * kWave) void score_kernel(ScoreArgs a) {
    using Gm = Geometry<T, D, GP>;
    using E = Elem<T>;
    using chunk_t = typename E::chunk_t;
    constexpr int LPR = Gm::kLpr, CPL = Gm::kCpl, NG = Gm::kNg, RPG = Gm::kRpg, RPW = Gm::kRpw;
    constexpr int RPI = Gm::kRpi, EPC = Gm::kEpc;

    extern __shared__ float zs[];
    __shared__ MaxSum red[kWaves][GP];

    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int grp = lane / LPR, p = lane % LPR;
    const int hh = p % GP, kk = p / GP;  // (head, row slot) this lane owns after the reduce-scatter

    int bid = blockIdx.x;
    int chunk = 0;
    if constexpr (SPLIT) {
        chunk = bid % a.nchunk;
        bid /= a.nchunk;
    }
    const int g = bid % a.hkv;
    bid /= a.hkv;
    const int b = bid % a.batch;
    const int l = bid / a.batch;

    const int row0 = chunk * a.chunk_rows;
    const int row_end = min(a.n, row0 + a.chunk_rows);
    const int nit = row_end > row0 ? (row_end - row0 + RPI - 1) / RPI : 0;

    const size_t slab = (size_t)(l * a.batch + b) * a.hkv + g;
    const T* kslab = static_cast<const T*>(a.k) + slab * a.cap * D;
    const T* qg = static_cast<const T*>(a.q) + ((size_t)(l * a.batch + b) * a.hq + (size_t)g * a.group) * D;
    const int* posb = a.pos + (size_t)b * a.cap;

    chunk_t qv[GP][CPL];
#pragma unroll
    for (int h = 0; h < GP; ++h)
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            if (h < a.group)
                qv[h][c] = *reinterpret_cast<const chunk_t*>(qg + h * D + (p + c * LPR) * EPC);
            else
                qv[h][c] = chunk_t{};
        }

    const int wave_row0 = row0 + wave * RPW + grp;
    auto load = [&](int it, chunk_t(&dst)[RPG][CPL]) {
        const int base = wave_row0 + it * RPI;
#pragma unroll
        for (int k = 0; k < RPG; ++k) {
            const int row = base + k * NG;
#pragma unroll
            for (int c = 0; c < CPL; ++c) {
                if (row < row_end)
                    dst[k][c] = __builtin_nontemporal_load(
                        reinterpret_cast<const chunk_t*>(kslab + (size_t)row * D + (p + c * LPR) * EPC));
                else
                    dst[k][c] = chunk_t{};
            }
        }
    };

    MaxSum ms{-INFINITY, 0.0f};
    float* zrow = nullptr;
    if constexpr (SPLIT) zrow = a.z + ((size_t)(l * a.batch + b) * a.hq + (size_t)g * a.group + hh) * a.n_stride;

    auto process = [&](int it, const chunk_t(&kb)[RPG][CPL]) {
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
        const int row = wave_row0 + it * RPI + kk * NG;
        const bool valid = (row < row_end) && (hh < a.group);
        float z = dotv * a.scale;
        if (a.bias != 0.0f && valid && posb[row] >= a.recent_from) z += a.bias;
        if (valid) {
            if (z > ms.m) {
                ms.s = ms.s * __expf(ms.m - z) + 1.0f;
                ms.m = z;
            } else {
                ms.s += __expf(z - ms.m);
            }
        }
        if constexpr (SPLIT) {
            if (valid) zrow[row] = z;
        } else {
            zs[it * (kWaves * kWave) + threadIdx.x] = valid ? z : -INFINITY;
        }
    };

    chunk_t ka[RPG][CPL], kb[RPG][CPL];
    if (nit > 0) load(0, ka);
    for (int it = 0; it < nit; it += 2) {
        if (it + 1 < nit) load(it + 1, kb);
        process(it, ka);
        if (it + 1 < nit) {
            if (it + 2 < nit) load(it + 2, ka);
            process(it + 1, kb);
        }
    }

    // per-head softmax statistics: lanes sharing a head differ in lane bits >= log2(GP)
#pragma unroll
    for (int o = GP; o < kWave; o <<= 1) {
        MaxSum other{__shfl_xor(ms.m, o, kWave), __shfl_xor(ms.s, o, kWave)};
        ms = ms_combine(ms, other);
    }
    if (lane < GP) red[wave][lane] = ms;
    __syncthreads();
    MaxSum tot = red[0][hh];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) tot = ms_combine(tot, red[w][hh]);

    if constexpr (SPLIT) {
        if (threadIdx.x < a.group)
            a.part[((size_t)(l * a.batch + b) * a.hq + (size_t)g * a.group + threadIdx.x) * a.nchunk + chunk] =
                make_float2(tot.m, tot.s);
    } else {
        const float m = tot.m;
        const float inv = tot.s > 0.0f ? 1.0f / tot.s : 0.0f;
        float* rrow = a.r + slab * a.n_stride;
        for (int it = 0; it < nit; ++it) {
            const float z = zs[it * (kWaves * kWave) + threadIdx.x];
            const float e = (z == -INFINITY) ? 0.0f : __expf(z - m) * inv;
            const float sum = group_allsum<GP>(e);
            const int row = row0 + it * RPI + wave * RPW + kk * NG + grp;
            if (hh == 0 && row < row_end) rrow[row] = sum;
        }
    }
}

// Combine the split partials per head and emit r(row) = sum_{h in group} exp(z_h - M_h) / S_h.
__global__ __launch_bounds__(256) void split_finish_kernel(ScoreArgs a) {
    __shared__ float mh[kMaxGroup], ih[kMaxGroup];
    const int g = blockIdx.y;
    const int lb = blockIdx.z;  // l * batch + b
    if (threadIdx.x < a.group) {
        const float2* pp = a.part + ((size_t)lb * a.hq + (size_t)g * a.group + threadIdx.x) * a.nchunk;
        MaxSum t{-INFINITY, 0.0f};
        for (int c = 0; c < a.nchunk; ++c) t = ms_combine(t, MaxSum{pp[c].x, pp[c].y});
        mh[threadIdx.x] = t.m;
        ih[threadIdx.x] = t.s > 0.0f ? 1.0f / t.s : 0.0f;
    }
    __syncthreads();
    const int row = blockIdx.x * blockDim.x + threadIdx.x;
    if (row >= a.n) return;
    const float* zb = a.z + ((size_t)lb * a.hq + (size_t)g * a.group) * a.n_stride + row;
    float acc = 0.0f;
    for (int h = 0; h < a.group; ++h) acc += __expf(zb[(size_t)h * a.n_stride] - mh[h]) * ih[h];
    a.r[((size_t)lb * a.hkv + g) * a.n_stride + row] = acc;
}

template <typename T, int D, int GP, bool SPLIT>
hipError_t launch_one(const ScorePlan& plan, const ScoreArgs& a, hipStream_t s) {
    auto kern = score_kernel<T, D, GP, SPLIT>;
    if (!SPLIT && plan.lds_bytes > 64 * 1024) {
        static bool raised = false;  // idempotent attribute; a benign race between threads
        if (!raised) {
            hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)kFastLdsMax);
            if (e != hipSuccess) return e;
            raised = true;
        }
    }
    hipLaunchKernelGGL(kern, dim3(plan.grid), dim3(kWaves * kWave), SPLIT ? 0 : plan.lds_bytes, s, a);
    return hipGetLastError();
}

template <typename T, int D, int GP>
hipError_t launch_gp(const ScorePlan& plan, const ScoreArgs& a, hipStream_t s) {
    if constexpr (Geometry<T, D, 1>::kLpr < GP) {
        return hipErrorInvalidValue;
    } else {
        return plan.split ? launch_one<T, D, GP, true>(plan, a, s) : launch_one<T, D, GP, false>(plan, a, s);
    }
}

template <typename T, int D>
hipError_t launch_d(const ScorePlan& plan, const ScoreArgs& a, hipStream_t s) {
    switch (plan.group_pad) {
        case 1: return launch_gp<T, D, 1>(plan, a, s);
        case 2: return launch_gp<T, D, 2>(plan, a, s);
        case 4: return launch_gp<T, D, 4>(plan, a, s);
        case 8: return launch_gp<T, D, 8>(plan, a, s);
        case 16: return launch_gp<T, D, 16>(plan, a, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

bool score_plan(int dtype, int head_dim, int group, int n, ScorePlan* plan) {
    if (group < 1 || group > kMaxGroup || n < 1) return false;
    if (head_dim != 64 && head_dim != 128) return false;
    int gp = 1;
    while (gp < group) gp <<= 1;
    const int esize = dtype == 0 ? 4 : 2;
    const int chunks = head_dim * esize / 16;
    const int lpr = chunks >= 16 ? 16 : chunks;
    if (gp > lpr) return false;
    const int rpi = kWaves * (kWave / lpr) * (lpr / gp);
    const int nit = (n + rpi - 1) / rpi;
    plan->group_pad = gp;
    plan->waves = kWaves;
    plan->rows_per_iter = rpi;
    const size_t lds = (size_t)nit * kWaves * kWave * sizeof(float);
    if (lds <= kFastLdsMax) {
        plan->split = false;
        plan->chunk_rows = nit * rpi;
        plan->nchunk = 1;
        plan->lds_bytes = lds;
    } else {
        const int target = rpi * kSplitIters;
        int nchunk = (n + target - 1) / target;
        int rows = (n + nchunk - 1) / nchunk;
        rows = (rows + rpi - 1) / rpi * rpi;
        plan->split = true;
        plan->chunk_rows = rows;
        plan->nchunk = (n + rows - 1) / rows;
        plan->lds_bytes = 0;
    }
    plan->grid = 0;
    return true;
}

hipError_t launch_score(int dtype, int head_dim, const ScorePlan& plan, const ScoreArgs& a, hipStream_t s) {
    if (dtype == 0) {
        if (head_dim == 64) return launch_d<float, 64>(plan, a, s);
        if (head_dim == 128) return launch_d<float, 128>(plan, a, s);
    } else {
        if (head_dim == 64) return launch_d<bf16_t, 64>(plan, a, s);
        if (head_dim == 128) return launch_d<bf16_t, 128>(plan, a, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_split_finish(const ScoreArgs& a, hipStream_t s) {
    dim3 grid((a.n + 255) / 256, a.hkv, a.layers * a.batch);
    hipLaunchKernelGGL(split_finish_kernel, grid, dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace ikv
