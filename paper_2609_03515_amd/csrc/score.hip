// Last-query attention scoring (Eq. 1 with GQA-shared KV heads) for gfx950.
//
// The work is a matrix-vector product per (layer, sequence, KV head) slab: every cached key row meets the G
// query heads of its group.  It is bound by the HBM stream of K (2G flop per 2-byte element).  Small groups
// run on the vector ALUs with packed bf16 dot products; padded groups of 8 and 16 over bf16 keys take the
// logits from the matrix cores instead (KUnit in stream_lane.h), whose result lands in the same LDS layout.
//
// Lane layout (vector form): a K row of d elements is LPR 16-byte chunks, one per lane of an aligned LPR-lane group (16 for
// d = 128 bf16 / d = 64 f32, 8 for d = 64 bf16); a wave load instruction therefore covers 64/LPR consecutive
// rows, 1 KiB contiguous.  Each lane handles RPG = LPR / GP rows per iteration (GP = group size rounded up to
// a power of two), producing RPG * GP = LPR partial dot products; a DPP reduce-scatter over the group leaves
// each lane with one complete (row, head) logit.
//
// One workgroup per slab keeps the slab's logits in LDS; after the per-head (max, sum) reduction it writes
// r(row) = sum over the group's heads of exp(z - max) / sum.  Slabs too long for one workgroup's LDS (long
// first steps) are scored in chunks that exchange their softmax statistics (split.hip); where the exchange
// words would not fit, by the attention kernel's K pass (attend.hip), which writes logits and per-chunk
// (max, sum), combined by the finish kernel below.
#include <algorithm>

#include "stream_lane.h"

namespace ikv {
namespace {

// Work items: `merge` consecutive KV heads (slabs) of one (layer, sequence), scored in turn, their group sums
// added in LDS (in KV-head order) and written once: one row of r per item.  A workgroup takes items
// blockIdx.x, blockIdx.x + gridDim.x, ... (one item when the grid covers them); the next slab's first loads
// are issued before each slab's epilogue.  Each slab is cut into units of RPW rows; waves claim units from an LDS counter when they issue
// the units' loads, so a wave whose loads come back late simply processes fewer units instead of holding the
// whole workgroup at the barrier (with a static split the last wave finished ~40% after the first).  Logits
// are stored per unit; after a barrier the epilogue walks the units in a fixed pattern.
// The multi-slab variant's LDS also holds the item's sums, so it runs fewer workgroups per CU: it asks for at
// most the waves of two workgroups per SIMD, which leaves it the registers of the slab loop.
template <typename T, int D, int GP, bool kMulti>
constexpr int score_waves_per_eu() {
    constexpr int w = Geometry<T, D, GP>::kMinWavesLds;
    return kMulti && w > 2 * kWaves / 4 ? 2 * kWaves / 4 : w;
}

// K units in flight per wave: three in the multi-slab form over bf16 keys when a lane's share of a unit is at
// most four 16-byte chunks and the logits are the vector form (8B steady step, alternating builds in one
// process: 261.6 against 264.0 us, within the register budget of two workgroups per CU), else the default two
// (the matrix-core form measured no faster with three; the one-slab form runs three workgroups per CU, and the
// float32 forms would leave that budget).
template <typename T, int D, int GP, bool kMulti>
constexpr int score_nbuf() {
    using G = Geometry<T, D, GP>;
    return (IKV_NBUF == 0 && kMulti && std::is_same<T, bf16_t>::value && !use_mfma<T, D, GP>() &&
            G::kRpg * G::kCpl <= 4)
               ? 3
               : G::kNbufLds;
}

// kVN (multi-slab, vector-form logits only): VNorm (Sec. 5.1) applied to each slab's group sums before they are
// added into the item's sums: the sum of row i is multiplied by |v_i| / mean_j |v_j| over the slab's n rows
// (factor 1 when all norms are zero).  The norms come from the caller's value-norm cache, read with the K rows
// (each owned row's norm with its position), staged in LDS beside the item sums; the newcomer's (row n - 1, V
// not cached yet) is computed from v_new with the same arithmetic as the cache's.  The mean is summed in the
// epilogue in a fixed order (each thread its rows, then the wave, then the waves in order).
template <typename T, int D, int GP, bool kMulti, bool kVN = false>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(score_waves_per_eu<T, D, GP, kMulti>())))
void score_lds_kernel(ScoreArgs a) {
    using L = Lane<T, D, GP>;
    using KP = KUnit<T, D, GP>;
    constexpr int RPW = L::RPW;
    constexpr int kNbuf = score_nbuf<T, D, GP, kMulti>();
    static_assert(!kVN || (kMulti && !use_mfma<T, D, GP>()), "VNorm is fused into the multi-slab vector form");

    extern __shared__ float zs[];
    __shared__ float red_m[kWaves][GP], red_s[kWaves][GP], red_n[kVN ? kWaves : 1];
    __shared__ int next_unit[2];  // claim counters of the slab being streamed and of the next one

    const L ln;
    const KP kp;
    const int merge = kMulti ? a.merge : 1;
    const int blocks = a.hkv / merge;  // items per (layer, sequence)
    const int items = a.layers * a.batch * blocks;
    const int nslab = kMulti ? (items - (int)blockIdx.x + (int)gridDim.x - 1) / (int)gridDim.x * merge : 1;
    // global slab index (lb * hkv + g) of this workgroup's si-th slab; items are lb * blocks + block
    auto slab_at = [&](int si) { return ((int)blockIdx.x + si / merge * (int)gridDim.x) * merge + si % merge; };
    const int n = a.n;
    const int nunits = (n + RPW - 1) / RPW;      // LDS blocks of logits
    const int nku = (n + KP::kRows - 1) / KP::kRows;  // claimed units of the K pass
    // item sums after the logits (sized by the plan: the logits' units rounded up to whole iterations), then
    // with kVN the slab's value norms (as many words)
    float* racc = zs + (size_t)((nunits + kWaves - 1) / kWaves) * kThreads;
    float* zn = racc + (size_t)((nunits + kWaves - 1) / kWaves) * kWaves * RPW;
    // with the newcomer given apart, rows [0, n - 1) come from the cache and row n - 1 is substituted into the
    // buffers of its unit before its logits are taken (the same arithmetic as a cached row)
    const bool has_new = a.k_new != nullptr;
    const int cached = n - (has_new ? 1 : 0);
    const int unit_new = has_new ? (n - 1) / KP::kRows : -1;
    auto p_rsrc = [&](int sidx) {
        return raw_rsrc(a.pos + (size_t)(sidx / a.hkv % a.batch) * a.cap, cached * 4);
    };
    auto k_rsrc = [&](int sidx) {
        return raw_rsrc(static_cast<const T*>(a.k) + (size_t)sidx * a.cap * D, cached * L::kRowBytes);
    };
    auto new_row = [&](int sidx) { return static_cast<const T*>(a.k_new) + (size_t)sidx * D; };
    auto n_rsrc = [&](int sidx) { return raw_rsrc(a.vn_cache + (size_t)sidx * a.cap, kVN ? cached * 4 : 0); };
    typename KP::row_t vn;  // kVN: the newcomer's V row (this lane's chunks)
    auto load_slab_consts = [&](int sidx, typename KP::q_t& qv, typename KP::row_t& kn) {
        kp.load_q(a, (size_t)(sidx / a.hkv), sidx % a.hkv, qv);
        if (has_new) kp.load_row(new_row(sidx), kn);
        if (kVN && has_new) kp.load_row(static_cast<const T*>(a.v_new) + (size_t)sidx * D, vn);
    };

    if (threadIdx.x < 2) next_unit[threadIdx.x] = 0;
    int sidx = slab_at(0);
    __amdgpu_buffer_rsrc_t krs = k_rsrc(sidx), prs = p_rsrc(sidx), nrs = n_rsrc(sidx);
    typename KP::q_t qv;
    typename KP::row_t kn;
    load_slab_consts(sidx, qv, kn);
    __syncthreads();
    auto claim = [&](int si) -> int {
        int u = 0;
        if (ln.lane == 0) u = atomicAdd(&next_unit[si & 1], 1);
        return __builtin_amdgcn_readfirstlane(u);
    };

    // stream: claim a unit, issue its loads kNbuf-1 units ahead of the one being reduced.  Loads are issued on
    // every path (claims past the end read zeros), so the wait before a reduction covers only its own buffer.
    typename KP::buf_t kbuf[kNbuf];
    int pbuf[kNbuf], ubuf[kNbuf];
    float nbuf[kNbuf];  // kVN: the value norm of the row this lane owns in each buffered unit
    auto load_unit = [&](int slot) {
        kp.load(krs, prs, ubuf[slot], kbuf[slot], pbuf[slot]);
        if constexpr (kVN)
            nbuf[slot] = __builtin_bit_cast(
                float, __builtin_amdgcn_raw_buffer_load_b32(nrs, ln.unit_row(ubuf[slot]) * 4, 0, 0));
    };
    auto prime = [&](int si) {
#pragma unroll
        for (int j = 0; j < kNbuf - 1; ++j) {
            ubuf[j] = claim(si);
            load_unit(j);
        }
    };
    prime(0);
    for (int si = 0; si < nslab; ++si) {
        const int gi = si % merge;  // position of the slab in its item
        typename KP::max_t mk = kp.max_init();
        bool more = true;
        while (more) {
#pragma unroll
            for (int j = 0; j < kNbuf; ++j) {
                const int slot = (j + kNbuf - 1) % kNbuf;
                ubuf[slot] = claim(si);
                load_unit(slot);
                if (more && ubuf[j] < nku) {
                    if (ubuf[j] == unit_new) kp.put_row(kbuf[j], pbuf[j], kn, a.new_pos, unit_new, n - 1);
                    kp.logits(a, kbuf[j], qv, pbuf[j], ubuf[j], n, zs, mk);
                    if constexpr (kVN) {
                        float nv = nbuf[j];
                        if (ubuf[j] == unit_new) {  // (every lane: the norm is a sum over the row's lane group)
                            const float vnew = row_norm_lanes<T, L::LPR, L::CPL>(vn);
                            if (ln.unit_row(ubuf[j]) == n - 1) nv = vnew;
                        }
                        const int row = ln.unit_row(ubuf[j]);
                        if (ln.hh == 0 && row < n) zn[row] = nv;
                    }
                } else {
                    more = false;  // claims only grow: every later unit of this wave is past the end too
                }
            }
        }
        const int item = slab_at(si) / merge;
        if (si + 1 < nslab) {  // the next slab's first loads overlap this slab's epilogue
            sidx = slab_at(si + 1);
            krs = k_rsrc(sidx);
            prs = p_rsrc(sidx);
            nrs = n_rsrc(sidx);
            prime(si + 1);
        }

        // epilogue: per-head softmax statistics, then normalised group sums.  Thread (wave w, lane) visits
        // units w, w + kWaves, ...; a lane's head is the same in every unit.
        float* zl = zs + ln.wave * kWave + ln.lane;
        constexpr int kStep = kWaves * kWave;  // LDS words between a thread's consecutive units
        const int mine = nunits > ln.wave ? (nunits - ln.wave + kWaves - 1) / kWaves : 0;
        kp.publish_max(mk, red_m[ln.wave]);
        __syncthreads();
        // every wave has left this slab's claims: its counter is free for the slab after next (primed only
        // after the barrier that ends this epilogue)
        if (threadIdx.x == 0) next_unit[si & 1] = 0;
        float m = red_m[0][ln.hh];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) m = fmaxf(m, red_m[w][ln.hh]);
        auto expo = [&](float z) { return z == -INFINITY ? 0.0f : __expf(z - m); };
        float ssum = 0.0f;
        int i = 0;
        for (; i + kEpi <= mine; i += kEpi) {
            float e[kEpi];
#pragma unroll
            for (int v = 0; v < kEpi; ++v) e[v] = zl[(i + v) * kStep];
#pragma unroll
            for (int v = 0; v < kEpi; ++v) {
                e[v] = expo(e[v]);
                ssum += e[v];
                zl[(i + v) * kStep] = e[v];
            }
        }
        for (; i < mine; ++i) {
            const float e = expo(zl[i * kStep]);
            ssum += e;
            zl[i * kStep] = e;
        }
#pragma unroll
        for (int o = GP; o < kWave; o <<= 1) ssum += __shfl_xor(ssum, o, kWave);
        if (ln.lane < GP) red_s[ln.wave][ln.lane] = ssum;
        const int row_in = ln.kk * L::NG + ln.grp;  // this lane's row inside a unit
        if constexpr (kVN) {  // the slab's norm sum: a lane per row (hh = 0) over its rows, the wave, the waves
            float nsum = 0.0f;
            if (ln.hh == 0)
                for (int u = 0; u < mine; ++u) {
                    const int row = (ln.wave + u * kWaves) * RPW + row_in;
                    if (row < n) nsum += zn[row];
                }
            nsum = wave_sum(nsum);
            if (ln.lane == 0) red_n[ln.wave] = nsum;
        }
        __syncthreads();
        float inv_mean = 0.0f;  // kVN: n / (sum of the norms), 0 when every norm is zero (factor 1)
        if constexpr (kVN) {
            float t = red_n[0];
#pragma unroll
            for (int w = 1; w < kWaves; ++w) t += red_n[w];
            inv_mean = t > 0.0f ? (float)n / t : 0.0f;
        }
        // VNorm factor of row `row` of this slab (rows past n hold no norm: their sums are zero)
        auto vfactor = [&](int row) { return (row < n && inv_mean > 0.0f) ? zn[row] * inv_mean : 1.0f; };
        float tot = red_s[0][ln.hh];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) tot += red_s[w][ln.hh];
        const float inv = tot > 0.0f ? 1.0f / tot : 0.0f;
        auto prob = [&](float e) { return e * inv; };
        // group sum of the normalised probabilities of each row.  One slab per workgroup: staged by one lane per
        // row in the first RPW words of the row's unit block (only this wave reads that block, and it has
        // already read the words) for the coalesced store below.  Several: added to the row's item sum.
        static_assert(RPW % 4 == 0, "the coalesced store moves 4 rows at a time");
        auto emit = [&](int unit, float sum) {
            if (ln.hh == 0) {
                const int row = ln.kk * L::NG + ln.grp;
                if (!kMulti) {
                    zs[unit * kWave + row] = sum;
                } else {
                    if constexpr (kVN) sum *= vfactor(unit * RPW + row);
                    float* acc = racc + unit * RPW + row;
                    *acc = gi == 0 ? sum : *acc + sum;
                }
            }
        };
        // kEpi units at a time: the emitting lanes read the item sums of all of them before adding and storing
        // (one at a time, each read-add-store waited for its own LDS round trip: 2.5 of the epilogue's 5.4 us
        // at the 8B step)
        i = 0;
        for (; i + kEpi <= mine; i += kEpi) {
            float e[kEpi];
#pragma unroll
            for (int v = 0; v < kEpi; ++v) e[v] = zl[(i + v) * kStep];
#pragma unroll
            for (int v = 0; v < kEpi; ++v) e[v] = group_allsum<GP>(prob(e[v]));
            if (ln.hh == 0) {
                if constexpr (!kMulti) {
#pragma unroll
                    for (int v = 0; v < kEpi; ++v) zs[(ln.wave + (i + v) * kWaves) * kWave + row_in] = e[v];
                } else {
                    float* acc = racc + (ln.wave + i * kWaves) * RPW + row_in;  // units kWaves apart
                    if constexpr (kVN) {
#pragma unroll
                        for (int v = 0; v < kEpi; ++v) e[v] *= vfactor((ln.wave + (i + v) * kWaves) * RPW + row_in);
                    }
                    if (gi != 0) {
                        float old[kEpi];
#pragma unroll
                        for (int v = 0; v < kEpi; ++v) old[v] = acc[v * kWaves * RPW];
#pragma unroll
                        for (int v = 0; v < kEpi; ++v) e[v] = old[v] + e[v];
                    }
#pragma unroll
                    for (int v = 0; v < kEpi; ++v) acc[v * kWaves * RPW] = e[v];
                }
            }
        }
        for (; i < mine; ++i) emit(ln.wave + i * kWaves, group_allsum<GP>(prob(zl[i * kStep])));
        __syncthreads();  // also: every read of this slab's logits is done before the next slab's K pass
        if (gi == merge - 1) {
            // the item is complete: its row of r.  Rows [4j, 4j + 4) lie in one unit (RPW is a multiple of 4);
            // rows up to the padded stride are scratch.  The next item's sums are written only after the next
            // epilogue's first barrier, when every thread has issued these stores.
            const __amdgpu_buffer_rsrc_t rrs = raw_rsrc(a.r + (size_t)item * a.n_stride, a.n_stride * 4);
            for (int j = threadIdx.x; j * 4 < n; j += kThreads) {
                const int row = j * 4;
                const float* src = !kMulti ? &zs[(row / RPW) * kWave + row % RPW] : &racc[row];
                store_stream(rrs, row * 4, *reinterpret_cast<const f32x4*>(src));
            }
        }
        if (si + 1 < nslab) load_slab_consts(sidx, qv, kn);
    }
}

// Combine the split partials per head and emit r(row) = sum_{h in group} exp(z_h - M_h) / S_h.  A workgroup
// covers kFinishRows rows of one (layer, sequence, KV head): each thread handles 4 consecutive rows per pass
// with 16-byte loads (logit rows are padded to a multiple of 64).
constexpr int kFinishThreads = 256;
constexpr int kFinishRows = kFinishThreads * 4 * 2;

__global__ __launch_bounds__(kFinishThreads) void split_finish_kernel(ScoreArgs a) {
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
    const float* zb = a.z + ((size_t)lb * a.hq + (size_t)g * a.group) * a.n_stride;
    float* rb = a.r + ((size_t)lb * a.hkv + g) * a.n_stride;
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
        const int row = blockIdx.x * kFinishRows + (pass * kFinishThreads + threadIdx.x) * 4;
        if (row >= a.n) continue;
        f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
        for (int h = 0; h < a.group; ++h) {
            const f32x4 z = *reinterpret_cast<const f32x4*>(zb + (size_t)h * a.n_stride + row);
            const float m = mh[h], inv = ih[h];
            acc.x += __expf(z.x - m) * inv;
            acc.y += __expf(z.y - m) * inv;
            acc.z += __expf(z.z - m) * inv;
            acc.w += __expf(z.w - m) * inv;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (row + j < a.n) rb[row + j] = acc[j];
    }
}

template <typename T, int D, int GP>
hipError_t launch_lds(const ScorePlan& plan, const ScoreArgs& a, hipStream_t s) {
    const int items = a.layers * a.batch * (a.hkv / a.merge);
    const bool multi = a.merge > 1 || (plan.grid > 0 && plan.grid < items);
    auto kern = multi ? score_lds_kernel<T, D, GP, true> : score_lds_kernel<T, D, GP, false>;
    int which = multi ? 1 : 0;
    if (a.vn_cache) {  // VNorm fused: multi-slab vector form only (the planner's choice, checked again here)
        if constexpr (use_mfma<T, D, GP>()) {
            return hipErrorInvalidValue;
        } else {
            if (!multi) return hipErrorInvalidValue;
            kern = score_lds_kernel<T, D, GP, true, true>;
            which = 2;
        }
    }
    if (plan.lds_bytes > 64 * 1024) {
        static std::atomic<bool> raised[3][kMaxDevices];
        const hipError_t e = raise_lds_limit(reinterpret_cast<const void*>(kern), raised[which]);
        if (e != hipSuccess) return e;
    }
    const int grid = plan.grid > 0 && plan.grid < items ? plan.grid : items;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kThreads), plan.lds_bytes, s, a);
    return hipGetLastError();
}

template <typename T, int D, int GP>
hipError_t launch_gp(const ScorePlan& plan, const ScoreArgs& a, hipStream_t s) {
    if constexpr (Geometry<T, D, 1>::kChunks < GP) {
        return hipErrorInvalidValue;
    } else {
        if (!plan.split) return launch_lds<T, D, GP>(plan, a, s);
        return hipErrorInvalidValue;  // long slabs are scored in chunks (launch_score_chunks)
    }
}

// Workgroups of the single-slab (kMulti false) or multi-slab variant one CU holds by its registers (0 when
// the query fails); cached per instance and device (atomics: concurrent first calls store the same value).
template <typename T, int D, int GP, bool kMulti>
int kernel_occupancy() {
    if constexpr (Geometry<T, D, 1>::kChunks < GP) {
        return 0;
    } else {
        static std::atomic<int> cached[kMaxDevices];  // occupancy + 1; 0 = not queried yet
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) dev = -1;
        if (dev >= 0) {
            const int c = cached[dev].load(std::memory_order_relaxed);
            if (c > 0) return c - 1;
        }
        int v = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&v, score_lds_kernel<T, D, GP, kMulti>, kThreads, 0) !=
            hipSuccess)
            v = 0;
        if (dev >= 0) cached[dev].store(v + 1, std::memory_order_relaxed);
        return v;
    }
}

template <typename T, int D>
int occupancy_d(int gp, bool multi) {
    switch (gp) {
        case 1: return multi ? kernel_occupancy<T, D, 1, true>() : kernel_occupancy<T, D, 1, false>();
        case 2: return multi ? kernel_occupancy<T, D, 2, true>() : kernel_occupancy<T, D, 2, false>();
        case 4: return multi ? kernel_occupancy<T, D, 4, true>() : kernel_occupancy<T, D, 4, false>();
        case 8: return multi ? kernel_occupancy<T, D, 8, true>() : kernel_occupancy<T, D, 8, false>();
        case 16: return multi ? kernel_occupancy<T, D, 16, true>() : kernel_occupancy<T, D, 16, false>();
        default: return 0;
    }
}

int kernel_occupancy(int dtype, int head_dim, int gp, bool multi) {
    if (dtype == 0) return head_dim == 64 ? occupancy_d<float, 64>(gp, multi) : occupancy_d<float, 128>(gp, multi);
    return head_dim == 64 ? occupancy_d<bf16_t, 64>(gp, multi) : occupancy_d<bf16_t, 128>(gp, multi);
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

int device_cus() {
    static std::atomic<int> cached[kMaxDevices];  // CU count + 1; 0 = not queried yet
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 0;
    if (dev < kMaxDevices) {
        const int c = cached[dev].load(std::memory_order_relaxed);
        if (c > 0) return c - 1;
    }
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) return 0;
    if (dev < kMaxDevices) cached[dev].store(cus + 1, std::memory_order_relaxed);
    return cus;
}

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
    const size_t lds = (size_t)nit * kThreads * sizeof(float);
    if (lds <= kFastLdsMax) {
        plan->split = false;
        plan->merge = 1;
        plan->chunk_rows = nit * rpi;
        plan->nchunk = 1;
        plan->lds_bytes = lds;
    } else {  // scored in chunks, planned by attend_plan
        plan->split = true;
        plan->merge = 1;
        plan->chunk_rows = 0;
        plan->nchunk = 0;
        plan->lds_bytes = 0;
    }
    plan->grid = 0;
    return true;
}

// Schedule of the LDS-resident scorer: how many consecutive KV heads of one (layer, sequence) one workgroup
// scores in turn (merge m, a divisor of hkv up to kMaxMerge; `forced` > 0: that one), one item of m slabs per
// workgroup.  The hardware hands items to CUs as slots free up, so the busiest CU streams
// ceil(items / CUs) x m slabs: the cost to minimise.  Ties go to (1) two or more workgroups per CU (one hides
// less latency) and (2) the larger merge: the group sums written while K still streams cost far more than
// their bytes, and a multi-slab workgroup issues the next slab's first loads before each epilogue.  Measured at
// the 8B steady step (2,048 slabs, all costs 8): m = 4 285.5 us, m = 2 291.7, m = 8 (one workgroup per CU)
// 295.0, m = 1 302.8; at the Qwen-shaped step (3,584 slabs): m = 2 (cost 14) 327 us, m = 1 (14) 347, m = 4
// (16) 347.
int score_merge(ScorePlan* plan, int dtype, int head_dim, int hkv, int lb_count, int forced, bool vnorm) {
    plan->merge = 1;
    plan->grid = 0;
    if (plan->split) return 1;
    // an item's sums (and with VNorm fused its slab's value norms)
    const size_t racc = (size_t)plan->chunk_rows * sizeof(float) * (vnorm ? 2 : 1);
    const size_t lds1 = plan->lds_bytes, ldsm = lds1 + racc;
    int best = 1;
    if (forced > 0) {
        best = forced;
    } else {
        const int cus = device_cus();
        const int occ1 = kernel_occupancy(dtype, head_dim, plan->group_pad, false);
        const int occm = ldsm <= kFastLdsMax ? kernel_occupancy(dtype, head_dim, plan->group_pad, true) : 0;
        if (occ1 < 1 || cus < 1) return 1;
        long best_cost = -1;
        bool best_conc = false;
        for (int m = 1; m <= kMaxMerge && m <= hkv; ++m) {
            if (hkv % m || (m > 1 && occm < 1)) continue;
            const long items = (long)lb_count * (hkv / m);
            const long per_cu = m == 1 ? std::min<long>((long)(kLdsPerCu / lds1), occ1)
                                       : std::min<long>((long)(kLdsPerCu / ldsm), occm);
            const long on_cu = (items + cus - 1) / cus;  // items of the busiest CU
            const long cost = on_cu * m;
            const bool conc = std::min(per_cu, on_cu) >= 2;
            if (best_cost < 0 || cost < best_cost || (cost == best_cost && conc >= best_conc)) {
                best_cost = cost;
                best_conc = conc;
                best = m;
            }
        }
    }
    if (best > 1 && ldsm > kFastLdsMax) best = 1;  // the item sums do not fit beside the logits
    plan->merge = best;
    if (best > 1) plan->lds_bytes = ldsm;
    return best;
}

bool score_vnorm_fusable(int dtype, int head_dim, int group_pad) {
    return !(dtype == 1 && (group_pad == 8 || group_pad == 16) && head_dim * 2 / 16 >= group_pad);
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
    dim3 grid((a.n + kFinishRows - 1) / kFinishRows, a.hkv, a.layers * a.batch);
    hipLaunchKernelGGL(split_finish_kernel, grid, dim3(kFinishThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace ikv
