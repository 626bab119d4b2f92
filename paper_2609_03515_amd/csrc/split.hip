// Scoring of slabs too long for one workgroup's LDS (first decode steps: a 32k- or 128k-token prefill), Eq. 1
// over chunks of a slab whose logits stay in LDS.
//
// Each chunk needs the softmax statistics of the whole slab: per query head, the maximum M and the sum S of
// exp(z - M) over every chunk.  The chunks of a slab therefore exchange their own (max, sum) pairs: each pair is
// one 64-bit word (max bits high, sum bits low) written with a single device-scope atomic store, so a reader
// that sees the word sees both halves, and a chunk's sum is at least 1 (its maximum contributes exp(0)), so a
// zero word means "not written yet".  No other data crosses workgroups, so no fence is needed.  A workgroup then
// scales its chunk's exponentials by exp(m - M) / S and writes the chunk's group sums r directly: no logits
// round trip through memory.
//
// With merge > 1 a team of chunks scores the `merge` consecutive KV heads of one (layer, sequence) in
// consecutive rounds and adds their group sums in LDS (in KV-head order, as the multi-slab scorer does),
// writing one row of r per item instead of one per KV head.  Those writes, made while the rest of the grid
// streams K, had cost more than their bytes: the 8B first step with only every fourth KV head's sums written
// (a timing probe) took 3.825 instead of 3.994 ms.
//
// The grid is persistent and no larger than the workgroups the chip holds at once: workgroup w always takes
// chunk w % C of the slabs of items w / C, w / C + P, ... (P = grid / C items at a time), so the C chunks of a
// slab are consecutive workgroups that are dispatched together and only ever wait for one another.  That
// holds only while the grid has the device to itself: work of other streams or processes that holds CUs can
// keep a slab's later chunks from being dispatched while its earlier ones wait.  Every wait is therefore bounded
// (a limit of ~64-clock sleeps, about 0.1 s by default); a chunk that gives up sets its group sums to NaN
// and raises KV_FAULT_EXCHANGE_TIMEOUT in the workspace's fault word, so the failure is visible to the caller
// (kv_fault_status) instead of folding a softmax that misses part of the slab.  The exchange words are zeroed
// by a fill kernel before each launch.
#include <algorithm>

#include "stream_lane.h"

namespace ikv {
namespace {

constexpr int kMaxWords = 4;  // exchange words per lane: chunks x padded group <= 256

__device__ __forceinline__ uint64_t pack_ms(float m, float s) {
    return ((uint64_t)__float_as_uint(m) << 32) | (uint64_t)__float_as_uint(s);
}

template <typename T, int D, int GP>
constexpr int coop_waves_per_eu() {
    return Geometry<T, D, GP>::kMinWavesLds;
}

template <typename T, int D, int GP>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(coop_waves_per_eu<T, D, GP>())))
void score_coop_kernel(ScoreArgs a, uint64_t* xchg, int items_per_round, uint32_t* faults, int spin_limit) {
    using L = Lane<T, D, GP>;
    using KP = KUnit<T, D, GP>;
    constexpr int RPW = L::RPW;
    constexpr int kNbuf = Geometry<T, D, GP>::kNbufLds;

    extern __shared__ float zs[];
    __shared__ float red_m[kWaves][GP], red_s[kWaves][GP];
    __shared__ float fh[GP];
    __shared__ int next_unit[2];

    const L ln;
    const KP kp;
    const int n = a.n, C = a.nchunk;
    const int merge = a.merge;  // KV heads per item: their group sums are added, one row of r per item
    const int items = a.layers * a.batch * a.hkv / merge;
    const int cw = blockIdx.x % C;  // this workgroup's chunk of every slab it scores
    const int row0 = cw * a.chunk_rows;
    const int rows = min(a.chunk_rows, n - row0);
    const int nunits = (rows + RPW - 1) / RPW;          // LDS blocks of logits
    const int nku = (rows + KP::kRows - 1) / KP::kRows;  // claimed units of the K pass
    // merge > 1: the item's sums of this chunk's rows after the logits (units rounded up to whole iterations)
    float* racc = zs + (size_t)((nunits + kWaves - 1) / kWaves) * kThreads;
    auto k_rsrc = [&](int slab) {
        return raw_rsrc(static_cast<const T*>(a.k) + ((size_t)slab * a.cap + row0) * D, rows * L::kRowBytes);
    };
    auto p_rsrc = [&](int slab) {
        return raw_rsrc(a.pos + (size_t)(slab / a.hkv % a.batch) * a.cap + row0, rows * 4);
    };

    int item = (int)blockIdx.x / C, gi = 0;  // the item being scored and the place of its slab in it
    if (item >= items) return;
    int slab = item * merge;
    if (threadIdx.x < 2) next_unit[threadIdx.x] = 0;
    __amdgpu_buffer_rsrc_t krs = k_rsrc(slab), prs = p_rsrc(slab);
    typename KP::q_t qv;
    kp.load_q(a, (size_t)(slab / a.hkv), slab % a.hkv, qv);
    __syncthreads();
    auto claim = [&](int si) -> int {
        int u = 0;
        if (ln.lane == 0) u = atomicAdd(&next_unit[si & 1], 1);
        return __builtin_amdgcn_readfirstlane(u);
    };
    typename KP::buf_t kbuf[kNbuf];
    int pbuf[kNbuf], ubuf[kNbuf];
    auto prime = [&](int si) {
#pragma unroll
        for (int j = 0; j < kNbuf - 1; ++j) {
            ubuf[j] = claim(si);
            kp.load(krs, prs, ubuf[j], kbuf[j], pbuf[j]);
        }
    };
    prime(0);
    for (int si = 0;; ++si) {
        const int cur = slab, cur_item = item, cur_gi = gi;
        typename KP::max_t mk = kp.max_init();
        bool more = true;
        while (more) {
#pragma unroll
            for (int j = 0; j < kNbuf; ++j) {
                const int slot = (j + kNbuf - 1) % kNbuf;
                ubuf[slot] = claim(si);
                kp.load(krs, prs, ubuf[slot], kbuf[slot], pbuf[slot]);
                if (more && ubuf[j] < nku) {
                    kp.logits(a, kbuf[j], qv, pbuf[j], ubuf[j], rows, zs, mk);
                } else {
                    more = false;
                }
            }
        }
        if (++gi == merge) {
            gi = 0;
            item += items_per_round;
        }
        slab = item * merge + gi;
        const bool next = item < items;
        if (next) {  // the next slab's first loads overlap this chunk's epilogue and exchange
            krs = k_rsrc(slab);
            prs = p_rsrc(slab);
            prime(si + 1);
        }

        // the chunk's per-head maximum and sum of exponentials (exponentials kept in LDS)
        float* zl = zs + ln.wave * kWave + ln.lane;
        constexpr int kStep = kWaves * kWave;
        const int mine = nunits > ln.wave ? (nunits - ln.wave + kWaves - 1) / kWaves : 0;
        kp.publish_max(mk, red_m[ln.wave]);
        __syncthreads();
        if (threadIdx.x == 0) next_unit[si & 1] = 0;  // every wave has left this chunk's claims
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
        __syncthreads();

        // exchange (wave 0): publish this chunk's pairs, then gather every chunk's pairs (lane l holds words
        // l, l + 64, ... of the [chunk][padded head] grid, so a lane's head is l % GP) and combine them per head
        // in a fixed order (a lane's words, then butterflies over the lanes of the same head)
        uint64_t* xs = xchg + (size_t)cur * C * a.group;  // [chunk][head]
        if (ln.wave == 0) {
            // the lane index made opaque for this round: the word addresses below are recomputed here instead of
            // being hoisted out of the slab loop, whose registers they would overflow (spilled, they came back
            // from scratch memory on every round's exchange)
            int lane = ln.lane;
            asm volatile("" : "+v"(lane));
            const int h = lane % GP;
            float mh = -INFINITY;  // this chunk's statistics of head h
            if (h < a.group) {
                float sh = 0.0f;
                mh = red_m[0][h];
                sh = red_s[0][h];
                for (int w = 1; w < kWaves; ++w) {
                    mh = fmaxf(mh, red_m[w][h]);
                    sh += red_s[w][h];
                }
                if (ln.lane < GP)
                    __hip_atomic_store(xs + (size_t)cw * a.group + h, pack_ms(mh, sh), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
            }
            float cm[kMaxWords], cs[kMaxWords];
            bool done[kMaxWords];
#pragma unroll
            for (int k = 0; k < kMaxWords; ++k) {
                const int c = (lane + k * kWave) / GP;
                cm[k] = -INFINITY;
                cs[k] = 0.0f;
                done[k] = !(c < C && h < a.group);
            }
            // polls, at most spin_limit of them (0: none, every chunk gives up at once), with a sleep after each
            // unsuccessful one
            for (int spin = 0; spin < spin_limit; ++spin) {
                bool all = true;
#pragma unroll
                for (int k = 0; k < kMaxWords; ++k) {
                    if (done[k]) continue;
                    const int c = (lane + k * kWave) / GP;
                    const uint64_t v = __hip_atomic_load(xs + (size_t)c * a.group + h, __ATOMIC_RELAXED,
                                                         __HIP_MEMORY_SCOPE_AGENT);
                    if ((uint32_t)v != 0u) {
                        cm[k] = __uint_as_float((uint32_t)(v >> 32));
                        cs[k] = __uint_as_float((uint32_t)v);
                        done[k] = true;
                    } else {
                        all = false;
                    }
                }
                if (all) break;
                __builtin_amdgcn_s_sleep(1);
            }
            bool complete = true;
#pragma unroll
            for (int k = 0; k < kMaxWords; ++k) complete = complete && done[k];
            // a peer's word never arrived: report it and poison this chunk's sums rather than fold a softmax
            // that misses part of the slab (the atomic is a vector-memory instruction, as every store here)
            const bool gave_up = __builtin_amdgcn_ballot_w64(!complete) != 0;
            if (gave_up && ln.lane == 0) atomicOr(faults, kFaultExchangeTimeout);
            float M = cm[0];
#pragma unroll
            for (int k = 1; k < kMaxWords; ++k) M = fmaxf(M, cm[k]);
#pragma unroll
            for (int o = GP; o < kWave; o <<= 1) M = fmaxf(M, __shfl_xor(M, o, kWave));
            float S = 0.0f;
#pragma unroll
            for (int k = 0; k < kMaxWords; ++k)
                if (cs[k] > 0.0f) S += cs[k] * __expf(cm[k] - M);
#pragma unroll
            for (int o = GP; o < kWave; o <<= 1) S += __shfl_xor(S, o, kWave);
            if (ln.lane < GP) fh[h] = gave_up ? __builtin_nanf("") : ((h < a.group && S > 0.0f) ? __expf(mh - M) / S : 0.0f);
        }
        __syncthreads();

        // group sums of the normalised probabilities: one slab per item, staged in the first RPW words of each
        // unit's block (only this wave reads that block, and it has read the words); several, added to the
        // item's sums (kEpi units read before they are added and stored)
        const float f = fh[ln.hh];
        const int row_in = ln.kk * L::NG + ln.grp;  // this lane's row inside a unit
        auto emit = [&](int unit, float sum) {
            if (ln.hh == 0) {
                if (merge == 1) {
                    zs[unit * kWave + row_in] = sum;
                } else {
                    float* acc = racc + unit * RPW + row_in;
                    *acc = cur_gi == 0 ? sum : *acc + sum;
                }
            }
        };
        i = 0;
        for (; i + kEpi <= mine; i += kEpi) {
            float e[kEpi];
#pragma unroll
            for (int v = 0; v < kEpi; ++v) e[v] = zl[(i + v) * kStep];
#pragma unroll
            for (int v = 0; v < kEpi; ++v) e[v] = group_allsum<GP>(e[v] * f);
            if (merge == 1) {
#pragma unroll
                for (int v = 0; v < kEpi; ++v) emit(ln.wave + (i + v) * kWaves, e[v]);
            } else if (ln.hh == 0) {
                float* acc = racc + (ln.wave + i * kWaves) * RPW + row_in;  // units kWaves apart
                if (cur_gi != 0) {
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
        for (; i < mine; ++i) emit(ln.wave + i * kWaves, group_allsum<GP>(zl[i * kStep] * f));
        __syncthreads();
        if (cur_gi == merge - 1) {
            // the item's row of r for this chunk's rows: rows [4j, 4j + 4) lie in one unit; rows up to the
            // padded stride are scratch
            const __amdgpu_buffer_rsrc_t rrs =
                raw_rsrc(a.r + (size_t)cur_item * a.n_stride + row0, (a.n_stride - row0) * 4);
            int tid = threadIdx.x;
            asm volatile("" : "+v"(tid));  // (as the lane index above: recomputed, not held across the slab loop)
            for (int j = tid; j * 4 < rows; j += kThreads) {
                const int row = j * 4;
                const float* src = merge == 1 ? &zs[(row / RPW) * kWave + row % RPW] : &racc[row];
                store_stream(rrs, row * 4, *reinterpret_cast<const f32x4*>(src));
            }
        }
        if (!next) break;
        __syncthreads();  // every thread has read its staged sums before the next chunk's logits land
        kp.load_q(a, (size_t)(slab / a.hkv), slab % a.hkv, qv);
    }
}

// Zeroes the exchange words before a launch (a kernel, not a memset, so that the step can be captured).
__global__ __launch_bounds__(256) void zero_words_kernel(uint64_t* w, size_t count) {
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < count; i += (size_t)gridDim.x * 256) w[i] = 0;
}

// The workspace's fault word: copied to `out` (when non-null), then zeroed when asked (one thread).
__global__ __launch_bounds__(64) void fault_word_kernel(uint32_t* word, uint32_t* out, int clear) {
    if (threadIdx.x != 0) return;
    const uint32_t v = __hip_atomic_load(word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (out) *out = v;
    if (clear) __hip_atomic_store(word, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Polls a chunk makes before it gives up (process-wide; a test hook can lower it to force the report).
constexpr int kDefaultSpinLimit = 1 << 22;  // 64-clock sleeps: about 0.1 s, far beyond any chunk's streaming
std::atomic<int> g_spin_limit{kDefaultSpinLimit};

template <typename T, int D, int GP>
hipError_t launch_coop_gp(const ScorePlan& plan, const ScoreArgs& a, uint64_t* xchg, int grid, uint32_t* faults,
                          hipStream_t s) {
    if constexpr (Geometry<T, D, 1>::kChunks < GP) {
        return hipErrorInvalidValue;
    } else {
        auto kern = score_coop_kernel<T, D, GP>;
        if (plan.lds_bytes > 64 * 1024) {
            static std::atomic<bool> raised[kMaxDevices];
            const hipError_t e = raise_lds_limit(reinterpret_cast<const void*>(kern), raised);
            if (e != hipSuccess) return e;
        }
        hipLaunchKernelGGL(kern, dim3(grid), dim3(kThreads), plan.lds_bytes, s, a, xchg, grid / a.nchunk, faults,
                           g_spin_limit.load(std::memory_order_relaxed));
        return hipGetLastError();
    }
}

// Workgroups of the chunk-exchange kernel one CU holds with `lds` bytes of dynamic LDS (0 when the query
// fails), cached per device and LDS size class (the plan's LDS is one of a few chunk sizes; a different size
// on the same device re-queries).
template <typename T, int D, int GP>
int coop_occupancy(size_t lds) {
    if constexpr (Geometry<T, D, 1>::kChunks < GP) {
        return 0;
    } else {
        static std::atomic<uint64_t> cached[kMaxDevices];  // (lds << 8) | (occupancy + 1); 0 = not queried
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) dev = -1;
        if (dev >= 0) {
            const uint64_t c = cached[dev].load(std::memory_order_relaxed);
            if (c != 0 && (c >> 8) == lds) return (int)(c & 0xff) - 1;
        }
        int v = 0;
        static std::atomic<bool> raised[kMaxDevices];
        if (lds > 64 * 1024 &&
            raise_lds_limit(reinterpret_cast<const void*>(score_coop_kernel<T, D, GP>), raised) != hipSuccess)
            return 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&v, score_coop_kernel<T, D, GP>, kThreads, lds) !=
            hipSuccess)
            return 0;
        if (dev >= 0 && v >= 0 && v < 255) cached[dev].store(((uint64_t)lds << 8) | (uint64_t)(v + 1),
                                                            std::memory_order_relaxed);
        return v;
    }
}

template <typename T, int D>
hipError_t launch_coop_d(const ScorePlan& plan, const ScoreArgs& a, uint64_t* xchg, int grid, uint32_t* faults,
                         hipStream_t s) {
    switch (plan.group_pad) {
        case 1: return launch_coop_gp<T, D, 1>(plan, a, xchg, grid, faults, s);
        case 2: return launch_coop_gp<T, D, 2>(plan, a, xchg, grid, faults, s);
        case 4: return launch_coop_gp<T, D, 4>(plan, a, xchg, grid, faults, s);
        case 8: return launch_coop_gp<T, D, 8>(plan, a, xchg, grid, faults, s);
        case 16: return launch_coop_gp<T, D, 16>(plan, a, xchg, grid, faults, s);
        default: return hipErrorInvalidValue;
    }
}

template <typename T, int D>
int coop_occupancy_d(int gp, size_t lds) {
    switch (gp) {
        case 1: return coop_occupancy<T, D, 1>(lds);
        case 2: return coop_occupancy<T, D, 2>(lds);
        case 4: return coop_occupancy<T, D, 4>(lds);
        case 8: return coop_occupancy<T, D, 8>(lds);
        case 16: return coop_occupancy<T, D, 16>(lds);
        default: return 0;
    }
}

}  // namespace

bool coop_plan(int dtype, int head_dim, int group, int n, int slabs, int merge, ScorePlan* plan) {
    ScorePlan p;
    if (merge < 1 || !score_plan(dtype, head_dim, group, 1, &p)) return false;
    const size_t budget = coop_chunk_lds(p.group_pad, merge > 1);
    const size_t block = kWave * sizeof(float);  // one LDS block of logits: rpw rows
    const int rpw = kWave / p.group_pad;
    // the kernel's LDS: the chunk's blocks of logits, then with merge > 1 the item sums of its rows (blocks
    // rounded up to whole iterations of kWaves blocks)
    auto lds_of = [&](int rows) {
        const size_t units = (size_t)(rows + rpw - 1) / rpw;
        if (merge == 1) return units * block;
        const size_t whole = (units + kWaves - 1) / kWaves * kWaves;
        return whole * block + whole * rpw * sizeof(float);
    };
    // the logits take group_pad / (group_pad + 1) of the budget when the sums share it
    size_t cap = merge == 1 ? budget : budget * p.group_pad / (p.group_pad + 1);
    for (;;) {
        if (!attend_plan(dtype, head_dim, group, n, slabs, plan, cap)) return false;
        const size_t need = lds_of(plan->chunk_rows);
        if (need <= budget) {
            plan->lds_bytes = need;
            break;
        }
        if (cap <= kWaves * block) return false;
        cap -= kWaves * block;
    }
    plan->merge = merge;
    return true;
}

int coop_workgroups(int dtype, int head_dim, const ScorePlan& plan) {
    int occ = 0;
    if (dtype == 0)
        occ = head_dim == 64 ? coop_occupancy_d<float, 64>(plan.group_pad, plan.lds_bytes)
                             : coop_occupancy_d<float, 128>(plan.group_pad, plan.lds_bytes);
    else
        occ = head_dim == 64 ? coop_occupancy_d<bf16_t, 64>(plan.group_pad, plan.lds_bytes)
                             : coop_occupancy_d<bf16_t, 128>(plan.group_pad, plan.lds_bytes);
    const int cus = device_cus();
    if (occ < 1 || cus < 1) return 0;
    return occ * cus;
}

hipError_t launch_fault_word(uint32_t* word, uint32_t* out, bool clear, hipStream_t s) {
    hipLaunchKernelGGL(fault_word_kernel, dim3(1), dim3(64), 0, s, word, out, clear ? 1 : 0);
    return hipGetLastError();
}

int set_exchange_wait_limit(int polls) {
    return g_spin_limit.exchange(polls < 0 ? kDefaultSpinLimit : polls, std::memory_order_relaxed);
}

hipError_t launch_score_coop(int dtype, int head_dim, const ScorePlan& plan, const ScoreArgs& a, uint64_t* xchg,
                             int grid, uint32_t* faults, hipStream_t s) {
    const size_t words = (size_t)a.layers * a.batch * a.hq * a.nchunk;
    const unsigned zb = (unsigned)std::min<size_t>((words + 255) / 256, 2048);
    hipLaunchKernelGGL(zero_words_kernel, dim3(zb), dim3(256), 0, s, xchg, words);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (dtype == 0) {
        if (head_dim == 64) return launch_coop_d<float, 64>(plan, a, xchg, grid, faults, s);
        if (head_dim == 128) return launch_coop_d<float, 128>(plan, a, xchg, grid, faults, s);
    } else {
        if (head_dim == 64) return launch_coop_d<bf16_t, 64>(plan, a, xchg, grid, faults, s);
        if (head_dim == 128) return launch_coop_d<bf16_t, 128>(plan, a, xchg, grid, faults, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace ikv
