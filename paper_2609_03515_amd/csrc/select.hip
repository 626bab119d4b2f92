// Top-B retention decision and hole-fill compaction plan (Sec. 3 eviction rule; ties keep the lower position).
//
// One 1024-thread workgroup per sequence.  Cases:
//  * n <= B: keep everything, nothing moves.
//  * n == B + 1 (every steady decode step): evict the single minimum under (u ascending, position
//    descending) -- one pass and a workgroup argmin.
//  * otherwise: MSB-first radix select (4 passes of 8 bits) over order-preserving utility keys finds the
//    B-th largest key tau; if more tokens tie at tau than are needed, a second radix select over positions
//    finds the largest kept position among the ties.
// The plan then pairs, in ascending order, the dropped slots below k = min(B, n) ("holes") with the kept
// slots at or above k ("tails"): per-segment counts from wave ballots, a scan over the segments, and ballot
// prefixes inside them; it records the pair count per sequence.  Measured on first-step-shaped utilities
// against one sweep of 1024-slot blocks with two barriers each: 76 -> 68 us at batch 8 x 32,769 tokens,
// 284 -> 235 us at batch 2 x 131,073, 23 -> 29 us at batch 32 x 8,193.
#include "kernels.h"
#include "kv_common.h"

namespace ikv {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;

constexpr int kMaxSegs = 2048;  // plan segments (a multiple of 64)
#ifndef IKV_SEL_BATCH
#define IKV_SEL_BATCH 8
#endif
constexpr int kBatch = IKV_SEL_BATCH;  // loads issued together by the histogram sweeps
constexpr int kPlanBatch = 16;  // 64-slot groups whose decisions a wave loads together in the plan sweeps

struct SelShared {
    unsigned hist[256];
    unsigned bcast[4];
    unsigned seg[kMaxSegs][2];  // per plan segment: holes, tails (then their offsets)
    uint32_t best_key[kWaves];
    int best_pos[kWaves];
    int best_idx[kWaves];
};

// Digit selection after a histogram pass: wave 0 scans the 256 bins in the requested order and publishes the
// digit whose bin holds the krem-th element, the count before it and the bin count.
__device__ void find_digit(SelShared& sh, unsigned krem, bool descending) {
    const int lane = threadIdx.x % kWave;
    if (threadIdx.x >= kWave) return;
    unsigned c[4], sum = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int bin = descending ? 255 - (lane * 4 + j) : lane * 4 + j;
        c[j] = sh.hist[bin];
        sum += c[j];
    }
    unsigned incl = sum;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const unsigned t = __shfl_up(incl, o, kWave);
        if (lane >= o) incl += t;
    }
    unsigned before = incl - sum;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if (before < krem && krem <= before + c[j]) {
            sh.bcast[0] = descending ? 255 - (lane * 4 + j) : lane * 4 + j;
            sh.bcast[1] = before;
            sh.bcast[2] = c[j];
        }
        before += c[j];
    }
}

// Histogram increments of one thread, aggregated over runs of equal digits: the utilities of a step cluster
// in a few exponents, so most keys of the leading passes fall in one or two bins, where one LDS atomic per key
// would serialise the whole workgroup on a single address.
struct RunCounter {
    unsigned bin = 0xffffffffu, count = 0;
    __device__ void add(unsigned* hist, unsigned d) {
        if (d != bin) {
            if (count) atomicAdd(&hist[bin], count);
            bin = d;
            count = 0;
        }
        ++count;
    }
    __device__ void flush(unsigned* hist) {
        if (count) atomicAdd(&hist[bin], count);
    }
};

__global__ __launch_bounds__(kThreads) void select_kernel(SelectArgs a, int plan_only) {
    __shared__ SelShared sh;
    const int b = blockIdx.x;
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    const float* ub = a.u + (size_t)b * a.cap;
    const int32_t* pb = a.pos + (size_t)b * a.cap;
    const int n = a.n, B = a.budget;
    const int k = min(B, n);

    // decision: mode 0 keep all, 1 evict `winner`, 2 threshold (tau, pi), 3 read keep_in
    int mode;
    int winner = -1;
    uint32_t tau = 0;
    int pi = 0x7fffffff;
    if (plan_only) {
        mode = 3;
    } else if (n <= B) {
        mode = 0;
    } else if (n == B + 1) {
        mode = 1;
        uint32_t bk = 0xffffffffu;
        int bp = -1, bi = -1;
        for (int i = tid; i < n; i += kThreads) {
            const uint32_t key = float_key(ub[i]);
            const int ps = pb[i];
            if (bi < 0 || key < bk || (key == bk && ps > bp)) {
                bk = key;
                bp = ps;
                bi = i;
            }
        }
#pragma unroll
        for (int o = kWave / 2; o >= 1; o >>= 1) {
            const uint32_t ok = __shfl_xor(bk, o, kWave);
            const int op = __shfl_xor(bp, o, kWave);
            const int oi = __shfl_xor(bi, o, kWave);
            if (oi >= 0 && (bi < 0 || ok < bk || (ok == bk && op > bp))) {
                bk = ok;
                bp = op;
                bi = oi;
            }
        }
        if (lane == 0) {
            sh.best_key[wave] = bk;
            sh.best_pos[wave] = bp;
            sh.best_idx[wave] = bi;
        }
        __syncthreads();
        bk = sh.best_key[0];
        bp = sh.best_pos[0];
        bi = sh.best_idx[0];
        for (int w = 1; w < kWaves; ++w) {
            const int oi = sh.best_idx[w];
            if (oi >= 0 && (bi < 0 || sh.best_key[w] < bk || (sh.best_key[w] == bk && sh.best_pos[w] > bp))) {
                bk = sh.best_key[w];
                bp = sh.best_pos[w];
                bi = oi;
            }
        }
        winner = bi;
    } else {
        mode = 2;
        uint32_t prefix = 0, pmask = 0;
        unsigned krem = (unsigned)B;
        unsigned ties = 0;
        for (int shift = 24; shift >= 0; shift -= 8) {
            if (tid < 256) sh.hist[tid] = 0;
            __syncthreads();
            RunCounter rc;
            for (int i0 = tid; i0 < n; i0 += kThreads * kBatch) {
                uint32_t key[kBatch];
#pragma unroll
                for (int j = 0; j < kBatch; ++j) {
                    const int i = i0 + j * kThreads;
                    key[j] = i < n ? float_key(ub[i]) : 0u;
                }
#pragma unroll
                for (int j = 0; j < kBatch; ++j)
                    if (i0 + j * kThreads < n && (key[j] & pmask) == prefix) rc.add(sh.hist, (key[j] >> shift) & 255u);
            }
            rc.flush(sh.hist);
            __syncthreads();
            find_digit(sh, krem, true);
            __syncthreads();
            prefix |= sh.bcast[0] << shift;
            pmask |= 255u << shift;
            krem -= sh.bcast[1];
            ties = sh.bcast[2];
            __syncthreads();
        }
        tau = prefix;
        if (krem < ties) {
            // keep the krem lowest positions among the ties: krem-th smallest position
            uint32_t pp = 0, pm = 0;
            for (int shift = 24; shift >= 0; shift -= 8) {
                if (tid < 256) sh.hist[tid] = 0;
                __syncthreads();
                RunCounter rc;
                for (int i = tid; i < n; i += kThreads) {
                    if (float_key(ub[i]) != tau) continue;
                    const uint32_t ps = (uint32_t)pb[i];
                    if ((ps & pm) == pp) rc.add(sh.hist, (ps >> shift) & 255u);
                }
                rc.flush(sh.hist);
                __syncthreads();
                find_digit(sh, krem, false);
                __syncthreads();
                pp |= sh.bcast[0] << shift;
                pm |= 255u << shift;
                krem -= sh.bcast[1];
                __syncthreads();
            }
            pi = (int)pp;
        }
    }

    auto keep_of = [&](int i) -> bool {
        switch (mode) {
            case 0: return true;
            case 1: return i != winner;
            case 2: {
                const uint32_t key = float_key(ub[i]);
                return key > tau || (key == tau && pb[i] <= pi);
            }
            default: return a.keep_in[(size_t)b * a.cap + i] != 0;
        }
    };

    int32_t* pdst = a.pair_dst + (size_t)b * a.max_pairs;
    int32_t* psrc = a.pair_src + (size_t)b * a.max_pairs;

    if (mode != 3 && a.keep_out) {
        uint8_t* ko = a.keep_out + (size_t)b * a.cap;
        for (int i0 = tid; i0 < n; i0 += kThreads * kBatch) {
            bool kp[kBatch];
#pragma unroll
            for (int j = 0; j < kBatch; ++j) kp[j] = i0 + j * kThreads < n && keep_of(i0 + j * kThreads);
#pragma unroll
            for (int j = 0; j < kBatch; ++j)
                if (i0 + j * kThreads < n) ko[i0 + j * kThreads] = kp[j] ? 1 : 0;
        }
    }

    if (mode == 0) {
        if (tid == 0) a.npairs[b] = 0;
        return;
    }
    if (mode == 1) {
        if (tid == 0) {
            // k = n - 1: the only slot >= k is n - 1
            int np = 0;
            if (winner != n - 1 && a.max_pairs > 0) {
                pdst[0] = winner;
                psrc[0] = n - 1;
                np = 1;
            }
            a.npairs[b] = np;
        }
        return;
    }

    // Plan: the ascending holes (dropped slots < k) pair with the ascending tails (kept slots >= k).  The slots
    // are cut into segments of kSegGroups x 64; wave w takes segments w, w + kWaves, ...  A first sweep counts
    // each segment's holes and tails, a scan over the segments gives their offsets, and a second sweep writes
    // every hole and tail at its rank (segment offset + earlier groups of the segment + ballot prefix).  The
    // sweeps have no barrier inside, so the loads of u and pos stay in flight.
    const int groups = (n + kWave - 1) / kWave;
    // 64-slot groups per segment: at least one batch of loads, and at most kMaxSegs segments
    const int seg_groups = max(kPlanBatch, (groups + kMaxSegs - 1) / kMaxSegs);
    const int nseg = (groups + seg_groups - 1) / seg_groups;
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
    // keep decisions of kBatch consecutive 64-slot groups from g0 (loads issued together)
    auto keep_batch = [&](int g0, int g1, bool (&kp)[kPlanBatch]) {
#pragma unroll
        for (int j = 0; j < kPlanBatch; ++j) {
            const int i = (g0 + j) * kWave + lane;
            kp[j] = g0 + j < g1 && i < n && keep_of(i);
        }
    };
    for (int sg = wave; sg < nseg; sg += kWaves) {
        unsigned ch = 0, ct = 0;
        const int g1 = min(groups, (sg + 1) * seg_groups);
        for (int g0 = sg * seg_groups; g0 < g1; g0 += kPlanBatch) {
            bool kp[kPlanBatch];
            keep_batch(g0, g1, kp);
#pragma unroll
            for (int j = 0; j < kPlanBatch; ++j) {
                const int i = (g0 + j) * kWave + lane;
                const bool in = g0 + j < g1 && i < n;
                ch += __popcll(__ballot(in && i < k && !kp[j]));
                ct += __popcll(__ballot(in && i >= k && kp[j]));
            }
        }
        if (lane == 0) {
            sh.seg[sg][0] = ch;
            sh.seg[sg][1] = ct;
        }
    }
    __syncthreads();
    // exclusive scan of the segment counts (wave 0; kMaxSegs / 64 entries per lane)
    if (wave == 0) {
        constexpr int kPer = kMaxSegs / kWave;
        unsigned h[kPer], t[kPer], sh_ = 0, st = 0;
#pragma unroll
        for (int j = 0; j < kPer; ++j) {
            const int sg = lane * kPer + j;
            h[j] = sg < nseg ? sh.seg[sg][0] : 0u;
            t[j] = sg < nseg ? sh.seg[sg][1] : 0u;
            sh_ += h[j];
            st += t[j];
        }
        unsigned ih = sh_, it = st;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const unsigned xh = __shfl_up(ih, o, kWave), xt = __shfl_up(it, o, kWave);
            if (lane >= o) {
                ih += xh;
                it += xt;
            }
        }
        unsigned oh = ih - sh_, ot = it - st;
#pragma unroll
        for (int j = 0; j < kPer; ++j) {
            const int sg = lane * kPer + j;
            if (sg < nseg) {
                sh.seg[sg][0] = oh;
                sh.seg[sg][1] = ot;
            }
            oh += h[j];
            ot += t[j];
        }
        if (lane == kWave - 1) {
            sh.bcast[0] = ih;  // totals
            sh.bcast[1] = it;
        }
    }
    __syncthreads();
    for (int sg = wave; sg < nseg; sg += kWaves) {
        unsigned oh = sh.seg[sg][0], ot = sh.seg[sg][1];
        const int g1 = min(groups, (sg + 1) * seg_groups);
        for (int g0 = sg * seg_groups; g0 < g1; g0 += kPlanBatch) {
            bool kp[kPlanBatch];
            keep_batch(g0, g1, kp);
#pragma unroll
            for (int j = 0; j < kPlanBatch; ++j) {
                const int i = (g0 + j) * kWave + lane;
                const bool in = g0 + j < g1 && i < n;
                const bool hole = in && i < k && !kp[j];
                const bool tail = in && i >= k && kp[j];
                const uint64_t mh = __ballot(hole), mt = __ballot(tail);
                if (hole) {
                    const unsigned r = oh + __popcll(mh & below);
                    if (r < (unsigned)a.max_pairs) pdst[r] = i;
                }
                if (tail) {
                    const unsigned r = ot + __popcll(mt & below);
                    if (r < (unsigned)a.max_pairs) psrc[r] = i;
                }
                oh += __popcll(mh);
                ot += __popcll(mt);
            }
        }
    }
    if (tid == 0) {
        const unsigned np = min(sh.bcast[0], sh.bcast[1]);
        a.npairs[b] = (int)min(np, (unsigned)a.max_pairs);
    }
}

// ---- Multi-workgroup selection: long sequences in a small batch ------------------------------------------
// One workgroup per sequence leaves most of the chip idle when the batch is small and the sequences long (the
// selection of a 128k-token first step at batch 2 took ~0.3 ms).  In the threshold case (n > B + 1) the same
// radix select then runs as a short sequence of launches over P slices of every sequence:
//   4 x (per-slice 256-bin histograms of the digit under the prefix found so far; one workgroup per sequence
//   adds the slices' bins and picks the digit),
//   one launch for ties at tau (the position select of the single-workgroup kernel; it returns at once unless
//   more tokens tie at tau than are kept),
//   per-slice hole and tail counts (and the decision, when asked for), then the pairs: every slice writes its
//   holes and tails at the ranks that follow the slices before it.
// The decisions and pairs are those of the single-workgroup kernel.  Scratch: P x 256 bins and P x 2 counts
// per sequence, and a few state words (prefix, mask, remaining rank, tie count, position bound).
__device__ __forceinline__ unsigned wave_sum_u(unsigned x) {
#pragma unroll
    for (int o = kWave / 2; o >= 1; o >>= 1) x += __shfl_xor(x, o, kWave);
    return x;
}

constexpr int kWideThreads = 256;
constexpr int kWideMaxParts = 128;
constexpr int kWideMinRows = 16384;  // shorter sequences keep the single-workgroup kernel
constexpr int kWideSlice = 1024;     // fewest slots per slice
constexpr int kStateWords = 8;

int wide_parts_max(int batch) {
    const int p = 512 / batch;
    return p < 4 ? 0 : (p > kWideMaxParts ? kWideMaxParts : p);
}

int wide_parts(int batch, int n) {
    if (n < kWideMinRows) return 0;
    int p = wide_parts_max(batch);
    if (p > n / kWideSlice) p = n / kWideSlice;
    return p < 4 ? 0 : p;
}

struct Wide {
    unsigned* hist;  // [batch][P][256]
    unsigned* cnt;   // [batch][P][2]
    unsigned* st;    // [batch][kStateWords]: prefix, mask, remaining rank, ties at tau, position bound
    int P, slice;
    __device__ int lo(int p) const { return p * slice; }
};

Wide wide_of(const SelectArgs& a, int P) {
    Wide w;
    const size_t pm = (size_t)wide_parts_max(a.batch);
    w.hist = a.wide;
    w.cnt = a.wide + (size_t)a.batch * pm * 256;
    w.st = w.cnt + (size_t)a.batch * pm * 2;
    w.P = P;
    w.slice = ((a.n + P - 1) / P + kWave - 1) / kWave * kWave;
    return w;
}

__global__ __launch_bounds__(kWideThreads) void wide_hist_kernel(SelectArgs a, Wide w, int shift) {
    __shared__ unsigned hist[256];
    const int p = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
    const unsigned* st = w.st + (size_t)b * kStateWords;
    const uint32_t prefix = shift == 24 ? 0u : st[0], pmask = shift == 24 ? 0u : st[1];
    const float* ub = a.u + (size_t)b * a.cap;
    const int lo = w.lo(p), hi = min(a.n, lo + w.slice);
    hist[tid] = 0;
    __syncthreads();
    RunCounter rc;
    for (int i0 = lo + tid; i0 < hi; i0 += kWideThreads * kBatch) {
        uint32_t key[kBatch];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            const int i = i0 + j * kWideThreads;
            key[j] = i < hi ? float_key(ub[i]) : 0u;
        }
#pragma unroll
        for (int j = 0; j < kBatch; ++j)
            if (i0 + j * kWideThreads < hi && (key[j] & pmask) == prefix) rc.add(hist, (key[j] >> shift) & 255u);
    }
    rc.flush(hist);
    __syncthreads();
    w.hist[((size_t)b * w.P + p) * 256 + tid] = hist[tid];
}

__global__ __launch_bounds__(kWideThreads) void wide_digit_kernel(SelectArgs a, Wide w, int shift) {
    __shared__ SelShared sh;
    const int b = blockIdx.x, tid = threadIdx.x;
    unsigned* st = w.st + (size_t)b * kStateWords;
    // the slices' bins, eight loads in flight per thread
    const unsigned* hb = w.hist + (size_t)b * w.P * 256 + tid;
    unsigned c = 0;
    int p = 0;
    for (; p + 8 <= w.P; p += 8) {
        unsigned x[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] = hb[(size_t)(p + j) * 256];
#pragma unroll
        for (int j = 0; j < 8; ++j) c += x[j];
    }
    for (; p < w.P; ++p) c += hb[(size_t)p * 256];
    sh.hist[tid] = c;
    const unsigned krem = shift == 24 ? (unsigned)a.budget : st[2];
    __syncthreads();
    find_digit(sh, krem, true);
    __syncthreads();
    if (tid == 0) {
        st[0] = (shift == 24 ? 0u : st[0]) | (sh.bcast[0] << shift);
        st[1] = (shift == 24 ? 0u : st[1]) | (255u << shift);
        st[2] = krem - sh.bcast[1];
        st[3] = sh.bcast[2];
    }
}

// Ties at tau: the krem lowest positions among them are kept (position radix select, one workgroup).
__global__ __launch_bounds__(kThreads) void wide_ties_kernel(SelectArgs a, Wide w) {
    __shared__ SelShared sh;
    const int b = blockIdx.x, tid = threadIdx.x;
    unsigned* st = w.st + (size_t)b * kStateWords;
    const uint32_t tau = st[0];
    unsigned krem = st[2];
    if (krem >= st[3]) {
        if (tid == 0) st[4] = 0x7fffffffu;
        return;
    }
    const float* ub = a.u + (size_t)b * a.cap;
    const int32_t* pb = a.pos + (size_t)b * a.cap;
    uint32_t pp = 0, pm = 0;
    for (int shift = 24; shift >= 0; shift -= 8) {
        if (tid < 256) sh.hist[tid] = 0;
        __syncthreads();
        RunCounter rc;
        for (int i = tid; i < a.n; i += kThreads) {
            if (float_key(ub[i]) != tau) continue;
            const uint32_t ps = (uint32_t)pb[i];
            if ((ps & pm) == pp) rc.add(sh.hist, (ps >> shift) & 255u);
        }
        rc.flush(sh.hist);
        __syncthreads();
        find_digit(sh, krem, false);
        __syncthreads();
        pp |= sh.bcast[0] << shift;
        pm |= 255u << shift;
        krem -= sh.bcast[1];
        __syncthreads();
    }
    if (tid == 0) st[4] = pp;
}

__device__ __forceinline__ bool wide_keep(const SelectArgs& a, const Wide& w, int b, int i) {
    const unsigned* st = w.st + (size_t)b * kStateWords;
    const uint32_t key = float_key(a.u[(size_t)b * a.cap + i]);
    return key > st[0] || (key == st[0] && a.pos[(size_t)b * a.cap + i] <= (int)st[4]);
}

// Per slice: holes (dropped slots < k) and tails (kept slots >= k), and the decision when asked for.
__global__ __launch_bounds__(kWideThreads) void wide_count_kernel(SelectArgs a, Wide w) {
    __shared__ unsigned part[kWideThreads / kWave][2];
    const int p = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
    const int k = min(a.budget, a.n);
    const int lo = w.lo(p), hi = min(a.n, lo + w.slice);
    unsigned ch = 0, ct = 0;
    for (int i = lo + tid; i < hi; i += kWideThreads) {
        const bool kp = wide_keep(a, w, b, i);
        if (a.keep_out) a.keep_out[(size_t)b * a.cap + i] = kp ? 1 : 0;
        ch += i < k && !kp;
        ct += i >= k && kp;
    }
    ch = wave_sum_u(ch);
    ct = wave_sum_u(ct);
    if (tid % kWave == 0) {
        part[tid / kWave][0] = ch;
        part[tid / kWave][1] = ct;
    }
    __syncthreads();
    if (tid == 0) {
        unsigned h = 0, t = 0;
        for (int j = 0; j < kWideThreads / kWave; ++j) {
            h += part[j][0];
            t += part[j][1];
        }
        w.cnt[((size_t)b * w.P + p) * 2] = h;
        w.cnt[((size_t)b * w.P + p) * 2 + 1] = t;
    }
}

// Pairs: wave j of a slice takes its j-th quarter (whole 64-slot groups) and writes its holes and tails at the
// ranks after the earlier slices and quarters; the last slice records the pair count.
__global__ __launch_bounds__(kWideThreads) void wide_plan_kernel(SelectArgs a, Wide w) {
    constexpr int kW = kWideThreads / kWave;
    __shared__ unsigned base[2], wc[kW][2];
    const int p = blockIdx.x, b = blockIdx.y, tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    const int k = min(a.budget, a.n);
    const int lo = w.lo(p), hi = min(a.n, lo + w.slice);
    if (wave == 0) {  // holes and tails of the slices before this one (P <= 128: two per lane)
        unsigned h = 0, t = 0;
        for (int q = lane; q < p; q += kWave) {
            h += w.cnt[((size_t)b * w.P + q) * 2];
            t += w.cnt[((size_t)b * w.P + q) * 2 + 1];
        }
        h = wave_sum_u(h);
        t = wave_sum_u(t);
        if (lane == 0) {
            base[0] = h;
            base[1] = t;
        }
    }
    const int groups = hi > lo ? (hi - lo + kWave - 1) / kWave : 0;
    const int per = (groups + kW - 1) / kW;
    const int g0 = wave * per, g1 = min(groups, g0 + per);
    unsigned ch = 0, ct = 0;
    for (int g = g0; g < g1; ++g) {
        const int i = lo + g * kWave + lane;
        const bool in = i < hi;
        const bool kp = in && wide_keep(a, w, b, i);
        ch += __popcll(__ballot(in && i < k && !kp));
        ct += __popcll(__ballot(in && i >= k && kp));
    }
    if (lane == 0) {
        wc[wave][0] = ch;
        wc[wave][1] = ct;
    }
    __syncthreads();
    unsigned oh = base[0], ot = base[1];
    for (int j = 0; j < wave; ++j) {
        oh += wc[j][0];
        ot += wc[j][1];
    }
    int32_t* pdst = a.pair_dst + (size_t)b * a.max_pairs;
    int32_t* psrc = a.pair_src + (size_t)b * a.max_pairs;
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
    for (int g = g0; g < g1; ++g) {
        const int i = lo + g * kWave + lane;
        const bool in = i < hi;
        const bool kp = in && wide_keep(a, w, b, i);
        const bool hole = in && i < k && !kp;
        const bool tail = in && i >= k && kp;
        const uint64_t mh = __ballot(hole), mt = __ballot(tail);
        if (hole) {
            const unsigned r = oh + __popcll(mh & below);
            if (r < (unsigned)a.max_pairs) pdst[r] = i;
        }
        if (tail) {
            const unsigned r = ot + __popcll(mt & below);
            if (r < (unsigned)a.max_pairs) psrc[r] = i;
        }
        oh += __popcll(mh);
        ot += __popcll(mt);
    }
    if (p == w.P - 1 && tid == 0) {
        unsigned h = base[0], t = base[1];
        for (int j = 0; j < kW; ++j) {
            h += wc[j][0];
            t += wc[j][1];
        }
        a.npairs[b] = (int)min(min(h, t), (unsigned)a.max_pairs);
    }
}

}  // namespace

size_t select_wide_words(int batch) {
    const size_t pm = (size_t)wide_parts_max(batch);
    return pm ? (size_t)batch * (pm * 258 + kStateWords) : 0;
}

hipError_t launch_select(const SelectArgs& a, bool plan_only, hipStream_t s) {
    const int P = a.wide ? wide_parts(a.batch, a.n) : 0;
    if (plan_only || a.n <= a.budget + 1 || P == 0) {
        hipLaunchKernelGGL(select_kernel, dim3(a.batch), dim3(kThreads), 0, s, a, plan_only ? 1 : 0);
        return hipGetLastError();
    }
    const Wide w = wide_of(a, P);
    const dim3 sliced(P, a.batch);
    for (int shift = 24; shift >= 0; shift -= 8) {
        hipLaunchKernelGGL(wide_hist_kernel, sliced, dim3(kWideThreads), 0, s, a, w, shift);
        hipLaunchKernelGGL(wide_digit_kernel, dim3(a.batch), dim3(kWideThreads), 0, s, a, w, shift);
    }
    hipLaunchKernelGGL(wide_ties_kernel, dim3(a.batch), dim3(kThreads), 0, s, a, w);
    hipLaunchKernelGGL(wide_count_kernel, sliced, dim3(kWideThreads), 0, s, a, w);
    hipLaunchKernelGGL(wide_plan_kernel, sliced, dim3(kWideThreads), 0, s, a, w);
    return hipGetLastError();
}

}  // namespace ikv
