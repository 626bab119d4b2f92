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
// slots at or above k ("tails") using a wave-ballot prefix scan, and records the pair count per sequence.
#include "kernels.h"
#include "kv_common.h"

namespace ikv {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;

struct SelShared {
    unsigned hist[256];
    unsigned bcast[4];
    unsigned cnt[kWaves][2];
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
            for (int i = tid; i < n; i += kThreads) {
                const uint32_t key = float_key(ub[i]);
                if ((key & pmask) == prefix) atomicAdd(&sh.hist[(key >> shift) & 255u], 1u);
            }
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
                for (int i = tid; i < n; i += kThreads) {
                    if (float_key(ub[i]) != tau) continue;
                    const uint32_t ps = (uint32_t)pb[i];
                    if ((ps & pm) == pp) atomicAdd(&sh.hist[(ps >> shift) & 255u], 1u);
                }
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
        for (int i = tid; i < n; i += kThreads) ko[i] = keep_of(i) ? 1 : 0;
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

    unsigned base_h = 0, base_t = 0;
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
    for (int start = 0; start < n; start += kThreads) {
        const int i = start + tid;
        const bool kp = (i < n) && keep_of(i);
        const bool hole = (i < n) && (i < k) && !kp;
        const bool tail = (i < n) && (i >= k) && kp;
        const uint64_t mh = __ballot(hole);
        const uint64_t mt = __ballot(tail);
        if (lane == 0) {
            sh.cnt[wave][0] = __popcll(mh);
            sh.cnt[wave][1] = __popcll(mt);
        }
        __syncthreads();
        unsigned off_h = base_h, off_t = base_t, tot_h = 0, tot_t = 0;
        for (int w = 0; w < kWaves; ++w) {
            if (w < wave) {
                off_h += sh.cnt[w][0];
                off_t += sh.cnt[w][1];
            }
            tot_h += sh.cnt[w][0];
            tot_t += sh.cnt[w][1];
        }
        if (hole) {
            const unsigned j = off_h + __popcll(mh & below);
            if (j < (unsigned)a.max_pairs) pdst[j] = i;
        }
        if (tail) {
            const unsigned j = off_t + __popcll(mt & below);
            if (j < (unsigned)a.max_pairs) psrc[j] = i;
        }
        base_h += tot_h;
        base_t += tot_t;
        __syncthreads();
    }
    if (tid == 0) {
        unsigned np = min(base_h, base_t);
        a.npairs[b] = (int)min(np, (unsigned)a.max_pairs);
    }
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, bool plan_only, hipStream_t s) {
    hipLaunchKernelGGL(select_kernel, dim3(a.batch), dim3(kThreads), 0, s, a, plan_only ? 1 : 0);
    return hipGetLastError();
}

}  // namespace ikv
