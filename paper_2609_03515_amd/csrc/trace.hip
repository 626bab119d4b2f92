// Rank-trace diagnostics of the stabilisation claim (Sec. 4 and appendix "Mechanistic Diagnostics"), taken on
// a refresh step over the n tokens cached before eviction:
//   R_t = top-k of the raw step score (the per-layer pooled score of Eq. 1 averaged over layers, no memory),
//   E_t = top-k of the folded utility, both by (value descending, position ascending), identified by position.
// The raw score comes from the fold and the top-k decisions from the selection kernel; this file computes, per
// sequence, the sizes |R_t|, |E_t|, |R_t & R_t-1|, |E_t & E_t-1|, |R_t & E_t|, |R_t & evicted_t| against the
// previous traced step's sets, which persist between steps as position bitmaps in caller-owned state.
#include "kernels.h"
#include "kv_common.h"

namespace ikv {
namespace {

constexpr int kStatThreads = 1024;
constexpr int kHeader = 4;  // state words per sequence before the bitmaps: has_prev, |R_t-1|, |E_t-1|, spare

// One workgroup per sequence.  Counting reads the previous bitmaps; after a barrier the bitmaps are cleared
// and refilled with this step's sets (atomic ORs: several positions share a word).  When both bitmaps fit,
// they are worked on in LDS and copied in and out with coalesced accesses.  Positions outside [0, max_pos)
// are not recorded and flag the step (counts[0] = -2).
template <bool kLds>
__global__ __launch_bounds__(kStatThreads) void trace_stats_kernel(TraceArgs a, int skip) {
    extern __shared__ uint32_t lbm[];
    __shared__ int cnt[7];
    const int b = blockIdx.x;
    int32_t* out = a.counts + (size_t)b * kTraceCounts;
    if (skip) {  // not a refresh step: nothing traced, the state stays as it was
        if (threadIdx.x < kTraceCounts) out[threadIdx.x] = 0;
        return;
    }
    uint32_t* st = a.state + (size_t)b * (kHeader + 2 * (size_t)a.words);
    uint32_t* gbm = st + kHeader;  // raw bitmap, then EMA bitmap
    uint32_t* bm = kLds ? lbm : gbm;
    const int32_t* pb = a.pos + (size_t)b * a.cap;
    const uint8_t* rk = a.raw_keep + (size_t)b * a.cap;
    const uint8_t* ek = a.ema_keep + (size_t)b * a.cap;
    const uint8_t* kp = a.keep + (size_t)b * a.cap;
    if (threadIdx.x < 7) cnt[threadIdx.x] = 0;
    if (kLds)
        for (int w = threadIdx.x; w < 2 * a.words; w += kStatThreads) lbm[w] = gbm[w];
    __syncthreads();
    const bool has_prev = st[0] != 0;
    int c_r = 0, c_e = 0, c_rr = 0, c_ee = 0, c_re = 0, c_rev = 0, oob = 0;
    for (int i = threadIdx.x; i < a.n; i += kStatThreads) {
        const int p = pb[i];
        const bool in_r = rk[i] != 0, in_e = ek[i] != 0;
        c_r += in_r;
        c_e += in_e;
        c_re += in_r && in_e;
        c_rev += in_r && kp[i] == 0;
        if (p < 0 || p >= a.max_pos) {
            oob |= in_r || in_e;
        } else if (has_prev) {
            const uint32_t bit = 1u << (p & 31);
            c_rr += in_r && (bm[p >> 5] & bit);
            c_ee += in_e && (bm[a.words + (p >> 5)] & bit);
        }
    }
    // one LDS atomic per wave and counter (a thousand same-address atomics would serialise)
#pragma unroll
    for (int o = kWave / 2; o >= 1; o >>= 1) {
        c_r += __shfl_xor(c_r, o, kWave);
        c_e += __shfl_xor(c_e, o, kWave);
        c_rr += __shfl_xor(c_rr, o, kWave);
        c_ee += __shfl_xor(c_ee, o, kWave);
        c_re += __shfl_xor(c_re, o, kWave);
        c_rev += __shfl_xor(c_rev, o, kWave);
        oob |= __shfl_xor(oob, o, kWave);
    }
    if ((threadIdx.x & (kWave - 1)) == 0) {
        atomicAdd(&cnt[0], c_r);
        atomicAdd(&cnt[1], c_e);
        atomicAdd(&cnt[2], c_rr);
        atomicAdd(&cnt[3], c_ee);
        atomicAdd(&cnt[4], c_re);
        atomicAdd(&cnt[5], c_rev);
        atomicOr(&cnt[6], oob);
    }
    __syncthreads();  // every read of the previous sets is done
    for (int w = threadIdx.x; w < 2 * a.words; w += kStatThreads) bm[w] = 0u;
    if (!kLds) __threadfence();
    __syncthreads();
    for (int i = threadIdx.x; i < a.n; i += kStatThreads) {
        const int p = pb[i];
        if (p < 0 || p >= a.max_pos) continue;
        const uint32_t bit = 1u << (p & 31);
        if (rk[i]) atomicOr(&bm[p >> 5], bit);
        if (ek[i]) atomicOr(&bm[a.words + (p >> 5)], bit);
    }
    if (kLds) {
        __syncthreads();
        for (int w = threadIdx.x; w < 2 * a.words; w += kStatThreads) gbm[w] = lbm[w];
    }
    if (threadIdx.x == 0) {
        out[0] = cnt[6] ? -2 : 1;
        out[1] = cnt[0];
        out[2] = cnt[1];
        out[3] = has_prev ? 1 : 0;
        out[4] = cnt[2];
        out[5] = cnt[3];
        out[6] = cnt[4];
        out[7] = cnt[5];
        out[8] = has_prev ? (int)st[1] : 0;
        out[9] = has_prev ? (int)st[2] : 0;
        st[0] = 1u;
        st[1] = (uint32_t)cnt[0];
        st[2] = (uint32_t)cnt[1];
    }
}

}  // namespace

hipError_t launch_trace_stats(const TraceArgs& a, bool skip, hipStream_t s) {
    const size_t lds = 2 * (size_t)a.words * sizeof(uint32_t);
    if (!skip && lds <= 64 * 1024)
        hipLaunchKernelGGL(trace_stats_kernel<true>, dim3(a.batch), dim3(kStatThreads), lds, s, a, 0);
    else
        hipLaunchKernelGGL(trace_stats_kernel<false>, dim3(a.batch), dim3(kStatThreads), 0, s, a, skip ? 1 : 0);
    return hipGetLastError();
}

}  // namespace ikv
