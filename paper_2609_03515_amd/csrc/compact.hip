// Cache row movement: append of the decode token and hole-fill compaction.
//
// Both are byte copies of whole K/V rows (d elements), done with 16-byte vector loads/stores by a group of
// row_bytes/16 lanes per row.  Compaction moves row src -> dst for every (layer, KV head) slab of K and V of
// one sequence; the plan guarantees src >= k > dst, so reads and writes never overlap within a launch.
#include "kernels.h"
#include "kv_common.h"

namespace ikv {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxBlocks = 65536;

__global__ __launch_bounds__(kThreads) void move_kernel(MoveArgs a) {
    const int lpr = a.row_bytes / 16;
    const long long total = (long long)a.batch * a.layers * a.hkv * 2 * a.max_pairs * lpr;
    const long long stride = (long long)gridDim.x * blockDim.x;
    for (long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x; gid < total; gid += stride) {
        const int c = (int)(gid % lpr);
        long long task = gid / lpr;
        const int j = (int)(task % a.max_pairs);
        task /= a.max_pairs;
        const int tensor = (int)(task & 1);
        task >>= 1;
        const int g = (int)(task % a.hkv);
        task /= a.hkv;
        const int l = (int)(task % a.layers);
        const int b = (int)(task / a.layers);
        if (j >= a.npairs[b]) continue;
        const int dst = a.pair_dst[(size_t)b * a.pair_stride + j];
        const int src = a.pair_src[(size_t)b * a.pair_stride + j];
        char* base = static_cast<char*>(tensor ? a.v : a.k);
        const size_t slab = ((size_t)(l * a.batch + b) * a.hkv + g) * a.cap;
        const u32x4* from = reinterpret_cast<const u32x4*>(base + (slab + src) * a.row_bytes) + c;
        u32x4* to = reinterpret_cast<u32x4*>(base + (slab + dst) * a.row_bytes) + c;
        *to = *from;
        if (l == 0 && g == 0 && tensor == 0 && c == 0) {
            a.u[(size_t)b * a.cap + dst] = a.u[(size_t)b * a.cap + src];
            a.pos[(size_t)b * a.cap + dst] = a.pos[(size_t)b * a.cap + src];
        }
    }
}

// Blocks [0, batch): prior utility and position of the appended token of one sequence.
// Blocks >= batch: copies of the new K/V rows into slot n_in of every slab.
__global__ __launch_bounds__(kThreads) void append_kernel(AppendArgs a) {
    if ((int)blockIdx.x < a.batch) {
        __shared__ float red[kThreads / kWave];
        const int b = blockIdx.x;
        const float* ub = a.u + (size_t)b * a.cap;
        float v = 0.0f;
        if (a.init_mode == 1) {
            for (int i = threadIdx.x; i < a.n_in; i += kThreads) v += ub[i];
            v = wave_sum(v);
        } else if (a.init_mode == 2) {
            v = INFINITY;
            for (int i = threadIdx.x; i < a.n_in; i += kThreads) v = fminf(v, ub[i]);
#pragma unroll
            for (int o = kWave / 2; o >= 1; o >>= 1) v = fminf(v, __shfl_xor(v, o, kWave));
        }
        if (threadIdx.x % kWave == 0) red[threadIdx.x / kWave] = v;
        __syncthreads();
        if (threadIdx.x == 0) {
            float r = red[0];
            for (int w = 1; w < kThreads / kWave; ++w) r = a.init_mode == 2 ? fminf(r, red[w]) : r + red[w];
            float prior = 0.0f;
            if (a.n_in > 0) {
                if (a.init_mode == 1) prior = r / (float)a.n_in;
                if (a.init_mode == 2) prior = r;
            }
            a.u[(size_t)b * a.cap + a.n_in] = prior;
            a.pos[(size_t)b * a.cap + a.n_in] = a.new_pos;
        }
        return;
    }
    const int lpr = a.row_bytes / 16;
    const long long gid = (long long)(blockIdx.x - a.batch) * blockDim.x + threadIdx.x;
    const long long total = (long long)a.layers * a.batch * a.hkv * 2 * lpr;
    if (gid >= total) return;
    const int c = (int)(gid % lpr);
    long long row = gid / lpr;  // (tensor, l, b, g) with tensor outermost
    const int tensor = (int)(row / ((long long)a.layers * a.batch * a.hkv));
    row %= (long long)a.layers * a.batch * a.hkv;  // == (l * batch + b) * hkv + g
    const char* src = static_cast<const char*>(tensor ? a.v_new : a.k_new) + (size_t)row * a.row_bytes;
    char* dst = static_cast<char*>(tensor ? a.v : a.k) + ((size_t)row * a.cap + a.n_in) * a.row_bytes;
    reinterpret_cast<u32x4*>(dst)[c] = reinterpret_cast<const u32x4*>(src)[c];
}

// A whole non-refresh step of one sequence whose cache holds n_in <= B tokens (every Lazy / Score-Free step
// after the first): the newcomer's prior from the n_in utilities (mean or min, as append_kernel), the single
// eviction among the n_in + 1 tokens (minimum under (u ascending, position descending), as select_kernel's
// one-eviction case) and the newcomer's K/V rows written straight into the slot it takes: the evicted one
// (the same cache, u and pos as append + select + hole-fill), or slot n_in when nothing is evicted.  When the
// newcomer itself is evicted nothing is written.
constexpr int kNrThreads = 1024;
constexpr int kNrWaves = kNrThreads / kWave;

__global__ __launch_bounds__(kNrThreads) void nonrefresh_kernel(AppendArgs a, uint8_t* keep_out, int budget) {
    __shared__ float red[kNrWaves];
    __shared__ uint32_t best_key[kNrWaves];
    __shared__ int best_pos[kNrWaves], best_idx[kNrWaves];
    __shared__ float prior_sh;
    __shared__ int slot_sh;
    const int b = blockIdx.x;
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    float* ub = a.u + (size_t)b * a.cap;
    int32_t* pb = a.pos + (size_t)b * a.cap;
    const int n = a.n_in;

    float v = a.init_mode == 2 ? INFINITY : 0.0f;
    for (int i = tid; i < n; i += kNrThreads) v = a.init_mode == 2 ? fminf(v, ub[i]) : v + ub[i];
#pragma unroll
    for (int o = kWave / 2; o >= 1; o >>= 1) {
        const float w = __shfl_xor(v, o, kWave);
        v = a.init_mode == 2 ? fminf(v, w) : v + w;
    }
    if (lane == 0) red[wave] = v;
    __syncthreads();
    if (tid == 0) {
        float r = red[0];
        for (int w = 1; w < kNrWaves; ++w) r = a.init_mode == 2 ? fminf(r, red[w]) : r + red[w];
        prior_sh = n > 0 ? (a.init_mode == 2 ? r : r / (float)n) : 0.0f;
    }
    __syncthreads();
    const float prior = prior_sh;

    int slot = n;  // no eviction: the newcomer takes slot n
    if (n + 1 > budget) {
        // argmin over the n cached tokens and the newcomer (index n)
        uint32_t bk = 0xffffffffu;
        int bp = -1, bi = -1;
        for (int i = tid; i <= n; i += kNrThreads) {
            const uint32_t key = float_key(i < n ? ub[i] : prior);
            const int ps = i < n ? pb[i] : a.new_pos;
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
            best_key[wave] = bk;
            best_pos[wave] = bp;
            best_idx[wave] = bi;
        }
        __syncthreads();
        if (tid == 0) {
            bk = best_key[0];
            bp = best_pos[0];
            bi = best_idx[0];
            for (int w = 1; w < kNrWaves; ++w) {
                const int oi = best_idx[w];
                if (oi >= 0 && (bi < 0 || best_key[w] < bk || (best_key[w] == bk && best_pos[w] > bp))) {
                    bk = best_key[w];
                    bp = best_pos[w];
                    bi = oi;
                }
            }
            slot_sh = bi;
        }
        __syncthreads();
        slot = slot_sh;
        if (keep_out)
            for (int i = tid; i <= n; i += kNrThreads) keep_out[(size_t)b * a.cap + i] = i != slot;
        if (slot == n) return;  // the newcomer is evicted at once
    } else if (keep_out) {
        for (int i = tid; i <= n; i += kNrThreads) keep_out[(size_t)b * a.cap + i] = 1;
    }
    if (tid == 0) {
        ub[slot] = prior;
        pb[slot] = a.new_pos;
    }
    const int lpr = a.row_bytes / 16;
    const int rows = a.layers * a.hkv * 2;
    for (int c = tid; c < rows * lpr; c += kNrThreads) {
        const int chunk = c % lpr;
        const int r = c / lpr;
        const int tensor = r / (a.layers * a.hkv);
        const int lg = r % (a.layers * a.hkv);  // l * hkv + g
        const size_t row = ((size_t)(lg / a.hkv) * a.batch + b) * a.hkv + lg % a.hkv;  // (l, b, g)
        const char* src = static_cast<const char*>(tensor ? a.v_new : a.k_new) + row * a.row_bytes;
        char* dst = static_cast<char*>(tensor ? a.v : a.k) + (row * a.cap + slot) * a.row_bytes;
        reinterpret_cast<u32x4*>(dst)[chunk] = reinterpret_cast<const u32x4*>(src)[chunk];
    }
}

}  // namespace

hipError_t launch_nonrefresh(const AppendArgs& a, uint8_t* keep_out, int budget, hipStream_t s) {
    hipLaunchKernelGGL(nonrefresh_kernel, dim3(a.batch), dim3(kNrThreads), 0, s, a, keep_out, budget);
    return hipGetLastError();
}

hipError_t launch_move(const MoveArgs& a, hipStream_t s) {
    const long long threads = (long long)a.batch * a.layers * a.hkv * 2 * a.max_pairs * (a.row_bytes / 16);
    if (threads <= 0) return hipSuccess;
    long long blocks = (threads + kThreads - 1) / kThreads;
    if (blocks > kMaxBlocks) blocks = kMaxBlocks;
    hipLaunchKernelGGL(move_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_append(const AppendArgs& a, hipStream_t s) {
    const long long threads = (long long)a.layers * a.batch * a.hkv * 2 * (a.row_bytes / 16);
    const long long blocks = a.batch + (threads + kThreads - 1) / kThreads;
    hipLaunchKernelGGL(append_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace ikv
