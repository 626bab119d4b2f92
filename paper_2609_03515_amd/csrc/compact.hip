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

// Grid (pair blocks, (layer, KV head, tensor), sequence): a workgroup moves kMoveUnroll passes of
// kThreads / lpr rows of one slab of K or V, each row by lpr lanes of 16 bytes; a thread issues its
// kMoveUnroll loads before its stores (the rows are disjoint), so several loads are in flight per lane.
// Rows are read and written once: non-temporal loads and stores.  Step 1 at the 8B shape, same process: 4.20
// ms with cached accesses and 4 rows per thread, 4.13 ms non-temporal; then 1 / 2 / 3 / 4 / 6 rows per thread:
// 4.14 / 4.05 / 4.08 / 4.13 / 4.35 ms (8: 5.36 ms).  Later (same method): 512-thread workgroups 3.893 and a grid
// whose first dimension runs over the slabs 3.986 against 3.808 ms (Qwen-shaped step 1: 2.379 / 2.357 against
// 2.386 ms).
constexpr int kMoveUnroll = 2;

__global__ __launch_bounds__(kThreads) void move_kernel(MoveArgs a) {
    const int lpr = a.row_bytes / 16;
    const int rows_per_pass = kThreads / lpr;
    const int b = blockIdx.z;
    const int tensor = (int)blockIdx.y & 1;
    const int g = ((int)blockIdx.y >> 1) % a.hkv;
    const int l = ((int)blockIdx.y >> 1) / a.hkv;
    const int np = a.npairs[b];
    const int j0 = (int)blockIdx.x * rows_per_pass * kMoveUnroll + (int)threadIdx.x / lpr;
    if (j0 >= np) return;
    const int c = (int)threadIdx.x % lpr;
    char* base = static_cast<char*>(tensor ? a.v : a.k) + ((size_t)(l * a.batch + b) * a.hkv + g) * a.cap * a.row_bytes;
    const int32_t* pd = a.pair_dst + (size_t)b * a.pair_stride;
    const int32_t* ps = a.pair_src + (size_t)b * a.pair_stride;
    u32x4 x[kMoveUnroll];
    int dst[kMoveUnroll];
#pragma unroll
    for (int i = 0; i < kMoveUnroll; ++i) {
        const int j = j0 + i * rows_per_pass;
        dst[i] = -1;
        if (j < np) {
            const int src = ps[j];
            dst[i] = pd[j];
            x[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(base + (size_t)src * a.row_bytes) + c);
        }
    }
#pragma unroll
    for (int i = 0; i < kMoveUnroll; ++i)
        if (dst[i] >= 0) __builtin_nontemporal_store(x[i], reinterpret_cast<u32x4*>(base + (size_t)dst[i] * a.row_bytes) + c);
    if (a.norms && tensor == 1 && c == 0) {  // V blocks also move their slab's value norms
        float* nb = a.norms + ((size_t)(l * a.batch + b) * a.hkv + g) * a.cap;
#pragma unroll
        for (int i = 0; i < kMoveUnroll; ++i) {
            const int j = j0 + i * rows_per_pass;
            if (j < np) nb[pd[j]] = nb[ps[j]];
        }
    }
    if (blockIdx.y == 0 && c == 0) {  // layer 0, KV head 0, K: the rows' utilities and positions
#pragma unroll
        for (int i = 0; i < kMoveUnroll; ++i) {
            const int j = j0 + i * rows_per_pass;
            if (j < np) {
                const int src = ps[j];
                a.u[(size_t)b * a.cap + pd[j]] = a.u[(size_t)b * a.cap + src];
                a.pos[(size_t)b * a.cap + pd[j]] = a.pos[(size_t)b * a.cap + src];
            }
        }
    }
}

// Blocks [0, batch): prior utility and position of the appended token of one sequence.
// Blocks [batch, batch + copy blocks): copies of the new K/V rows into slot n_in of every slab.
// Blocks after those (with a norm cache): the new V rows' norms into slot n_in of the cache.
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
    const long long total = (long long)a.layers * a.batch * a.hkv * 2 * lpr;
    const long long copy_blocks = (total + kThreads - 1) / kThreads;
    if ((long long)blockIdx.x >= a.batch + copy_blocks) {
        // one aligned lane group per row (l, b, g); groups leave or stay together
        const int nl = norm_lanes(a.row_bytes);
        const long long r = ((long long)blockIdx.x - a.batch - copy_blocks) * (kThreads / nl) + threadIdx.x / nl;
        if (r >= (long long)a.layers * a.batch * a.hkv) return;
        const float nrm = row_norm(static_cast<const char*>(a.v_new) + r * a.row_bytes, a.row_bytes, a.bf16 != 0,
                                   (int)threadIdx.x % nl);
        if ((int)threadIdx.x % nl == 0) a.norms[r * a.cap + a.n_in] = nrm;
        return;
    }
    const long long gid = (long long)(blockIdx.x - a.batch) * blockDim.x + threadIdx.x;
    if (gid >= total) return;
    const int c = (int)(gid % lpr);
    long long row = gid / lpr;  // (tensor, l, b, g) with tensor outermost
    const int tensor = (int)(row / ((long long)a.layers * a.batch * a.hkv));
    row %= (long long)a.layers * a.batch * a.hkv;  // == (l * batch + b) * hkv + g
    const char* src = static_cast<const char*>(tensor ? a.v_new : a.k_new) + (size_t)row * a.row_bytes;
    char* dst = static_cast<char*>(tensor ? a.v : a.k) + ((size_t)row * a.cap + a.n_in) * a.row_bytes;
    reinterpret_cast<u32x4*>(dst)[c] = reinterpret_cast<const u32x4*>(src)[c];
}

// Decision of a non-refresh step of one sequence whose cache holds n_in <= B tokens (every Lazy / Score-Free
// step after the first), in one pass over u and pos: the newcomer's prior (mean or min of the n_in utilities,
// as append_kernel) and the minimum of the cached tokens under (u ascending, position descending); the
// newcomer is then compared with that minimum (select_kernel's one-eviction rule over the n_in + 1 tokens).
// The newcomer takes the evicted slot (the same cache, u and pos as append + select + hole-fill), slot n_in
// when nothing is evicted, or no slot when it is itself evicted (slot[b] = -1); its rows are copied here
// (copy_rows) or by newcomer_rows_kernel.
constexpr int kNrThreads = 1024;
constexpr int kNrWaves = kNrThreads / kWave;

using Cand = EvictCand;

__global__ __launch_bounds__(kNrThreads) void nonrefresh_kernel(AppendArgs a, uint8_t* keep_out, int budget,
                                                                int* slot_out, int copy_rows) {
    __shared__ float red[kNrWaves];
    __shared__ Cand best[kNrWaves];
    __shared__ int slot_sh;
    const int b = blockIdx.x;
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    float* ub = a.u + (size_t)b * a.cap;
    int32_t* pb = a.pos + (size_t)b * a.cap;
    const int n = a.n_in;
    const bool use_min = a.init_mode == 2;

    float v = use_min ? INFINITY : 0.0f;
    Cand c{0xffffffffu, -1, -1};
    // kNrBatch tokens' loads in flight per thread; the reduction keeps the order of a plain sweep
    constexpr int kNrBatch = 8;
    for (int i0 = tid; i0 < n; i0 += kNrThreads * kNrBatch) {
        float uu[kNrBatch];
        int pp[kNrBatch];
#pragma unroll
        for (int j = 0; j < kNrBatch; ++j) {
            const int i = i0 + j * kNrThreads;
            if (i < n) {
                uu[j] = ub[i];
                pp[j] = pb[i];
            }
        }
#pragma unroll
        for (int j = 0; j < kNrBatch; ++j) {
            const int i = i0 + j * kNrThreads;
            if (i < n) {
                v = use_min ? fminf(v, uu[j]) : v + uu[j];
                const Cand o{float_key(uu[j]), pp[j], i};
                if (evicts_before(o, c)) c = o;
            }
        }
    }
#pragma unroll
    for (int o = kWave / 2; o >= 1; o >>= 1) {
        const float w = __shfl_xor(v, o, kWave);
        v = use_min ? fminf(v, w) : v + w;
        const Cand x = shfl_xor_cand(c, o);
        if (evicts_before(x, c)) c = x;
    }
    if (lane == 0) {
        red[wave] = v;
        best[wave] = c;
    }
    __syncthreads();
    if (tid == 0) {
        float r = red[0];
        c = best[0];
        for (int w = 1; w < kNrWaves; ++w) {
            r = use_min ? fminf(r, red[w]) : r + red[w];
            if (evicts_before(best[w], c)) c = best[w];
        }
        const float prior = n > 0 ? (use_min ? r : r / (float)n) : 0.0f;
        int slot = n;  // room left: the newcomer is appended
        if (n + 1 > budget) {
            const Cand mine{float_key(prior), a.new_pos, n};
            slot = evicts_before(mine, c) ? -1 : c.idx;
        }
        if (slot >= 0) {
            ub[slot] = prior;
            pb[slot] = a.new_pos;
        }
        slot_out[b] = slot;
        slot_sh = slot;
    }
    __syncthreads();
    const int slot = slot_sh;
    if (keep_out) {
        const int evicted = slot < 0 ? n : (slot < n ? slot : -1);
        for (int i = tid; i <= n; i += kNrThreads) keep_out[(size_t)b * a.cap + i] = i != evicted;
    }
    if (slot < 0) return;
    if (a.norms) {  // the newcomer's value norms, one aligned lane group per (layer, KV head) row
        const int nl = norm_lanes(a.row_bytes);
        for (int r = tid / nl; r < a.layers * a.hkv; r += kNrThreads / nl) {
            const size_t row = ((size_t)(r / a.hkv) * a.batch + b) * a.hkv + r % a.hkv;
            const float nrm = row_norm(static_cast<const char*>(a.v_new) + row * a.row_bytes, a.row_bytes,
                                       a.bf16 != 0, tid % nl);
            if (tid % nl == 0) a.norms[row * a.cap + slot] = nrm;
        }
    }
    if (!copy_rows) return;
    // rows r = (tensor, l, g) in [0, 2 L hkv), 16-byte chunk ch; quotients by float reciprocals (exact: the
    // numerators are far below 2^22 and the +0.5 keeps them off integer boundaries)
    const int lpr = a.row_bytes / 16;
    const int total = a.layers * a.hkv * 2 * lpr;
    const float inv_lpr = 1.0f / (float)lpr, inv_hkv = 1.0f / (float)a.hkv, inv_lg = 1.0f / (float)(a.layers * a.hkv);
    constexpr int kCopy = 8;
    for (int c0 = tid; c0 < total; c0 += kNrThreads * kCopy) {
        u32x4 buf[kCopy];
        size_t dsto[kCopy];
#pragma unroll
        for (int j = 0; j < kCopy; ++j) {
            const int c = c0 + j * kNrThreads;
            if (c < total) {
                const int r = (int)(((float)c + 0.5f) * inv_lpr);
                const int ch = c - r * lpr;
                const int tensor = (int)(((float)r + 0.5f) * inv_lg);
                const int lg = r - tensor * a.layers * a.hkv;
                const int l = (int)(((float)lg + 0.5f) * inv_hkv);
                const size_t row = ((size_t)l * a.batch + b) * a.hkv + (lg - l * a.hkv);
                buf[j] = reinterpret_cast<const u32x4*>(static_cast<const char*>(tensor ? a.v_new : a.k_new) +
                                                        row * a.row_bytes)[ch];
                dsto[j] = ((row * a.cap + slot) * a.row_bytes) / 16 + ch + (tensor ? (size_t)1 << 62 : 0);
            }
        }
#pragma unroll
        for (int j = 0; j < kCopy; ++j) {
            const int c = c0 + j * kNrThreads;
            if (c < total) {
                const bool isv = (dsto[j] >> 62) != 0;
                reinterpret_cast<u32x4*>(isv ? a.v : a.k)[dsto[j] & (((size_t)1 << 62) - 1)] = buf[j];
            }
        }
    }
}

// The newcomer's K/V rows of every (layer, KV head) into its slot (nothing where slot[b] < 0).
__global__ __launch_bounds__(kThreads) void newcomer_rows_kernel(AppendArgs a, const int* slot) {
    const int lpr = a.row_bytes / 16;
    const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    const long long total = (long long)a.layers * a.batch * a.hkv * 2 * lpr;
    if (gid >= total) return;
    const int ch = (int)(gid % lpr);
    long long row = gid / lpr;  // (tensor, l, b, g) with tensor outermost
    const int tensor = (int)(row / ((long long)a.layers * a.batch * a.hkv));
    row %= (long long)a.layers * a.batch * a.hkv;  // == (l * batch + b) * hkv + g
    const int s = slot[(row / a.hkv) % a.batch];
    if (s < 0) return;
    const char* src = static_cast<const char*>(tensor ? a.v_new : a.k_new) + (size_t)row * a.row_bytes;
    char* dst = static_cast<char*>(tensor ? a.v : a.k) + ((size_t)row * a.cap + s) * a.row_bytes;
    reinterpret_cast<u32x4*>(dst)[ch] = reinterpret_cast<const u32x4*>(src)[ch];
}

// Placement of a refresh step's newcomer after the fold (steady steps: exactly one eviction, or none while
// the cache is under budget).  Workgroup (l, b): the sequence's single eviction from the fold's candidates
// (every workgroup of the sequence reduces them the same way), then the newcomer's K and V rows of layer l
// into its slot; workgroup (0, b) also moves its utility and position, and every workgroup writes its share
// of the decision.  Reads (candidates, the newcomer's rows at row n - 1 or in k_new / v_new) never overlap
// writes (rows and entries of the slot < n - 1).
constexpr int kPlaceThreads = 256;

__global__ __launch_bounds__(kPlaceThreads) void place_kernel(PlaceArgs a) {
    __shared__ Cand best[kPlaceThreads / kWave];
    const int l = blockIdx.x, b = blockIdx.y;
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    const int n = a.n;
    // this thread's 16-byte chunks of the newcomer's rows (tensor, KV head, chunk) are loaded first, so their
    // latency overlaps the candidates' reduction
    const int lpr = a.row_bytes / 16;
    const int total = 2 * a.hkv * lpr;
    constexpr int kPre = 2;
    u32x4 pre[kPre];
    auto src_of = [&](int c) {
        const int ch = c % lpr;
        const int g = (c / lpr) % a.hkv;
        const int tensor = c / (lpr * a.hkv);
        const size_t slab = ((size_t)l * a.batch + b) * a.hkv + g;
        return reinterpret_cast<const u32x4*>(static_cast<const char*>(tensor ? a.src_v : a.src_k) +
                                              (slab * a.src_slab_rows + a.src_row0) * a.row_bytes) + ch;
    };
#pragma unroll
    for (int j = 0; j < kPre; ++j)
        if (tid + j * kPlaceThreads < total) pre[j] = *src_of(tid + j * kPlaceThreads);
    int evicted = -1;
    if (n > a.budget) {
        const Cand* cb = a.cand + (size_t)b * a.ncand;
        Cand c{0xffffffffu, -1, -1};
        for (int i = tid; i < a.ncand; i += kPlaceThreads)
            if (evicts_before(cb[i], c)) c = cb[i];
#pragma unroll
        for (int o = kWave / 2; o >= 1; o >>= 1) {
            const Cand x = shfl_xor_cand(c, o);
            if (evicts_before(x, c)) c = x;
        }
        if (lane == 0) best[wave] = c;
        __syncthreads();
        c = best[0];
        for (int w = 1; w < kPlaceThreads / kWave; ++w)
            if (evicts_before(best[w], c)) c = best[w];
        evicted = c.idx;
    }
    const int slot = evicted == n - 1 ? -1 : (evicted >= 0 ? evicted : n - 1);
    if (a.keep_out) {
        const int per = (n + a.layers - 1) / a.layers;
        const int i1 = min(n, (l + 1) * per);
        for (int i = l * per + tid; i < i1; i += kPlaceThreads) a.keep_out[(size_t)b * a.cap + i] = i != evicted;
    }
    if (slot < 0) return;
    if (a.norms) {  // the newcomer's value norms of this layer, into the slot it takes
        const int nl = norm_lanes(a.row_bytes);
        for (int g = tid / nl; g < a.hkv; g += kPlaceThreads / nl) {
            const size_t slab = ((size_t)l * a.batch + b) * a.hkv + g;
            const float nrm = row_norm(static_cast<const char*>(a.src_v) + (slab * a.src_slab_rows + a.src_row0) *
                                       a.row_bytes, a.row_bytes, a.bf16 != 0, tid % nl);
            if (tid % nl == 0) a.norms[slab * a.cap + slot] = nrm;
        }
    }
    if (l == 0 && tid == 0 && slot != n - 1) {
        a.u[(size_t)b * a.cap + slot] = a.u[(size_t)b * a.cap + n - 1];
        a.pos[(size_t)b * a.cap + slot] = a.pos[(size_t)b * a.cap + n - 1];
    }
    // the source is the cache's own row n - 1 when src_row0 == n - 1 and src is the cache: nothing to move
    auto put = [&](int c, const u32x4& x) {
        const int ch = c % lpr;
        const int g = (c / lpr) % a.hkv;
        const int tensor = c / (lpr * a.hkv);
        const size_t slab = ((size_t)l * a.batch + b) * a.hkv + g;
        u32x4* dst = reinterpret_cast<u32x4*>(static_cast<char*>(tensor ? a.v : a.k) + (slab * a.cap + slot) * a.row_bytes) +
                     ch;
        if (src_of(c) != dst) *dst = x;
    };
#pragma unroll
    for (int j = 0; j < kPre; ++j)
        if (tid + j * kPlaceThreads < total) put(tid + j * kPlaceThreads, pre[j]);
    for (int c = tid + kPre * kPlaceThreads; c < total; c += kPlaceThreads) put(c, *src_of(c));
}

}  // namespace

hipError_t launch_place(const PlaceArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(place_kernel, dim3(a.layers, a.batch), dim3(kPlaceThreads), 0, s, a);
    return hipGetLastError();
}

// Where the newcomer's rows are copied depends on the prior policy.  Under the minimum prior the newcomer
// ties the lowest utility and, holding the newest position, is normally evicted at once: the decision kernel
// copies the rows itself when needed (6.0 us per step at the 8B shape, against 8.0 with a second launch that
// then has nothing to do).  Under the mean prior the newcomer is normally kept: one workgroup per sequence
// copies 128 KB of rows slowly, a kernel over all rows does it in a fraction (8.6 us against 11.0).
hipError_t launch_nonrefresh(const AppendArgs& a, uint8_t* keep_out, int budget, int* slot, hipStream_t s) {
    const int copy_in_decision = a.init_mode == 2;
    hipLaunchKernelGGL(nonrefresh_kernel, dim3(a.batch), dim3(kNrThreads), 0, s, a, keep_out, budget, slot,
                       copy_in_decision);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || copy_in_decision) return e;
    const long long threads = (long long)a.layers * a.batch * a.hkv * 2 * (a.row_bytes / 16);
    hipLaunchKernelGGL(newcomer_rows_kernel, dim3((unsigned)((threads + kThreads - 1) / kThreads)), dim3(kThreads), 0,
                       s, a, slot);
    return hipGetLastError();
}

hipError_t launch_move(const MoveArgs& a, hipStream_t s) {
    if (a.max_pairs <= 0) return hipSuccess;
    const int rows_per_block = kThreads / (a.row_bytes / 16) * kMoveUnroll;
    const long long bx = (a.max_pairs + rows_per_block - 1) / rows_per_block;
    const long long by = 2LL * a.layers * a.hkv;
    if (bx > 0x7fffffffLL || by > 65535 || a.batch > 65535) return hipErrorInvalidValue;
    hipLaunchKernelGGL(move_kernel, dim3((unsigned)bx, (unsigned)by, (unsigned)a.batch), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_append(const AppendArgs& a, hipStream_t s) {
    const long long threads = (long long)a.layers * a.batch * a.hkv * 2 * (a.row_bytes / 16);
    const long long rows = (long long)a.layers * a.batch * a.hkv;
    const int groups = kThreads / (a.row_bytes >= 256 ? 16 : a.row_bytes / 16);  // norm rows per block
    const long long blocks = a.batch + (threads + kThreads - 1) / kThreads + (a.norms ? (rows + groups - 1) / groups : 0);
    hipLaunchKernelGGL(append_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace ikv
