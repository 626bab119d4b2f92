// The two order-preserving scorer perturbations of Sec. 5.1 (implementation appendix "Per-step scoring"),
// applied to the step's score before the fold:
//   VNorm: each head's attention to token i is multiplied by |v_i| / mean_j |v_j|, the l2 norm of the token's
//          value row under that head's KV head over the mean norm of the slab's cached tokens;
//   entropy weighting: the layer's pooled score is multiplied by the entropy of that pooled distribution
//          over ln(n), one factor per layer and sequence.
// These kernels produce the norms (with the reciprocal of each slab's mean) and the entropy factors; the
// fold applies them while it sums the group sums r (which stay the plain attention).
#include "stream_lane.h"

namespace ikv {
namespace {

constexpr int kVThreads = 512;

// One workgroup per (layer, sequence, KV head) slab: a value row is read as 16-byte chunks by an aligned
// group of LPR lanes; a wave covers kRows x (64 / LPR) consecutive rows per pass, and the next pass's loads are
// issued before the current pass is reduced (raw buffer loads over the slab's live rows: reads past the end
// return zero and are not stored).  The sum of squares is reduced over the lane group with DPP; the wave's
// norms are gathered in its own LDS row and written as 16-byte stores (one per four rows instead of one 4-byte
// store per row, while V streams), and summed in a fixed order for the mean.
constexpr int kRows = 4;

template <typename T, int D>
__global__ __launch_bounds__(kVThreads) void vnorm_kernel(VariantArgs a) {
    using E = Elem<T>;
    using chunk_t = typename E::chunk_t;
    constexpr int EPC = E::kPerChunk, CH = D / EPC, LPR = CH >= 16 ? 16 : CH, CPL = CH / LPR;
    constexpr int GPW = kWave / LPR;             // row groups per wave
    constexpr int RPW = GPW * kRows;              // consecutive rows per wave and pass
    constexpr int kWavesV = kVThreads / kWave;
    constexpr int kPass = kWavesV * RPW;          // rows per pass
    constexpr int kRowBytes = D * (int)sizeof(T);
    static_assert(RPW % 4 == 0, "16-byte norm stores");
    __shared__ float part[kWavesV];
    __shared__ float stage[kWavesV][RPW];
    const size_t slab = blockIdx.x;
    const __amdgpu_buffer_rsrc_t vrs =
        raw_rsrc(static_cast<const T*>(a.v) + slab * a.cap * D, a.n * kRowBytes);
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int p = lane % LPR;
    const int grp = lane / LPR;
    // workspace norms (stride n_stride, padded to 64 rows): staged 16-byte stores; the caller's norm cache
    // (stride cap, no padding): one 4-byte store per live row
    const bool direct = a.norms_direct != 0;
    float* nrow = a.vnorm + slab * a.vnorm_stride;
    const __amdgpu_buffer_rsrc_t out = raw_rsrc(nrow, direct ? 0 : a.n_stride * 4);
    // row of (pass base, k) for this lane: the wave's block, then k-major, row groups innermost
    auto row_of = [&](int base, int k) { return base + wave * RPW + k * GPW + grp; };
    auto load = [&](int base, chunk_t (&c)[kRows][CPL]) {
#pragma unroll
        for (int k = 0; k < kRows; ++k)
#pragma unroll
            for (int cc = 0; cc < CPL; ++cc)
                c[k][cc] = __builtin_bit_cast(
                    chunk_t, __builtin_amdgcn_raw_buffer_load_b128(
                                 vrs, row_of(base, k) * kRowBytes + (p + cc * LPR) * 16, 0, kNonTemporal));
    };
    float sum = 0.0f;
    auto reduce = [&](int base, const chunk_t (&c)[kRows][CPL]) {
#pragma unroll
        for (int k = 0; k < kRows; ++k) {
            const float nr = row_norm_lanes<T, LPR, CPL>(c[k]);  // DPP inside the row's aligned lane group
            const int row = row_of(base, k);
            if (p == 0) {
                const float nrm = row < a.n ? nr : 0.0f;
                stage[wave][k * GPW + grp] = nrm;
                sum += nrm;
                if (direct && row < a.n) nrow[row] = nrm;
            }
        }
        if (direct) return;
        // the wave's RPW consecutive norms, 4 per lane (a group starting below n ends inside the padded stride,
        // a multiple of 64); the wave's own LDS row, so only the wave's order matters
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        const int first = base + wave * RPW;
        if (lane * 4 < RPW && first + lane * 4 < a.n)
            store_stream(out, (first + lane * 4) * 4, *reinterpret_cast<const f32x4*>(&stage[wave][lane * 4]));
    };
    chunk_t c0[kRows][CPL], c1[kRows][CPL];
    load(0, c0);
    for (int base = 0; base < a.n; base += 2 * kPass) {  // uniform trip count: every lane joins the DPP sums
        load(base + kPass, c1);
        reduce(base, c0);
        load(base + 2 * kPass, c0);
        reduce(base + kPass, c1);
    }
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) sum += __shfl_xor(sum, o, kWave);
    if (lane == 0) part[wave] = sum;
    __syncthreads();
    if (threadIdx.x == 0 && a.vnorm_inv_mean) {
        float tot = 0.0f;
        for (int w = 0; w < kWavesV; ++w) tot += part[w];
        a.vnorm_inv_mean[slab] = tot > 0.0f ? (float)a.n / tot : 0.0f;
    }
}

// The slab's n / (sum of its n value norms) from the caller's norm cache (VNorm without reading V).  With
// v_new set, row n - 1 is the step's newcomer, not cached yet: one lane group computes its norm from v_new
// (row_norm_lanes, as at append) and writes it to the cache, the others add the n - 1 cached norms.  The sum
// runs in a fixed order (thread-strided partial sums, a fixed butterfly, the waves in order), so the result
// is deterministic.
constexpr int kMThreads = 256;

template <typename T, int D>
__global__ __launch_bounds__(kMThreads) void vnorm_mean_kernel(VariantArgs a) {
    using chunk_t = typename Elem<T>::chunk_t;
    constexpr int CH = D / Elem<T>::kPerChunk, LPR = CH >= 16 ? 16 : CH, CPL = CH / LPR;
    __shared__ float part[kMThreads / kWave];
    __shared__ float newcomer;
    const size_t slab = blockIdx.x;
    float* nb = a.vnorm + slab * a.vnorm_stride;
    const int m = a.v_new ? a.n - 1 : a.n;  // cached rows whose norms are read
    if (a.v_new && threadIdx.x < LPR) {
        const chunk_t* row = reinterpret_cast<const chunk_t*>(static_cast<const T*>(a.v_new) + slab * D);
        chunk_t c[CPL];
#pragma unroll
        for (int cc = 0; cc < CPL; ++cc) c[cc] = row[threadIdx.x + cc * LPR];
        const float nrm = row_norm_lanes<T, LPR, CPL>(c);
        if (threadIdx.x == 0) {
            nb[a.n - 1] = nrm;
            newcomer = nrm;
        }
    }
    constexpr int kU = 4;  // loads in flight per thread
    float sum = 0.0f;
    int i = threadIdx.x;
    for (; i + (kU - 1) * kMThreads < m; i += kU * kMThreads) {
        float x[kU];
#pragma unroll
        for (int j = 0; j < kU; ++j) x[j] = nb[i + j * kMThreads];
#pragma unroll
        for (int j = 0; j < kU; ++j) sum += x[j];
    }
    for (; i < m; i += kMThreads) sum += nb[i];
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) sum += __shfl_xor(sum, o, kWave);
    if ((threadIdx.x & (kWave - 1)) == 0) part[threadIdx.x / kWave] = sum;
    __syncthreads();
    if (threadIdx.x == 0) {
        float tot = 0.0f;
        for (int w = 0; w < kMThreads / kWave; ++w) tot += part[w];
        if (a.v_new) tot += newcomer;
        a.vnorm_inv_mean[slab] = tot > 0.0f ? (float)a.n / tot : 0.0f;
    }
}

// One workgroup per (layer, sequence): s(i) = (1/H) sum of the r rows of the (layer, sequence); with S = sum_i s(i) the entropy of
// p = s / S is ln S - (1/S) sum_i s(i) ln s(i); divided by ln n (factor 1 when n = 1 or S = 0).  Each thread
// reads 4 consecutive tokens of every KV head per pass (rows are padded to a multiple of 64; the padding is
// masked), so a 32k-token slab takes 8 passes.
constexpr int kEThreads = 1024;

__global__ __launch_bounds__(kEThreads) void entropy_kernel(VariantArgs a) {
    __shared__ float ps[kEThreads / kWave], pe[kEThreads / kWave];
    const size_t lb = blockIdx.x;
    const float* rb = a.r + lb * a.r_groups * a.n_stride;
    float S = 0.0f, E = 0.0f;
    for (int i = threadIdx.x * 4; i < a.n; i += kEThreads * 4) {
        f32x4 s = {0.0f, 0.0f, 0.0f, 0.0f};
        for (int g = 0; g < a.r_groups; g += a.rblock) {  // blocks of rows as the fold adds them
            f32x4 t = *reinterpret_cast<const f32x4*>(rb + (size_t)g * a.n_stride + i);
            for (int j = 1; j < a.rblock; ++j)
                t += *reinterpret_cast<const f32x4*>(rb + (size_t)(g + j) * a.n_stride + i);
            s += t;
        }
        s *= a.inv_hq;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (i + j < a.n) {
                S += s[j];
                if (s[j] > 0.0f) E = fmaf(s[j], logf(s[j]), E);
            }
        }
    }
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        S += __shfl_xor(S, o, kWave);
        E += __shfl_xor(E, o, kWave);
    }
    if ((threadIdx.x & (kWave - 1)) == 0) {
        ps[threadIdx.x / kWave] = S;
        pe[threadIdx.x / kWave] = E;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        float st = 0.0f, et = 0.0f;
        for (int w = 0; w < kEThreads / kWave; ++w) {
            st += ps[w];
            et += pe[w];
        }
        a.entropy[lb] = (a.n > 1 && st > 0.0f) ? (logf(st) - et / st) / logf((float)a.n) : 1.0f;
    }
}

}  // namespace

hipError_t launch_vnorm(int dtype, int head_dim, const VariantArgs& a, hipStream_t s) {
    const dim3 grid((unsigned)((size_t)a.layers * a.batch * a.hkv));
    if (dtype == 0) {
        if (head_dim == 64) hipLaunchKernelGGL((vnorm_kernel<float, 64>), grid, dim3(kVThreads), 0, s, a);
        else hipLaunchKernelGGL((vnorm_kernel<float, 128>), grid, dim3(kVThreads), 0, s, a);
    } else {
        if (head_dim == 64) hipLaunchKernelGGL((vnorm_kernel<bf16_t, 64>), grid, dim3(kVThreads), 0, s, a);
        else hipLaunchKernelGGL((vnorm_kernel<bf16_t, 128>), grid, dim3(kVThreads), 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_vnorm_mean(int dtype, int head_dim, const VariantArgs& a, hipStream_t s) {
    const dim3 grid((unsigned)((size_t)a.layers * a.batch * a.hkv));
    if (dtype == 0) {
        if (head_dim == 64) hipLaunchKernelGGL((vnorm_mean_kernel<float, 64>), grid, dim3(kMThreads), 0, s, a);
        else hipLaunchKernelGGL((vnorm_mean_kernel<float, 128>), grid, dim3(kMThreads), 0, s, a);
    } else {
        if (head_dim == 64) hipLaunchKernelGGL((vnorm_mean_kernel<bf16_t, 64>), grid, dim3(kMThreads), 0, s, a);
        else hipLaunchKernelGGL((vnorm_mean_kernel<bf16_t, 128>), grid, dim3(kMThreads), 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_entropy(const VariantArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(entropy_kernel, dim3((unsigned)((size_t)a.layers * a.batch)), dim3(kEThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace ikv
