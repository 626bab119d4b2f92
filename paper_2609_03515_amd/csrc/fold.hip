// Layer fold of the step scores into the running utility (Eq. 2-4, implementation appendix "Layer scoring").
//
// The sequential EMA over layers l = 1..K, u <- alpha u + (1 - alpha) s_l, is linear: it equals
// u <- alpha^K u + sum_l (1 - alpha) alpha^(K-l) s_l (the weights the appendix states).  The host passes the
// prior weight and the per-layer weights (also for the single-step and cumulative rules), so the layers can
// be reduced in parallel.  A workgroup covers 32 tokens of one sequence: each thread reads four consecutive
// tokens (16-byte loads) of the group sums r of one layer slice (one row per KV head, or per block of KV heads
// the scorer already added), weights them, and the
// partial sums of the 32 layer slices are added in a fixed order, so the result is deterministic.  On request
// the workgroup also reports the first of its tokens to leave under the single-eviction order (u ascending,
// position descending), from which the placement kernel takes a steady step's one eviction.
#include "kernels.h"
#include "kv_common.h"

namespace ikv {
namespace {

constexpr int kQuads = 8;          // 4-token groups per workgroup (32 tokens)
constexpr int kSlices = 32;        // layer slices per workgroup
constexpr int kThreads = kQuads * kSlices;

__global__ __launch_bounds__(kThreads) void fold_kernel(FoldArgs a) {
    __shared__ float partial[kSlices][kQuads * 4];
    __shared__ float partial_raw[kSlices][kQuads * 4];
    const int quad = threadIdx.x % kQuads;
    const int slice = threadIdx.x / kQuads;
    const int b = blockIdx.y;
    const int tok0 = blockIdx.x * (kQuads * 4) + quad * 4;  // r rows are padded to a multiple of 64
    f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
    f32x4 racc = {0.0f, 0.0f, 0.0f, 0.0f};  // rank trace: sum over layers of the plain group sums
    // wave 0's token (lane < 32): its utility and position are read now, their latency overlapping the layers'
    const int tok = blockIdx.x * (kQuads * 4) + threadIdx.x;
    const bool own = threadIdx.x < kQuads * 4 && tok < a.n;
    const bool newcomer = own && a.new_pos >= 0 && tok == a.n - 1;  // refresh prior 0, position not yet stored
    float u_old = 0.0f;
    int32_t p_old = 0;
    if (own && !newcomer) {
        u_old = a.u[(size_t)b * a.cap + tok];
        if (a.cand) p_old = a.pos[(size_t)b * a.cap + tok];
    }
    if (tok0 < a.n) {
        for (int l = slice; l < a.layers; l += kSlices) {
            const float* rl = a.r + ((size_t)(l * a.batch + b) * a.r_groups) * a.n_stride + tok0;
            f32x4 s = {0.0f, 0.0f, 0.0f, 0.0f};
            if (a.vnorm) {  // r_groups == hkv: one row per KV head
                // VNorm: each KV head's group sum times the token's value-norm factor norm / mean norm
                // (factor 1 where the slab's norms are all zero)
                // norms in the workspace (stride n_stride, rows padded to 64: 16-byte loads) or in the caller's
                // norm cache (stride cap, unpadded: the live rows only, one by one)
                const float* nl = a.vnorm + ((size_t)(l * a.batch + b) * a.hkv) * a.vnorm_stride + tok0;
                const float* il = a.vnorm_inv_mean + (size_t)(l * a.batch + b) * a.hkv;
                const bool padded = a.vnorm_stride == a.n_stride;
                f32x4 plain = {0.0f, 0.0f, 0.0f, 0.0f};
                for (int g = 0; g < a.hkv; ++g) {
                    const f32x4 rg = *reinterpret_cast<const f32x4*>(rl + (size_t)g * a.n_stride);
                    const float im = il[g];
                    const float* ng = nl + (size_t)g * a.vnorm_stride;
                    f32x4 nv;
                    if (padded) {
                        nv = *reinterpret_cast<const f32x4*>(ng);
                    } else {
#pragma unroll
                        for (int j = 0; j < 4; ++j) nv[j] = tok0 + j < a.n ? ng[j] : 0.0f;
                    }
                    const f32x4 f = im > 0.0f ? nv * im : f32x4{1.0f, 1.0f, 1.0f, 1.0f};
                    s += rg * f;
                    plain += rg;
                }
                racc += plain;
            } else {
                // block sums first, then the blocks in order
                for (int g = 0; g < a.r_groups; g += a.rblock) {
                    f32x4 t = *reinterpret_cast<const f32x4*>(rl + (size_t)g * a.n_stride);
                    for (int j = 1; j < a.rblock; ++j)
                        t += *reinterpret_cast<const f32x4*>(rl + (size_t)(g + j) * a.n_stride);
                    s += t;
                }
                racc += s;
            }
            s *= a.inv_hq;
            if (a.entropy) s *= a.entropy[l * a.batch + b];  // entropy weighting: one factor per layer and sequence
            if (a.s_out) {
                float* so = a.s_out + ((size_t)l * a.batch + b) * a.n + tok0;
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (tok0 + j < a.n) so[j] = s[j];
            }
            acc += a.w[l] * s;
        }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        partial[slice][quad * 4 + j] = acc[j];
        partial_raw[slice][quad * 4 + j] = racc[j];
    }
    __syncthreads();
    if (threadIdx.x >= kWave) return;
    // wave 0: one token per lane (lanes >= 32 hold none) and the workgroup's eviction candidate
    EvictCand c{0xffffffffu, -1, -1};
    if (own) {
        float tot = 0.0f;
        for (int sl = 0; sl < kSlices; ++sl) tot += partial[sl][threadIdx.x];
        const float un = fmaf(a.prior_w, u_old, tot);
        a.u[(size_t)b * a.cap + tok] = un;
        if (newcomer) a.pos[(size_t)b * a.cap + tok] = a.new_pos;
        if (a.cand) c = EvictCand{float_key(un), newcomer ? a.new_pos : p_old, tok};
        if (a.raw) {
            float rt = 0.0f;
            for (int sl = 0; sl < kSlices; ++sl) rt += partial_raw[sl][threadIdx.x];
            a.raw[(size_t)b * a.cap + tok] = rt * a.raw_scale;
        }
    }
    if (!a.cand) return;
#pragma unroll
    for (int o = kQuads * 2; o >= 1; o >>= 1) {
        const EvictCand x = shfl_xor_cand(c, o);
        if (evicts_before(x, c)) c = x;
    }
    if (threadIdx.x == 0) a.cand[(size_t)b * gridDim.x + blockIdx.x] = c;
}

}  // namespace

int fold_groups(int n) { return (n + kQuads * 4 - 1) / (kQuads * 4); }

hipError_t launch_fold(const FoldArgs& a, hipStream_t s) {
    dim3 grid(fold_groups(a.n), a.batch);
    hipLaunchKernelGGL(fold_kernel, grid, dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace ikv
