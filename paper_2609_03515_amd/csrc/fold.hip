// Layer fold of the step scores into the running utility (Eq. 2-4, implementation appendix "Layer scoring").
//
// The sequential EMA over layers l = 1..K, u <- alpha u + (1 - alpha) s_l, is linear: it equals
// u <- alpha^K u + sum_l (1 - alpha) alpha^(K-l) s_l (the weights the appendix states).  The host passes the
// prior weight and the per-layer weights (also for the single-step and cumulative rules), so the layers can
// be reduced in parallel: a workgroup covers 64 tokens of one sequence with four waves, each wave summing a
// quarter of the layers; partial sums are added in a fixed order, so results are deterministic.
#include "kernels.h"
#include "kv_common.h"

namespace ikv {
namespace {

constexpr int kTok = 64;
constexpr int kParts = 4;

__global__ __launch_bounds__(kTok * kParts) void fold_kernel(FoldArgs a) {
    __shared__ float partial[kParts][kTok];
    const int tl = threadIdx.x % kTok;
    const int part = threadIdx.x / kTok;
    const int b = blockIdx.y;
    const int tok = blockIdx.x * kTok + tl;
    const int per = (a.layers + kParts - 1) / kParts;
    const int l0 = part * per;
    const int l1 = min(a.layers, l0 + per);
    float acc = 0.0f;
    if (tok < a.n) {
        for (int l = l0; l < l1; ++l) {
            const float* rl = a.r + ((size_t)(l * a.batch + b) * a.hkv) * a.n_stride + tok;
            float s = 0.0f;
            for (int g = 0; g < a.hkv; ++g) s += rl[(size_t)g * a.n_stride];
            s *= a.inv_hq;
            if (a.s_out) a.s_out[((size_t)l * a.batch + b) * a.n + tok] = s;
            acc = fmaf(a.w[l], s, acc);
        }
    }
    partial[part][tl] = acc;
    __syncthreads();
    if (part == 0 && tok < a.n) {
        float tot = partial[0][tl];
#pragma unroll
        for (int q = 1; q < kParts; ++q) tot += partial[q][tl];
        float* up = a.u + (size_t)b * a.cap + tok;
        *up = fmaf(a.prior_w, *up, tot);
    }
}

}  // namespace

hipError_t launch_fold(const FoldArgs& a, hipStream_t s) {
    dim3 grid((a.n + kTok - 1) / kTok, a.batch);
    hipLaunchKernelGGL(fold_kernel, grid, dim3(kTok * kParts), 0, s, a);
    return hipGetLastError();
}

}  // namespace ikv
