// Relevance by attention weight (the softmax reading of Eq. 2): a token's
// score is the share of attention it received, averaged over the heads,
//     s_j = (1/H) sum_h softmax_j(q_h . k_j / sqrt(d)),
// which needs each head's normaliser over the whole active set.  The
// attention kernel keeps y_hj = q_h . k_j * log2(e)/sqrt(d) of every listed
// token, the split combine leaves (M_h, L_h) = (max, sum of 2^(y - M)), and
// this kernel forms H * s_j = sum_h 2^(y_hj - M_h) / L_h.  It then writes the
// token's score flag (s_j < tau, layer scope) or adds the score to the
// token's sum over layers (token scope); the freeze loop of Algorithm 1 runs
// at the end of the step on either.  One thread per listed token.
#include "kernels.h"

namespace asrkf {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxHeads = 256;

__global__ void __launch_bounds__(kThreads)
weight_relevance_kernel(RelevanceArgs a) {
    __shared__ float M[kMaxHeads], invL[kMaxHeads];
    const int b = blockIdx.y;
    for (int h = threadIdx.x; h < a.Hq; h += kThreads) {
        M[h] = a.norm[((size_t)b * a.Hq + h) * 2];
        invL[h] = 1.f / a.norm[((size_t)b * a.Hq + h) * 2 + 1];
    }
    __syncthreads();
    const int n = a.n_active[b];
    const size_t row = (size_t)b * a.cap;
    for (int i = blockIdx.x * kThreads + threadIdx.x; i < n; i += gridDim.x * kThreads) {
        const float* y = a.xlog + (row + i) * a.Hq;
        float s = 0.f;
        for (int h = 0; h < a.Hq; ++h) s = fmaf(__builtin_amdgcn_exp2f(y[h] - M[h]), invL[h], s);
        const int pos = a.list[row + i];
        const size_t o = row + pos;
        if (a.scope_token) a.rel_acc[o] = a.first_layer ? s : a.rel_acc[o] + s;
        else a.flag[o] = (s < a.tau_H ? 1 : 0) | (fabsf(s - a.tau_H) < a.margin_H ? 2 : 0);
    }
}

}  // namespace

hipError_t launch_weight_relevance(const RelevanceArgs& a, hipStream_t s) {
    if (a.Hq > kMaxHeads) return hipErrorInvalidValue;
    hipLaunchKernelGGL(weight_relevance_kernel, dim3(64, a.B), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace asrkf
