// Entropy of the next-token distribution and the recovery ladder (Sec. 3.6).
//
// One workgroup per sequence, one pass over the V logits.  Each thread keeps
// (m, S, T) with S = sum e^(x-m) and T = sum e^(x-m) (x-m) over its logits;
// the triples are merged across the block, and
//     H = ln S - T / S          (nats, softmax at temperature 1)
//     p_max = 1 / S.
// Thread 0 then updates the sequence's escalation count (one level per
// consecutive spike step, reset by a calm step) and writes the level that the
// end-of-step compaction applies: 1 SR, 2 WR, 3 FR; a count above 3 also
// records a Rewalk Regeneration request.
#include "kernels.h"

namespace asrkf {
namespace {

constexpr int kThreads = 1024;

struct Triple {
    float m, S, T;
};

__device__ __forceinline__ void push(Triple& a, float x) {
    if (x > a.m) {
        const float d = a.m - x;              // <= 0 (or -inf when empty)
        const float e = (a.S > 0.f) ? expf(d) : 0.f;
        a.T = (a.S > 0.f) ? e * (a.T + d * a.S) : 0.f;
        a.S = a.S * e + 1.f;
        a.m = x;
    } else {
        const float d = x - a.m;
        const float e = expf(d);
        a.S += e;
        a.T = fmaf(e, d, a.T);
    }
}

__device__ __forceinline__ Triple merge(const Triple& a, const Triple& b) {
    if (b.S == 0.f) return a;
    if (a.S == 0.f) return b;
    const float m = fmaxf(a.m, b.m);
    const float da = a.m - m, db = b.m - m;
    const float ea = expf(da), eb = expf(db);
    Triple r;
    r.m = m;
    r.S = ea * a.S + eb * b.S;
    r.T = ea * (a.T + da * a.S) + eb * (b.T + db * b.S);
    return r;
}

__global__ void __launch_bounds__(kThreads)
entropy_kernel(EntropyArgs a) {
    __shared__ Triple part[kThreads / 64];
    const int b = blockIdx.x;
    const float* x = a.logits + (size_t)b * a.V;
    Triple acc{-INFINITY, 0.f, 0.f};
    const bool vec = ((reinterpret_cast<uintptr_t>(x) & 15) == 0);
    int v0 = 0;
    if (vec) {
        const int nv = a.V / 4;
        for (int i = threadIdx.x; i < nv; i += kThreads) {
            const float4 f = reinterpret_cast<const float4*>(x)[i];
            push(acc, f.x); push(acc, f.y); push(acc, f.z); push(acc, f.w);
        }
        v0 = nv * 4;
    }
    for (int i = v0 + threadIdx.x; i < a.V; i += kThreads) push(acc, x[i]);

    for (int o = 32; o > 0; o >>= 1) {
        Triple other{__shfl_xor(acc.m, o), __shfl_xor(acc.S, o), __shfl_xor(acc.T, o)};
        acc = merge(acc, other);
    }
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        Triple r = part[0];
        for (int w = 1; w < kThreads / 64; ++w) r = merge(r, part[w]);
        const float H = logf(r.S) - r.T / r.S;
        const float pmax = 1.f / r.S;
        a.entropy[b] = H;
        a.pmax[b] = pmax;
        int level = 0;
        if (a.mode == 0) {
            const bool spike = (H > a.theta_H) || (a.theta_p > 0.f && pmax < a.theta_p);
            const int esc = spike ? a.escalation[b] + 1 : 0;
            a.escalation[b] = esc;
            level = min(esc, 3);
            if (esc > 3) atomicAdd(a.rr_requests, 1ull);
        } else if (a.mode >= 1 && a.mode <= 3) {
            level = a.mode;
        }
        a.level[b] = level;
        if (level > 0) atomicAdd(a.recoveries + level, 1ull);
    }
}

}  // namespace

hipError_t launch_entropy(const EntropyArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(entropy_kernel, dim3(a.B), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace asrkf
