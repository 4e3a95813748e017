// Entropy of the next-token distribution and the recovery ladder (Sec. 3.6).
//
// a.split workgroups per sequence, one pass over the V logits.  Each
// thread forms (m, S, T) with S = sum e^(x-m) and T = sum e^(x-m) (x-m) over
// its logits (all loads of a round in flight together, the round's maximum
// first); the triples are merged across the block and stored.  The last
// block of a sequence to finish (a per-sequence ticket) loads the stored
// triples, one per lane, merges them in a fixed lane tree and forms
//     H = ln S - T / S          (nats, softmax at temperature 1)
//     p_max = 1 / S,
// A logit of -inf has probability 0 and adds nothing; a row with no finite
// logit has no distribution: its entropy is NaN and it triggers nothing.
// Then the kernel updates the sequence's escalation count (one level per consecutive
// spike step, reset by a calm step) and writes the level that the end-of-step
// compaction applies: 1 SR, 2 WR, 3 FR; a count above 3 also records a
// Rewalk Regeneration request.
#include "kernels.h"

namespace asrkf {
namespace {

constexpr int kThreads = 256;

struct Triple {
    float m, S, T;
};

__device__ __forceinline__ Triple merge(const Triple& a, const Triple& b) {
    if (b.S == 0.f) return a;
    if (a.S == 0.f) return b;
    constexpr float kLog2e = 1.4426950408889634f;
    const float m = fmaxf(a.m, b.m);
    const float da = a.m - m, db = b.m - m;
    const float ea = __builtin_amdgcn_exp2f(da * kLog2e), eb = __builtin_amdgcn_exp2f(db * kLog2e);
    Triple r;
    r.m = m;
    r.S = ea * a.S + eb * b.S;
    r.T = ea * (a.T + da * a.S) + eb * (b.T + db * b.S);
    return r;
}

// (m, S, T) of a thread's logits: its maximum first, then one pass with
// e = exp(x - m) (as exp2 of pre-scaled differences), no data-dependent branch.
template <int N>
__device__ __forceinline__ Triple triple_of(const float (&x)[N], const bool (&ok)[N]) {
    constexpr float kLog2e = 1.4426950408889634f;
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < N; ++i) m = ok[i] ? fmaxf(m, x[i]) : m;
    // no finite logit: an empty triple (a -inf logit has probability 0)
    if (m == -INFINITY) return Triple{-INFINITY, 0.f, 0.f};
    float S = 0.f, T = 0.f;
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const float d = x[i] - m;
        const float e = ok[i] ? __builtin_amdgcn_exp2f(d * kLog2e) : 0.f;
        S += e;
        // a term with e = 0 adds nothing (0 ln 0 = 0), also where d = -inf
        T = fmaf(e, (ok[i] && e > 0.f) ? d : 0.f, T);
    }
    return Triple{m, S, T};
}

constexpr int kVec = 4;             // float4 loads per thread per round

__global__ void __launch_bounds__(kThreads)
entropy_kernel(EntropyArgs a) {
    __shared__ Triple part[kThreads / 64];
    __shared__ int last;
    const int b = blockIdx.y;
    const int sp = blockIdx.x;
    const float* x = a.logits + (size_t)b * a.V;
    Triple acc{-INFINITY, 0.f, 0.f};
    if (((reinterpret_cast<uintptr_t>(x) & 15) == 0) && (a.V % 4 == 0)) {
        const int n4 = a.V / 4;
        const int i0 = (int)((int64_t)sp * n4 / a.split), i1 = (int)((int64_t)(sp + 1) * n4 / a.split);
        // all of a round's loads are issued before any of them is used
        for (int base = i0; base < i1; base += kThreads * kVec) {
            float v[4 * kVec];
            bool ok[4 * kVec];
#pragma unroll
            for (int u = 0; u < kVec; ++u) {
                const int i = base + u * kThreads + threadIdx.x;
                const bool in = i < i1;
                typedef float f4 __attribute__((ext_vector_type(4)));
                const f4 f = in ? __builtin_nontemporal_load(reinterpret_cast<const f4*>(x) + i)
                                : f4{0.f, 0.f, 0.f, 0.f};
                v[4 * u] = f.x; v[4 * u + 1] = f.y; v[4 * u + 2] = f.z; v[4 * u + 3] = f.w;
                ok[4 * u] = ok[4 * u + 1] = ok[4 * u + 2] = ok[4 * u + 3] = in;
            }
            acc = merge(acc, triple_of(v, ok));
        }
    } else {
        const int i0 = (int)((int64_t)sp * a.V / a.split), i1 = (int)((int64_t)(sp + 1) * a.V / a.split);
        for (int i = i0 + threadIdx.x; i < i1; i += kThreads) {
            const float v[1] = {x[i]};
            const bool ok[1] = {true};
            acc = merge(acc, triple_of(v, ok));
        }
    }
    for (int o = 32; o > 0; o >>= 1) {
        Triple other{__shfl_xor(acc.m, o), __shfl_xor(acc.S, o), __shfl_xor(acc.T, o)};
        acc = merge(acc, other);
    }
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        Triple r = part[0];
        for (int w = 1; w < kThreads / 64; ++w) r = merge(r, part[w]);
        float* dst = a.partial + ((size_t)b * a.split + sp) * 3;
        __hip_atomic_store(dst, r.m, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(dst + 1, r.S, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(dst + 2, r.T, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        // the device-scope stores above have completed before the ticket is taken,
        // so no cache-wide write-back is needed
        __builtin_amdgcn_s_waitcnt(0);
        last = (__hip_atomic_fetch_add(a.ticket + b, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                == a.split - 1);
    }
    __syncthreads();
    if (!last || threadIdx.x >= 64) return;
    // the blocks' triples, one per lane, read at device scope (they may sit in
    // another XCD's L2); merged in a fixed lane tree, so every run rounds alike
    static_assert(kEntropySplitMax <= 64, "one triple per lane");
    const float* src = a.partial + (size_t)b * a.split * 3;
    const int k = threadIdx.x;
    Triple r{-INFINITY, 0.f, 0.f};
    if (k < a.split) {
        r.m = __hip_atomic_load(src + 3 * k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        r.S = __hip_atomic_load(src + 3 * k + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        r.T = __hip_atomic_load(src + 3 * k + 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    for (int o = 1; o < 64; o <<= 1) {
        Triple other{__shfl_xor(r.m, o), __shfl_xor(r.S, o), __shfl_xor(r.T, o)};
        r = (k & o) ? merge(other, r) : merge(r, other);
    }
    if (k != 0) return;
    a.ticket[b] = 0;                           // ready for the next step
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

}  // namespace

hipError_t launch_entropy(const EntropyArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(entropy_kernel, dim3(a.split, a.B), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace asrkf
