// End-of-step rebuild of every active cache, with staged recovery fused in.
//
// One workgroup per (layer, sequence).  It streams the unfreeze steps U_p of
// the n_t positions once and:
//   1. applies the recovery level chosen for the sequence (Sec. 3.6):
//        SR: remaining timer U_p - (t+1) > 1     ->  U_p = t+1
//        WR: p >= n_t - N and U_p > t+1          ->  U_p = t+1
//        FR: U_p > t+1                           ->  U_p = t+1
//   2. compacts the positions with U_p <= t+1 into the ascending active list
//      of step t+1 (Sec. 3.5: restored tokens attend again) and appends the
//      position n_t that the next token will take.
// A token frozen at step t' for d steps carries U = t' + d: stepping the
// timers of Algorithm 1's second loop is the comparison against t+1, so the
// per-step decrement pass over frozen storage disappears.
//
// The in-order compaction uses wave ballots: every thread owns 4 consecutive
// positions (one 16-byte load), mbcnt over 4 ballots gives the exclusive
// count inside the wave, and an LDS scan over the wave totals gives the
// offset inside the tile.
#include "kernels.h"

namespace asrkf {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;

__device__ __forceinline__ int lanes_below(unsigned long long mask) {
    return __builtin_amdgcn_mbcnt_hi((unsigned)(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo((unsigned)mask, 0));
}

__global__ void __launch_bounds__(kThreads)
compact_kernel(CompactArgs a) {
    __shared__ int wave_tot[kWaves];
    __shared__ int tile_base;

    const int inst = blockIdx.x;
    const int b = inst % a.B;
    const int n = a.plen[b] + a.t;            // positions after step t
    const int t1 = a.t + 1;
    const int level = a.forced_level >= 0 ? a.forced_level : (a.level ? a.level[b] : 0);
    int32_t* U = a.unfreeze + (size_t)inst * a.cap;
    int32_t* list = a.list + (size_t)inst * a.cap;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr_from = n - a.wr_last_N;
    const bool sr = level == 1, wr = level == 2, fr = level == 3;

    if (tid == 0) tile_base = 0;
    __syncthreads();

    for (int p0 = 0; p0 < n; p0 += 4 * kThreads) {
        const int p = p0 + 4 * tid;
        int u[4] = {0, 0, 0, 0};
        if (p + 3 < n) {
            const int4 v = *reinterpret_cast<const int4*>(U + p);
            u[0] = v.x; u[1] = v.y; u[2] = v.z; u[3] = v.w;
        } else {
            for (int k = 0; k < 4; ++k) if (p + k < n) u[k] = U[p + k];
        }
        // branch-free: one select per position, no short-circuit control flow
        bool flag[4];
        bool dirty = false;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int q = p + k;
            const bool live = q < n;
            const bool frozen_now = live & (u[k] > t1);
            const bool hit = frozen_now & ((sr & (u[k] > t1 + 1)) | (wr & (q >= wr_from)) | fr);
            u[k] = hit ? t1 : u[k];
            dirty |= hit;
            flag[k] = live & (u[k] <= t1);
        }
        if (dirty) {
            for (int k = 0; k < 4; ++k) if (p + k < n) U[p + k] = u[k];
        }
        unsigned long long bal[4];
        int before = 0, mine = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            bal[k] = __ballot(flag[k]);
            before += lanes_below(bal[k]);
            mine += flag[k];
        }
        if (lane == 63) wave_tot[wave] = before + mine;
        __syncthreads();
        int wave_off = 0, tile_tot = 0;
        for (int w = 0; w < kWaves; ++w) {
            const int c = wave_tot[w];
            wave_off += (w < wave) ? c : 0;
            tile_tot += c;
        }
        int out = tile_base + wave_off + before;
#pragma unroll
        for (int k = 0; k < 4; ++k) if (flag[k]) list[out++] = p + k;
        __syncthreads();
        if (tid == 0) tile_base += tile_tot;
        __syncthreads();
    }
    if (tid == 0) {
        list[tile_base] = n;                  // the next token's position
        a.n_active[inst] = tile_base + 1;
        atomicAdd(a.listed_total, (unsigned long long)(tile_base + 1));
    }
}

}  // namespace

hipError_t launch_compact(const CompactArgs& a, int n_instances, hipStream_t s) {
    hipLaunchKernelGGL(compact_kernel, dim3(n_instances), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace asrkf
