// Row copies between the device KV cache and the pinned host store (spill
// mode; Sec. 3.2 moves frozen tokens' KV off the GPU and back).
//
// The lists of rows to move are made on the device by the end-of-step
// compaction, so the host never learns which tokens move: each launch walks
// the per-(layer, sequence) lists it is given and copies every listed token's
// K row and V row (n_kv_heads * head_dim elements each, contiguous in both
// stores) one wave per token, 16 bytes per lane.  The host store is
// position-indexed, the device cache row-indexed.  Loads of a token's K and
// V pieces are issued before its stores, so each wave keeps two rows in
// flight over the host link.
#include "kernels.h"

namespace asrkf {
namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / 64;
constexpr int kBlocksPerLaunch = 1024;

__global__ void __launch_bounds__(kThreads)
xfer_kernel(XferArgs a) {
    const int inst = a.inst0 + blockIdx.y;
    const int n = a.count[inst];
    const int lane = threadIdx.x & 63;
    const int w0 = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    const int wstride = gridDim.x * kWavesPerBlock;
    const int32_t* pos = a.pos + (size_t)inst * a.cap;
    const int32_t* row = a.row + (size_t)inst * a.cap;
    const size_t host0 = (size_t)inst * a.cap;
    const size_t dev0 = (size_t)inst * a.pool_rows;
    for (int i = w0; i < n; i += wstride) {
        const size_t h = (host0 + (size_t)pos[i]) * a.row_bytes;
        const size_t d = (dev0 + (size_t)row[i]) * a.row_bytes;
        const char* ks = a.to_host ? a.kpool + d : a.khost + h;
        const char* vs = a.to_host ? a.vpool + d : a.vhost + h;
        char* kd = a.to_host ? a.khost + h : a.kpool + d;
        char* vd = a.to_host ? a.vhost + h : a.vpool + d;
        for (int o = lane * 16; o < a.row_bytes; o += 64 * 16) {
            const uint4 kx = *reinterpret_cast<const uint4*>(ks + o);
            const uint4 vx = *reinterpret_cast<const uint4*>(vs + o);
            *reinterpret_cast<uint4*>(kd + o) = kx;
            *reinterpret_cast<uint4*>(vd + o) = vx;
        }
    }
}

// Test hook: one wave that waits, without touching memory, until the given
// number of 100 MHz real-time ticks has passed.  It always ends.
__global__ void __launch_bounds__(64) delay_kernel(uint64_t ticks) {
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    while (__builtin_amdgcn_s_memrealtime() - t0 < ticks) __builtin_amdgcn_s_sleep(100);
}

}  // namespace

hipError_t launch_delay(int microseconds, hipStream_t s) {
    if (microseconds <= 0) return hipSuccess;
    hipLaunchKernelGGL(delay_kernel, dim3(1), dim3(64), 0, s, (uint64_t)microseconds * 100u);
    return hipGetLastError();
}

hipError_t launch_xfer(const XferArgs& a, int n_instances, hipStream_t s) {
    if (n_instances < 1 || a.row_bytes % 16) return hipErrorInvalidValue;
    constexpr int kMaxY = 32768;                  // instances per launch (grid y limit)
    for (int i0 = 0; i0 < n_instances; i0 += kMaxY) {
        XferArgs part = a;
        part.inst0 = a.inst0 + i0;
        const int ni = n_instances - i0 < kMaxY ? n_instances - i0 : kMaxY;
        const int gx = (kBlocksPerLaunch + ni - 1) / ni;
        hipLaunchKernelGGL(xfer_kernel, dim3(gx, ni), dim3(kThreads), 0, s, part);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace asrkf
