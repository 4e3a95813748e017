// Active-set GQA flash-decode for gfx950, fused with the relevance score and
// the freeze schedule.
//
// Per launch (one layer, every sequence):
//   Eq. 1  o_h = softmax_j(q_h . k_j / sqrt(D)) v_j over the active list A_t;
//   Eq. 2  s_j = (1/Hq) sum_h |q_h . k_j| for every j in A_t;
//   Alg. 1 freeze loop: j outside the window with s_j < tau gets c_j += 1 and,
//          when d = floor(sqrt(c_j)/k) >= 1, the unfreeze step U_j = t + d.
//
// Work decomposition.  The active lists of all sequences, concatenated, are
// cut into equal contiguous ranges, one per workgroup of a persistent grid;
// each workgroup derives the cut from the active counts on the device and
// leaves one partial (m, l, acc) per sequence its range touches, at slot
// (workgroup + sequence).  A workgroup has one wave per KV head; all its waves
// walk the same tokens, so the per-token relevance is summed over every head
// in LDS and the schedule applied in place.
//
// Lane layout inside a wave: 8 token slots x 8 lanes.  The 8 lanes of a slot
// read one token's row of this KV head (D * elem bytes) as 16-byte pieces, so
// each load instruction moves 8 contiguous 128-byte segments.  The row is
// used by the G query heads of the group from registers (GQA sharing).  The
// dot products are reduced across the 8 lanes with DPP; each slot keeps its
// own running maximum so the inner loop has no cross-slot traffic; slots are
// merged once per sequence segment.
#include "kernels.h"

namespace asrkf {
namespace {

constexpr int kSlots = 8;      // tokens per wave per iteration
constexpr int kUnroll = 4;     // iterations per tile
constexpr int kMinPerGroup = 128;  // fewest tokens worth a workgroup

template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Sum over the 8 lanes of a slot; every lane of the slot gets the same bits.
__device__ __forceinline__ float slot_sum(float v) {
    v += dpp_mov<0xB1>(v);   // quad_perm [1,0,3,2]
    v += dpp_mov<0x4E>(v);   // quad_perm [2,3,0,1]
    v += dpp_mov<0x141>(v);  // row_half_mirror
    return v;
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                           __builtin_bit_cast(bf16x2_t, b), c, false);
}

template <bool BF16, int D>
struct Row {
    static constexpr int kElem = BF16 ? 2 : 4;
    static constexpr int kBytes = D * kElem;       // one token, one KV head
    static constexpr int kChunks = kBytes / 128;   // 16-byte pieces per lane
    static constexpr int kPerChunk = 16 / kElem;
    static constexpr int kPerLane = kChunks * kPerChunk;  // = D / 8
};

template <bool BF16, int D>
using Pieces = uint4[Row<BF16, D>::kChunks];      // the lane's 16-byte pieces of a row
template <bool BF16, int D>
using LaneAcc = float[Row<BF16, D>::kPerLane];    // the lane's accumulators of one head

// Dot product of the lane's part of a row with the lane's part of q.
template <bool BF16, int D>
__device__ __forceinline__ float lane_dot(const Pieces<BF16, D>& k, const Pieces<BF16, D>& q) {
    float x = 0.f;
#pragma unroll
    for (int c = 0; c < Row<BF16, D>::kChunks; ++c) {
        if constexpr (BF16) {
            x = dot2_bf16(k[c].x, q[c].x, x);
            x = dot2_bf16(k[c].y, q[c].y, x);
            x = dot2_bf16(k[c].z, q[c].z, x);
            x = dot2_bf16(k[c].w, q[c].w, x);
        } else {
            x = fmaf(__uint_as_float(k[c].x), __uint_as_float(q[c].x), x);
            x = fmaf(__uint_as_float(k[c].y), __uint_as_float(q[c].y), x);
            x = fmaf(__uint_as_float(k[c].z), __uint_as_float(q[c].z), x);
            x = fmaf(__uint_as_float(k[c].w), __uint_as_float(q[c].w), x);
        }
    }
    return x;
}

// acc[e] += p * v[e] over the lane's elements.
template <bool BF16, int D>
__device__ __forceinline__ void lane_axpy(LaneAcc<BF16, D>& acc, float p, const Pieces<BF16, D>& v) {
#pragma unroll
    for (int c = 0; c < Row<BF16, D>::kChunks; ++c) {
        const uint32_t w[4] = {v[c].x, v[c].y, v[c].z, v[c].w};
        if constexpr (BF16) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                acc[c * 8 + 2 * i] = fmaf(p, bf16_lo(w[i]), acc[c * 8 + 2 * i]);
                acc[c * 8 + 2 * i + 1] = fmaf(p, bf16_hi(w[i]), acc[c * 8 + 2 * i + 1]);
            }
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[c * 4 + i] = fmaf(p, __uint_as_float(w[i]), acc[c * 4 + i]);
        }
    }
}

// Element index (within the D of a row) of lane element e for dim-lane r.
template <bool BF16, int D>
__device__ __forceinline__ int lane_dim(int r, int e) {
    using R = Row<BF16, D>;
    const int c = e / R::kPerChunk, i = e % R::kPerChunk;
    return c * (128 / R::kElem) + r * R::kPerChunk + i;
}

// Token offsets of every sequence in the concatenated active lists:
// seq_off[b] = sum of n_active[b'] for b' < b, seq_off[B] = T.  Wave 0 scans.
__device__ void plan_ranges(const int32_t* n_active, int B, int32_t* seq_off) {
    const int tid = threadIdx.x;
    if (tid < 64) {
        const int per = (B + 63) / 64;
        const int b0 = tid * per;
        const int b1 = min(B, b0 + per);
        int mine = 0;
        for (int b = b0; b < b1; ++b) mine += n_active[b];
        int incl = mine;
        for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_up(incl, o);
            if (tid >= o) incl += y;
        }
        int run = incl - mine;
        for (int b = b0; b < b1; ++b) {
            seq_off[b] = run;
            run += n_active[b];
        }
        if (tid == 63) seq_off[B] = incl;
    }
    __syncthreads();
}

// Workgroups that share the work: enough that each gets kMinPerGroup tokens.
__device__ __forceinline__ int active_groups(int T, int grid) {
    return max(1, min(grid, (T + kMinPerGroup - 1) / kMinPerGroup));
}

// Workgroup holding token x of the concatenated lists when T tokens are cut
// into G ranges [floor(w T / G), floor((w+1) T / G)).
__device__ __forceinline__ int group_of(int64_t x, int64_t T, int64_t G) {
    return (int)(((x + 1) * G - 1) / T);
}

template <bool BF16, int D, int G>
__global__ void __launch_bounds__(512)
attention_kernel(AttnArgs a) {
    using R = Row<BF16, D>;
    constexpr int NC = R::kChunks;
    constexpr int EL = R::kPerLane;

    extern __shared__ int32_t lds[];
    int32_t* seq_off = lds;                           // [B + 1]
    int32_t* pos_lds = lds + ((a.B + 1 + 3) & ~3);    // [kChunkMax]
    float* rel_lds = reinterpret_cast<float*>(pos_lds + kChunkMax);  // [Hkv][kChunkMax]

    plan_ranges(a.n_active, a.B, seq_off);
    const int T = seq_off[a.B];
    const int Gn = active_groups(T, gridDim.x);
    if (blockIdx.x == 0) {
        for (int b = threadIdx.x; b < a.B; b += blockDim.x) {
            const int s0 = seq_off[b], s1 = seq_off[b + 1];
            a.slot_first[b] = s1 > s0 ? group_of(s0, T, Gn) + b : 0;
            a.slot_end[b] = s1 > s0 ? group_of(s1 - 1, T, Gn) + b + 1 : 0;
        }
    }
    const int w = blockIdx.x;
    if (w >= Gn) return;

    const int lane = threadIdx.x & 63;
    const int g = threadIdx.x >> 6;          // KV head of this wave
    const int slot = lane >> 3;
    const int r = lane & 7;
    const size_t row_stride = (size_t)a.Hkv * R::kBytes;   // bytes per token (all KV heads)

    int lo = (int)((int64_t)w * T / Gn);
    const int hi = (int)((int64_t)(w + 1) * T / Gn);
    int b = 0;
    {
        int l0 = 0, h0 = a.B - 1;             // last b with seq_off[b] <= lo
        while (l0 < h0) {
            const int mid = (l0 + h0 + 1) >> 1;
            if (seq_off[mid] <= lo) l0 = mid; else h0 = mid - 1;
        }
        b = l0;
    }

    while (lo < hi) {
        while (seq_off[b + 1] <= lo) ++b;     // skip sequences with nothing listed
        const int nb = seq_off[b + 1] - seq_off[b];
        const int i0 = lo - seq_off[b];
        const int i1 = min(hi, seq_off[b + 1]) - seq_off[b];
        const int n_pos = a.plen[b] + a.t;       // positions after the append
        const int new_pos = n_pos - 1;
        const int32_t* list_b = a.list + (size_t)b * a.cap;

        // append: the workgroup holding the new position copies it into the cache
        if (i1 == nb) {
            const size_t dst = ((size_t)b * a.cap + new_pos) * row_stride;
            const size_t src = (size_t)b * row_stride;
            for (size_t o = threadIdx.x * 16; o < row_stride; o += blockDim.x * 16) {
                *reinterpret_cast<uint4*>((char*)a.kpool_w + dst + o) =
                    *reinterpret_cast<const uint4*>((const char*)a.knew + src + o);
                *reinterpret_cast<uint4*>((char*)a.vpool_w + dst + o) =
                    *reinterpret_cast<const uint4*>((const char*)a.vnew + src + o);
            }
        }

        // query heads g*G .. g*G+G-1, this lane's elements
        uint4 qr[G][NC];
        {
            const char* qb = (const char*)a.q + ((size_t)b * a.Hq + (size_t)g * G) * R::kBytes;
#pragma unroll
            for (int h = 0; h < G; ++h)
#pragma unroll
                for (int c = 0; c < NC; ++c)
                    qr[h][c] = *reinterpret_cast<const uint4*>(qb + h * R::kBytes + c * 128 + r * 16);
        }

        float m[G], l[G], acc[G][EL];
#pragma unroll
        for (int h = 0; h < G; ++h) {
            m[h] = -INFINITY;
            l[h] = 0.f;
#pragma unroll
            for (int e = 0; e < EL; ++e) acc[h][e] = 0.f;
        }

        const char* kbase = (const char*)a.kpool + (size_t)b * a.cap * row_stride + g * R::kBytes;
        const char* vbase = (const char*)a.vpool + (size_t)b * a.cap * row_stride + g * R::kBytes;
        const char* knew_row = (const char*)a.knew + ((size_t)b * a.Hkv + g) * R::kBytes;
        const char* vnew_row = (const char*)a.vnew + ((size_t)b * a.Hkv + g) * R::kBytes;
        const int wedge = n_pos - a.window_K;    // positions < wedge are outside the window

        for (int c0 = i0; c0 < i1; c0 += kChunkMax) {
            const int len = min(kChunkMax, i1 - c0);
            for (int i = threadIdx.x; i < len; i += blockDim.x) pos_lds[i] = list_b[c0 + i];
            __syncthreads();

            for (int base = 0; base < len; base += kSlots * kUnroll) {
                uint4 kr[kUnroll][NC], vr[kUnroll][NC];
                bool valid[kUnroll];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) {
                    const int idx = base + u * kSlots + slot;
                    valid[u] = idx < len;
                    const int p = pos_lds[valid[u] ? idx : 0];
                    const char* kp = (p == new_pos) ? knew_row : kbase + (size_t)p * row_stride;
                    const char* vp = (p == new_pos) ? vnew_row : vbase + (size_t)p * row_stride;
#pragma unroll
                    for (int c = 0; c < NC; ++c) {
                        kr[u][c] = *reinterpret_cast<const uint4*>(kp + c * 128 + r * 16);
                        vr[u][c] = *reinterpret_cast<const uint4*>(vp + c * 128 + r * 16);
                    }
                }
                float y[kUnroll][G];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) {
                    float rel = 0.f;
#pragma unroll
                    for (int h = 0; h < G; ++h) {
                        const float x = slot_sum(lane_dot<BF16, D>(kr[u], qr[h]));
                        rel += fabsf(x);
                        y[u][h] = valid[u] ? x * a.scale_log2 : -INFINITY;
                    }
                    if (valid[u] && r == 0) rel_lds[g * kChunkMax + base + u * kSlots + slot] = rel;
                }
                // per-slot running maximum; rescale only when some slot's maximum grows
#pragma unroll
                for (int h = 0; h < G; ++h) {
                    float mt = m[h];
#pragma unroll
                    for (int u = 0; u < kUnroll; ++u) mt = fmaxf(mt, y[u][h]);
                    if (__any(mt > m[h])) {
                        const float sc = (mt > m[h]) ? exp2f(m[h] - mt) : 1.f;
                        l[h] *= sc;
#pragma unroll
                        for (int e = 0; e < EL; ++e) acc[h][e] *= sc;
                        m[h] = mt;
                    }
                }
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) {
#pragma unroll
                    for (int h = 0; h < G; ++h) {
                        const float p = valid[u] ? exp2f(y[u][h] - m[h]) : 0.f;
                        l[h] += p;
                        lane_axpy<BF16, D>(acc[h], p, vr[u]);
                    }
                }
            }
            __syncthreads();

            // freeze loop over this chunk: relevance summed over KV heads in fixed order
            for (int i = threadIdx.x; i < len; i += blockDim.x) {
                const int p = pos_lds[i];
                if (p >= wedge) continue;
                float sH = 0.f;
                for (int gg = 0; gg < a.Hkv; ++gg) sH += rel_lds[gg * kChunkMax + i];
                if (sH < a.tau_H) {
                    const size_t o = (size_t)b * a.cap + p;
                    const int c = a.count[o] + 1;
                    a.count[o] = c;
                    const int d = a.dur[min(c, a.dur_len - 1)];
                    if (d >= 1) a.unfreeze[o] = a.t + d;
                }
            }
            __syncthreads();
        }

        // merge the 8 slots: common maximum, then sums over lanes r, r+8, ..., r+56
#pragma unroll
        for (int h = 0; h < G; ++h) {
            float mm = m[h];
            mm = fmaxf(mm, __shfl_xor(mm, 8));
            mm = fmaxf(mm, __shfl_xor(mm, 16));
            mm = fmaxf(mm, __shfl_xor(mm, 32));
            const float sc = (m[h] == -INFINITY) ? 0.f : exp2f(m[h] - mm);
            float lh = l[h] * sc;
            lh += __shfl_xor(lh, 8);
            lh += __shfl_xor(lh, 16);
            lh += __shfl_xor(lh, 32);
#pragma unroll
            for (int e = 0; e < EL; ++e) {
                float v = acc[h][e] * sc;
                v += __shfl_xor(v, 8);
                v += __shfl_xor(v, 16);
                v += __shfl_xor(v, 32);
                acc[h][e] = v;
            }
            m[h] = mm;
            l[h] = lh;
        }
        // partial of (workgroup w, sequence b) at slot w + b; slot h writes query head g*G + h
        const size_t part = (size_t)(w + b);
#pragma unroll
        for (int h = 0; h < G; ++h) {
            if (slot == h) {
                const size_t head = part * a.Hq + (size_t)g * G + h;
                float* dst = a.part_acc + head * D;
#pragma unroll
                for (int e = 0; e < EL; ++e) dst[lane_dim<BF16, D>(r, e)] = acc[h][e];
                if (r == 0) {
                    a.part_ml[head * 2 + 0] = m[h];
                    a.part_ml[head * 2 + 1] = l[h];
                }
            }
        }
        lo = i1 + seq_off[b];
    }
}

// out[b][h] = sum_s 2^(m_s - M) acc_s / sum_s 2^(m_s - M) l_s over the partial
// slots of sequence b, in a fixed order.
template <int D>
__global__ void __launch_bounds__(256)
combine_kernel(CombineArgs a) {
    constexpr int NG = 256 / D;                  // slot groups
    __shared__ float red_o[256];
    __shared__ float red_l[256];
    __shared__ float red_m[256];
    const int b = blockIdx.x, h = blockIdx.y;
    const int tid = threadIdx.x;
    const int s0 = a.slot_first[b], s1 = a.slot_end[b];
    float mx = -INFINITY;
    for (int s = s0 + tid; s < s1; s += 256) mx = fmaxf(mx, a.part_ml[((size_t)s * a.Hq + h) * 2]);
    red_m[tid] = mx;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if (tid < o) red_m[tid] = fmaxf(red_m[tid], red_m[tid + o]);
        __syncthreads();
    }
    const float M = red_m[0];
    const int grp = tid / D, d = tid % D;
    float L = 0.f, acc = 0.f;
#pragma unroll 4
    for (int s = s0 + grp; s < s1; s += NG) {
        const size_t head = (size_t)s * a.Hq + h;
        const float wgt = exp2f(a.part_ml[head * 2] - M);
        L = fmaf(wgt, a.part_ml[head * 2 + 1], L);
        acc = fmaf(wgt, a.part_acc[head * D + d], acc);
    }
    red_o[tid] = acc;
    red_l[tid] = L;
    __syncthreads();
    if (grp == 0) {
        float o = 0.f, lt = 0.f;
        for (int k = 0; k < NG; ++k) { o += red_o[k * D + d]; lt += red_l[k * D + d]; }
        a.out[((size_t)b * a.Hq + h) * D + d] = o / lt;
    }
}

size_t lds_bytes(const AttnArgs& a) {
    return (size_t)(((a.B + 1 + 3) & ~3) + kChunkMax + a.Hkv * kChunkMax) * 4;
}

template <bool BF16, int D, int G>
hipError_t launch_t(const AttnArgs& a, int grid, hipStream_t s) {
    const size_t lds = lds_bytes(a);
    hipLaunchKernelGGL((attention_kernel<BF16, D, G>), dim3(grid), dim3(64 * a.Hkv), lds, s, a);
    return hipGetLastError();
}

template <bool BF16, int D, int G>
hipError_t occupancy_t(const AttnArgs& a, int* blocks) {
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, attention_kernel<BF16, D, G>,
                                                        64 * a.Hkv, lds_bytes(a));
}

template <bool BF16, int D>
hipError_t launch_g(const AttnArgs& a, int group, int grid, hipStream_t s, int* occ) {
    switch (group) {
        case 1: return occ ? occupancy_t<BF16, D, 1>(a, occ) : launch_t<BF16, D, 1>(a, grid, s);
        case 2: return occ ? occupancy_t<BF16, D, 2>(a, occ) : launch_t<BF16, D, 2>(a, grid, s);
        case 4: return occ ? occupancy_t<BF16, D, 4>(a, occ) : launch_t<BF16, D, 4>(a, grid, s);
        case 8: return occ ? occupancy_t<BF16, D, 8>(a, occ) : launch_t<BF16, D, 8>(a, grid, s);
    }
    return hipErrorInvalidValue;
}

hipError_t dispatch(const AttnArgs& a, int dtype_bf16, int head_dim, int group, int grid,
                    hipStream_t s, int* occ) {
    if (dtype_bf16) {
        if (head_dim == 128) return launch_g<true, 128>(a, group, grid, s, occ);
        if (head_dim == 64) return launch_g<true, 64>(a, group, grid, s, occ);
    } else {
        if (head_dim == 128) return launch_g<false, 128>(a, group, grid, s, occ);
        if (head_dim == 64) return launch_g<false, 64>(a, group, grid, s, occ);
    }
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, int dtype_bf16, int head_dim, int group,
                            int grid, hipStream_t s) {
    return dispatch(a, dtype_bf16, head_dim, group, grid, s, nullptr);
}

hipError_t attention_occupancy(const AttnArgs& a, int dtype_bf16, int head_dim, int group,
                               int* blocks_per_cu) {
    return dispatch(a, dtype_bf16, head_dim, group, 0, nullptr, blocks_per_cu);
}

hipError_t launch_combine(const CombineArgs& a, int head_dim, hipStream_t s) {
    if (head_dim == 128) {
        hipLaunchKernelGGL(combine_kernel<128>, dim3(a.B, a.Hq), dim3(256), 0, s, a);
    } else if (head_dim == 64) {
        hipLaunchKernelGGL(combine_kernel<64>, dim3(a.B, a.Hq), dim3(256), 0, s, a);
    } else {
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace asrkf
