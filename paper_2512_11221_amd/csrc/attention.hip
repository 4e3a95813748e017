// Active-set GQA flash-decode for gfx950, fused with the relevance score, and
// the per-layer split combine.
//
// Per launch (one layer, every sequence):
//   Eq. 1  o_h = softmax_j(q_h . k_j / sqrt(D)) v_j over the active list A_t;
//   Eq. 2  s_j = (1/Hq) sum_h |q_h . k_j| for every j in A_t, and the flag
//          s_j < tau stored per position; Algorithm 1's freeze loop reads the
//          flags at the end of the step (in the list rebuild, which streams
//          every position's state anyway), so no count or unfreeze step is
//          read or written here.
//
// Work decomposition.  The active lists of all sequences, concatenated (each
// preceded by a few virtual tokens that stand for the fixed cost of a
// sequence), are cut into equal contiguous ranges, one per workgroup of a
// fixed grid, computed on the device from the active counts.  Inside a
// workgroup the range is walked in tiles dealt round-robin to its waves (a
// static deal, so every run sums in the same order); a wave that falls
// behind the others raises its issue priority until it has caught up.  The
// waves' softmax states are merged through LDS once per sequence the range
// touches, giving one partial (m, l, acc) of every query head at slot
// (workgroup + sequence): when all eight states fit in LDS each wave folds
// them for a slice of the rows in one round, otherwise a three-round tree
// folds pairs.
//
// Lane layout inside a wave: 8 slots x 8 lanes.  Slot s holds KV head
// s % Hkv of token s / Hkv of the iteration (8 / Hkv tokens per iteration),
// so a wave reads whole token rows (every KV head) and every load
// instruction moves 8 contiguous 128-byte segments.  A slot's row serves the
// G query heads of its KV head from registers (GQA sharing); dot products are
// reduced over the slot's 8 lanes with DPP, the relevance over the token's
// KV-head slots with lane exchanges, so the score flag is decided in the
// wave and stored by the workgroup after each chunk.
//
// Wide groups and many KV heads.  With G = 8 a slot holds a virtual KV head,
// one KV head with half of its query heads (two slots read the same row, in
// the same load instruction).  When a token has more than 8 (virtual) heads,
// 2 or 4 waves share each token, each with 8 of them; their parts of the
// relevance sum meet in LDS after the tiles, where the flag is decided.
#include "kernels.h"

namespace asrkf {
namespace {

constexpr int kWaves = 8;           // waves per workgroup
constexpr int kChunk = 2048;        // tokens per LDS chunk (positions, score flags)
constexpr int kMinPerGroup = 32;    // fewest tokens worth a workgroup
// Each sequence a workgroup takes part in costs it a fixed set-up and merge
// (list staging, q, the freeze loop, the wave-state merge, a partial), about
// what streaming this many tokens takes; the planner charges it as virtual
// tokens ahead of every non-empty list, so a workgroup whose range straddles
// two sequences gets correspondingly fewer real tokens.
constexpr int kSeqCost = 48;
constexpr int kStage = kChunk / (64 * kWaves);   // chunk entries per thread
// raw buffer descriptor word 3 for gfx9-class targets (32-bit data, no swizzle)
constexpr int kBufferFlags = 0x00020000;
// cache policy of the K/V row loads: non-temporal.  Each row is read once per
// launch, so the loads should not displace anything in L2 / MALL; on gfx950
// this raised the streaming rate of this kernel by about a tenth.
constexpr int kStreamPolicy = 2;

// A value the whole wave agrees on, moved to a scalar register.
__device__ __forceinline__ int wave_uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// value of lane (lane ^ mask) for mask in {8, 16, 32}
template <int MASK>
__device__ __forceinline__ float lane_xor(float v) {
    if constexpr (MASK == 8) return dpp_mov<0x128>(v);    // row_ror:8
    else return __shfl_xor(v, MASK);
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

// Iterations per tile: four, or two when a lane holds four pieces of a row
// (bf16 rows of 256, fp32 rows of 128), so that a tile's rows stay in registers.
template <bool BF16, int D>
constexpr int tile_unroll() { return Row<BF16, D>::kChunks >= 4 ? 2 : 4; }

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

// Offsets of every sequence in the concatenated, cost-padded active lists:
// sequence b owns [seq_off[b], seq_off[b+1]), whose first kSeqCost entries
// are virtual (none for an empty list); seq_off[B] = T.  Wave 0 scans.
__device__ void plan_ranges(const int32_t* n_active, int B, int32_t* seq_off) {
    const int tid = threadIdx.x;
    if (tid < 64) {
        constexpr int kBatch = 8;                 // counts loaded together
        const int per = (B + 63) / 64;
        const int b0 = tid * per;
        const int b1 = min(B, b0 + per);
        int mine = 0;
        for (int bb = b0; bb < b1; bb += kBatch) {
            int cost[kBatch];
#pragma unroll
            for (int k = 0; k < kBatch; ++k) {
                const int n = bb + k < b1 ? n_active[bb + k] : 0;
                cost[k] = n > 0 ? n + kSeqCost : 0;
            }
#pragma unroll
            for (int k = 0; k < kBatch; ++k) {
                if (bb + k < b1) seq_off[bb + k] = cost[k];      // kept here until the scan is done
                mine += cost[k];
            }
        }
        int incl = mine;
        for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_up(incl, o);
            if (tid >= o) incl += y;
        }
        int run = incl - mine;
        for (int bb = b0; bb < b1; ++bb) {
            const int c = seq_off[bb];
            seq_off[bb] = run;
            run += c;
        }
        if (tid == 63) seq_off[B] = incl;
    }
}

// Workgroups that share the tokens: enough that each gets kMinPerGroup of them.
__device__ __forceinline__ int active_groups(int T, int grid) {
    return max(1, min(grid, (T + kMinPerGroup - 1) / kMinPerGroup));
}

// Workgroup holding token x when T tokens are cut into G ranges
// [floor(w T / G), floor((w+1) T / G)).
__device__ __forceinline__ int group_of(int64_t x, int64_t T, int64_t G) {
    return (int)(((x + 1) * G - 1) / T);
}

// Online-softmax state of one lane: its slot's G query heads.
template <bool BF16, int D, int G>
struct SoftState {
    float m[G], l[G];
    float acc[G][Row<BF16, D>::kPerLane];
};

// Fold state b into state a (both of the same lane), fixed order.
template <bool BF16, int D, int G>
__device__ __forceinline__ void fold(SoftState<BF16, D, G>& a, const float* bm, const float* bl,
                                     const float (*bacc)[Row<BF16, D>::kPerLane]) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
        const float M = fmaxf(a.m[h], bm[h]);
        const float sa = (a.m[h] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(a.m[h] - M);
        const float sb = (bm[h] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(bm[h] - M);
        a.l[h] = a.l[h] * sa + bl[h] * sb;
#pragma unroll
        for (int e = 0; e < Row<BF16, D>::kPerLane; ++e) a.acc[h][e] = a.acc[h][e] * sa + bacc[h][e] * sb;
        a.m[h] = M;
    }
}

// How many parts a KV head's query heads are split into, so that a lane keeps
// the softmax state of at most four heads (two for rows of 256): the state of
// more does not fit in a wave's registers.
template <bool BF16, int D, int G>
constexpr int split_of() {
    constexpr int kMaxHeads = Row<BF16, D>::kPerLane >= 32 ? 2 : 4;
    return G > kMaxHeads ? G / kMaxHeads : 1;
}

// Shapes the kernel handles: a token row (every KV head) goes into the cache
// with one 16-byte piece per thread, and after the split no more waves share a
// token than there are waves per state part to fold a head's rows.
template <bool BF16, int D, int G, int HKV>
constexpr bool shape_supported() {
    constexpr int GS = G / split_of<BF16, D, G>();
    constexpr int VH = HKV * split_of<BF16, D, G>();
    constexpr int NWG = VH > 8 ? VH / 8 : 1;
    return (D != 256 || BF16) && HKV * Row<BF16, D>::kBytes <= 64 * kWaves * 16 && NWG <= 4 &&
           GS <= kWaves / NWG;
}

// All 8 wave states fit in LDS next to the other buffers: merge in one round.
template <bool BF16, int D, int G>
constexpr bool merge_one_round() {
    return (size_t)kWaves * (2 * G + G * Row<BF16, D>::kPerLane) * 64 * 4 <= 148 * 1024;
}

// Shapes whose first tile can come from the plan records: one token per wave
// iteration, one wave per token, the first tiles of all waves within the
// record's positions.
template <bool BF16, int D, int G, int HKV>
constexpr bool prefetch_shape() {
    constexpr int VH = HKV * split_of<BF16, D, G>();
    constexpr int NWG = VH > 8 ? VH / 8 : 1;
    constexpr int TPI = 8 / (VH > 8 ? 8 : VH);
    return TPI == 1 && NWG == 1 && kWaves * tile_unroll<BF16, D>() <= kPlanTokens;
}

// PF: the first tile of a range's first chunk is requested from the plan
// record (a.plan must be set); without it the kernel never reads a.plan.
template <bool BF16, int D, int G, int HKV, bool PF>
__global__ void __launch_bounds__(64 * kWaves)
attention_kernel(AttnArgs a) {
    using R = Row<BF16, D>;
    // Wide query groups (G = 8) are split in halves of GS heads: a lane keeps the
    // softmax state of GS query heads only, so it fits in registers.  A virtual
    // KV head is a (KV head, half) pair, VH of them.  When a token has more
    // virtual heads than a wave has slots, NWG waves share each token (wave
    // part p takes virtual heads 8p .. 8p + 7) and the relevance of the parts is
    // summed in LDS after the tiles.
    constexpr int kSplit = split_of<BF16, D, G>();
    constexpr int kUnroll = tile_unroll<BF16, D>();
    constexpr int GS = G / kSplit;               // query heads per lane
    constexpr int VH = HKV * kSplit;             // virtual KV heads
    constexpr int NWG = VH > 8 ? VH / 8 : 1;     // waves sharing a token
    constexpr int SV = VH > 8 ? 8 : VH;          // virtual heads of a token in one wave
    constexpr int kGroups = kWaves / NWG;        // tiles are dealt to groups of NWG waves
    using S = SoftState<BF16, D, GS>;
    constexpr int NC = R::kChunks;
    constexpr int EL = R::kPerLane;
    constexpr int TPI = 8 / SV;                  // tokens per iteration
    constexpr int TT = kUnroll * TPI;            // tokens per tile
    constexpr int NV = 2 * GS + GS * EL;         // floats of a lane's state
    constexpr bool kOneRound = merge_one_round<BF16, D, GS>();
    static_assert(shape_supported<BF16, D, G, HKV>(), "unsupported head layout");

    extern __shared__ int32_t lds[];
    __shared__ unsigned tile_lead;                               // most tiles any wave has finished
    int32_t* seq_off = lds;                                      // [B + 1]
    int32_t* pos_lds = lds + ((a.B + 1 + 3) & ~3);               // [kChunk]
    int32_t* row_lds = pos_lds + kChunk;                         // [kChunk] (spill mode)
    float* rel_lds = reinterpret_cast<float*>(row_lds + kChunk);   // [kChunk][NWG <= 4] (token
                                                                 // scope; the parts' sums)
    uint8_t* flag_lds = reinterpret_cast<uint8_t*>(rel_lds + 4 * kChunk);   // [kChunk]
    // the wave-state merge runs after the chunk loop: it reuses the chunk buffers
    float* merge_lds = reinterpret_cast<float*>(pos_lds);        // [kWaves/2][NV][64]

    // the step's first launch advances the device step counter that the
    // end-of-step rebuild reads (a graph replay of the step then sees its step)
    if (a.t_dev && blockIdx.x == 0 && threadIdx.x == 0) *a.t_dev += 1;
    // The first-tile record of the range this workgroup takes when every
    // workgroup has one (checked once the ranges are known), requested
    // together with the counts: with it the first K/V rows are requested
    // before the chunk's positions and q arrive.
    constexpr bool kPrefetch = PF && prefetch_shape<BF16, D, G, HKV>();
    static_assert(!kPrefetch || (TPI == 1 && NWG == 1 && kGroups * TT <= kPlanTokens), "record layout");
    const int w_full = gridDim.x % 8 == 0 ? (int)((blockIdx.x % 8) * (gridDim.x / 8) + blockIdx.x / 8)
                                          : (int)blockIdx.x;
    int rec_b = -1, rec_i0 = 0, rec_len = 0;
    int rec_pos[kUnroll] = {};
    if constexpr (kPrefetch) {
        // a.plan is always set for this variant; the test stays: without it the
        // compiler scheduled the tile loop differently and the launch took 1.3 %
        // longer (interleaved runs)
        if (a.plan) {
            const int32_t* rec = a.plan + (size_t)w_full * kPlanInts;
            const int t0 = 4 + wave_uniform(threadIdx.x >> 6) * TT;
            rec_b = rec[0];
            rec_i0 = rec[1];
            rec_len = rec[2];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) rec_pos[u] = rec[t0 + u];
        }
    }
    plan_ranges(a.n_active, a.B, seq_off);
    __syncthreads();
    const int T = wave_uniform(seq_off[a.B]);
    const int Gn = active_groups(T, gridDim.x);
    if (blockIdx.x == 0) {
        for (int b = threadIdx.x; b < a.B; b += blockDim.x) {
            // the workgroups holding the list's first and last real tokens
            const int x0 = seq_off[b] + kSeqCost, x1 = seq_off[b + 1];
            a.slot_first[b] = x1 > x0 ? group_of(x0, T, Gn) + b : 0;
            a.slot_end[b] = x1 > x0 ? group_of(x1 - 1, T, Gn) + b + 1 : 0;
        }
    }
    // the range this workgroup takes.  Workgroups are dealt to the 8 XCDs round
    // robin; when every workgroup has a range, each XCD takes a contiguous block
    // of ranges (measured: the slowest XCD's share ends sooner).  Any one-to-one
    // map gives the same partials, so the results do not depend on it; with
    // fewer ranges than workgroups the ranges stay spread over the XCDs.
    const bool blocked = Gn == (int)gridDim.x && gridDim.x % 8 == 0;
    const int w = blocked ? (int)((blockIdx.x % 8) * (gridDim.x / 8) + blockIdx.x / 8) : (int)blockIdx.x;
    if (w >= Gn) return;

    const int wave = wave_uniform(threadIdx.x >> 6);
    const int wpart = wave % NWG;                 // the wave's share of each token's heads
    const int wgrp = wave / NWG;                  // the wave's tile group
    const int lane = threadIdx.x & 63;
    const int slot = lane >> 3;
    const int tk = slot / SV;                     // token of the iteration
    const int vh = wpart * SV + slot % SV;        // virtual KV head
    const int g = vh / kSplit;                    // KV head
    const int qh0 = g * G + (vh % kSplit) * GS;   // the lane's first query head
    const int r = lane & 7;
    const int row_stride = HKV * R::kBytes;       // bytes per token (all KV heads)
    const int lane_off = g * R::kBytes + r * 16;

    int x = wave_uniform((int)((int64_t)w * T / Gn));
    const int x_end = wave_uniform((int)((int64_t)(w + 1) * T / Gn));
    int b = 0;
    {
        int l0 = 0, h0 = a.B - 1;                 // last b with seq_off[b] <= x
        while (l0 < h0) {
            const int mid = (l0 + h0 + 1) >> 1;
            if (wave_uniform(seq_off[mid]) <= x) l0 = mid; else h0 = mid - 1;
        }
        b = l0;
    }
    bool first_piece = true;
    while (x < x_end) {
        while (wave_uniform(seq_off[b + 1]) <= x) ++b;   // skip empty lists
        const int sb = wave_uniform(seq_off[b]) + kSeqCost;   // the list's first real token
        const int se = wave_uniform(seq_off[b + 1]);
        if (x_end <= sb) break;                  // the range ends among the virtual tokens
        const int nb = se - sb;
        const int i0 = max(x, sb) - sb;
        const int i1 = min(se, x_end) - sb;
        const size_t seq_row = (size_t)b * a.cap;
        const size_t seg = (size_t)b * a.pool_rows * row_stride;
        const int32_t* list_b = a.list + seq_row;
        const int32_t* lrow_b = a.list_row + seq_row;
        const bool spill = a.spill != 0;
        const bool rel_abs = a.rel_mode == 0;
        const bool scope_token = a.scope_token != 0;

        S st;
#pragma unroll
        for (int h = 0; h < GS; ++h) {
            st.m[h] = -INFINITY;
            st.l[h] = 0.f;
#pragma unroll
            for (int e = 0; e < EL; ++e) st.acc[h][e] = 0.f;
        }
        const int nbytes = a.pool_rows * row_stride;
        const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
            (void*)((const char*)a.kpool + seg), (short)0, nbytes, kBufferFlags);
        const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
            (void*)((const char*)a.vpool + seg), (short)0, nbytes, kBufferFlags);

        for (int c0 = i0; c0 < i1; c0 += kChunk) {
            const int len = min(kChunk, i1 - c0);
            // the first tile of the range's first chunk comes from the record when it
            // describes this chunk and the tile does not reach the appended token
            uint4 kp[kUnroll][NC], vp[kUnroll][NC];
            bool have = false;
            if constexpr (kPrefetch)
                have = first_piece && c0 == i0 && w == w_full && b == wave_uniform(rec_b) &&
                       i0 == wave_uniform(rec_i0) && len == wave_uniform(rec_len) && wgrp * TT < len &&
                       c0 + kGroups * TT < nb && !spill;
            // a chunk that ends with the new token appends its row to the cache
            // (a token row is at most 8 heads x 128 x 4 bytes, one 16-byte piece
            // per thread); its loads overlap the staging loads below
            const int app_off = threadIdx.x * 16;
            const bool append = c0 + len == nb && app_off < row_stride;
            uint4 knew_piece, vnew_piece;
            int new_row = 0;
            if (append) {
                const size_t src = (size_t)b * row_stride + app_off;
                knew_piece = *reinterpret_cast<const uint4*>((const char*)a.knew + src);
                vnew_piece = *reinterpret_cast<const uint4*>((const char*)a.vnew + src);
                // the list's last entry is the new token (its position; its row in spill mode)
                new_row = spill ? lrow_b[nb - 1] : list_b[nb - 1];
            }
            // stage the chunk's positions (and device rows): every load first, then the
            // stores; the query rows are requested in between, so the chunk's set-up
            // costs one memory round trip
            uint4 qr[GS][NC];
            {
                int sp[kStage], sr[kStage];
#pragma unroll
                for (int k = 0; k < kStage; ++k) {
                    // every load issued (the last entry past the chunk's end), so the
                    // waits below count loads instead of waiting for all of them
                    const int i = min((int)threadIdx.x + k * 64 * kWaves, len - 1);
                    sp[k] = list_b[c0 + i];
                    if (spill) sr[k] = lrow_b[c0 + i];
                }
                const __amdgpu_buffer_rsrc_t rq = __builtin_amdgcn_make_buffer_rsrc(
                    (void*)((const char*)a.q + (size_t)b * a.Hq * R::kBytes), (short)0, a.Hq * R::kBytes,
                    kBufferFlags);
                const int qo = qh0 * R::kBytes + r * 16;
#pragma unroll
                for (int h = 0; h < GS; ++h)
#pragma unroll
                    for (int c = 0; c < NC; ++c)
                        qr[h][c] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                            rq, qo + h * R::kBytes + c * 128, 0, 0));
                // the first tile's rows, requested after the staging loads so that the
                // staging waits for those only (rows of tokens past the chunk's end: the
                // tile's first token, as in the tile loop).  Without a record the loads
                // are still issued, at an offset past the cache's range (a sequence's
                // rows stay below 2 GiB): they return zeros without a memory access,
                // and the waits are counted alike on both paths.
                if constexpr (kPrefetch) {
#pragma unroll
                    for (int u = 0; u < kUnroll; ++u) {
                        const int li = wgrp * TT + u < len ? u : 0;
                        const int so = have ? wave_uniform(rec_pos[li]) * row_stride : 0;
#pragma unroll
                        for (int c = 0; c < NC; ++c) {
                            const int vo = have ? lane_off + c * 128 : (int)0x80000000;
                            kp[u][c] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rk, vo, so, kStreamPolicy));
                            vp[u][c] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rv, vo, so, kStreamPolicy));
                        }
                    }
                }
#pragma unroll
                for (int k = 0; k < kStage; ++k) {
                    const int i = threadIdx.x + k * 64 * kWaves;
                    if (i < len) {
                        pos_lds[i] = sp[k];
                        if (spill) row_lds[i] = sr[k];
                        flag_lds[i] = 0;
                    }
                }
            }
            if (append) {
                const size_t dst = seg + (size_t)new_row * row_stride + app_off;
                *reinterpret_cast<uint4*>((char*)a.kpool_w + dst) = knew_piece;
                *reinterpret_cast<uint4*>((char*)a.vpool_w + dst) = vnew_piece;
            }
            if (threadIdx.x == 0) tile_lead = 0;
            __threadfence_block();
            __syncthreads();

            // One tile: rows kr, vr of the tokens from tb on (rows of tokens past the
            // chunk's end are the tile's first token's, masked here).
            auto tile = [&](const uint4 (&kr)[kUnroll][NC], const uint4 (&vr)[kUnroll][NC], int tb)
                __attribute__((always_inline)) {
                bool valid[kUnroll];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) valid[u] = tb + u * TPI + tk < len;
                float xs[kUnroll][GS];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u)
#pragma unroll
                    for (int h = 0; h < GS; ++h) xs[u][h] = lane_dot<BF16, D>(kr[u], qr[h]);
                // 8-lane sums (every lane of a slot ends with the same bits)
#pragma unroll
                for (int u = 0; u < kUnroll; ++u)
#pragma unroll
                    for (int h = 0; h < GS; ++h) xs[u][h] += dpp_mov<0xB1>(xs[u][h]);   // quad_perm [1,0,3,2]
#pragma unroll
                for (int u = 0; u < kUnroll; ++u)
#pragma unroll
                    for (int h = 0; h < GS; ++h) xs[u][h] += dpp_mov<0x4E>(xs[u][h]);   // quad_perm [2,3,0,1]
#pragma unroll
                for (int u = 0; u < kUnroll; ++u)
#pragma unroll
                    for (int h = 0; h < GS; ++h) xs[u][h] += dpp_mov<0x141>(xs[u][h]);  // row_half_mirror

                // relevance (Eq. 2): sum over the slot's heads, then over the token's KV-head slots
                if (rel_abs) {
#pragma unroll
                    for (int u = 0; u < kUnroll; ++u) {
                        float rel = 0.f;
#pragma unroll
                        for (int h = 0; h < GS; ++h) rel += fabsf(xs[u][h]);
                        if constexpr (SV >= 2) rel += lane_xor<8>(rel);
                        if constexpr (SV >= 4) rel += lane_xor<16>(rel);
                        if constexpr (SV >= 8) rel += lane_xor<32>(rel);
                        if (valid[u] && slot % SV == 0 && r == 0) {
                            if (NWG > 1) {
                                // this wave's part of the sum: the parts meet after the tiles
                                rel_lds[(tb + u * TPI + tk) * NWG + wpart] = rel;
                            } else if (scope_token) {
                                rel_lds[tb + u * TPI + tk] = rel;
                            } else {                      // the freeze loop picks the candidates
                                const int f = (rel < a.tau_H ? 1 : 0) |
                                              (fabsf(rel - a.tau_H) < a.margin_H ? 2 : 0);
                                if (f) flag_lds[tb + u * TPI + tk] = (uint8_t)f;
                            }
                        }
                    }
                }

                float y[kUnroll][GS];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u)
#pragma unroll
                    for (int h = 0; h < GS; ++h) y[u][h] = valid[u] ? xs[u][h] * a.scale_log2 : -INFINITY;
                if (!rel_abs) {
                    // relevance by attention weight needs the sequence's normaliser: keep the logits
#pragma unroll
                    for (int u = 0; u < kUnroll; ++u) {
                        if (valid[u] && r == 0) {
                            float* xl = a.xlog + (seq_row + c0 + tb + u * TPI + tk) * a.Hq + qh0;
#pragma unroll
                            for (int h = 0; h < GS; ++h) xl[h] = y[u][h];
                        }
                    }
                }
#pragma unroll
                for (int h = 0; h < GS; ++h) {
                    float mt = st.m[h];
#pragma unroll
                    for (int u = 0; u < kUnroll; ++u) mt = fmaxf(mt, y[u][h]);
                    if (__any(mt > st.m[h])) {
                        const float sc = (mt > st.m[h]) ? __builtin_amdgcn_exp2f(st.m[h] - mt) : 1.f;
                        st.l[h] *= sc;
#pragma unroll
                        for (int e = 0; e < EL; ++e) st.acc[h][e] *= sc;
                        st.m[h] = mt;
                    }
                }
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) {
#pragma unroll
                    for (int h = 0; h < GS; ++h) {
                        const float pr = valid[u] ? __builtin_amdgcn_exp2f(y[u][h] - st.m[h]) : 0.f;
                        st.l[h] += pr;
                        lane_axpy<BF16, D>(st.acc[h], pr, vr[u]);
                    }
                }
                // Pacing.  The tiles are dealt statically (every run sums in the same
                // order), but when several waves can issue the hardware favours the
                // older ones, and over a long range the younger waves fall behind by
                // about a tenth.  A wave that has finished fewer tiles than the
                // workgroup's leader issues at a raised priority until it catches up.
                {
                    const unsigned done = (unsigned)((tb - wgrp * TT) / (kGroups * TT) + 1);
                    unsigned lead = 0;
                    if (lane == 0) lead = atomicMax(&tile_lead, done);
                    if (done < (unsigned)wave_uniform((int)lead)) __builtin_amdgcn_s_setprio(2);
                    else __builtin_amdgcn_s_setprio(0);
                }
            };
            int tb0 = wgrp * TT;
            if constexpr (kPrefetch) {
                if (have) {                       // rows requested with the staging loads
                    tile(kp, vp, tb0);
                    tb0 += kGroups * TT;
                }
            }
            for (int tb = tb0; tb < len; tb += kGroups * TT) {
                uint4 kr[kUnroll][NC], vr[kUnroll][NC];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) {
                    const int idx = tb + u * TPI + tk;
                    const int li = idx < len ? idx : tb;
                    const int drow = spill ? row_lds[li] : pos_lds[li];     // device row of the token
                    int vo = lane_off, so = 0;
                    if constexpr (TPI == 1) so = wave_uniform(drow) * row_stride;
                    else vo += drow * row_stride;
#pragma unroll
                    for (int c = 0; c < NC; ++c) {
                        kr[u][c] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rk, vo + c * 128, so, kStreamPolicy));
                        vr[u][c] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rv, vo + c * 128, so, kStreamPolicy));
                    }
                }
                tile(kr, vr, tb);
            }
            __builtin_amdgcn_s_setprio(0);
            __syncthreads();

            if constexpr (NWG > 1) {
                // the token's score is the sum of its parts (fixed order); in layer
                // scope it decides the flag here, in token scope the sum is kept below
#pragma unroll
                for (int k = 0; k < kStage; ++k) {
                    const int i = threadIdx.x + k * 64 * kWaves;
                    if (i < len) {
                        float sum = 0.f;
#pragma unroll
                        for (int p2 = 0; p2 < NWG; ++p2) sum += rel_lds[i * NWG + p2];
                        if (scope_token) rel_lds[i * NWG] = sum;
                        else flag_lds[i] = rel_abs ? (uint8_t)((sum < a.tau_H ? 1 : 0) |
                                                               (fabsf(sum - a.tau_H) < a.margin_H ? 2 : 0))
                                                   : (uint8_t)0;
                    }
                }
            }
            if (scope_token && rel_abs) {
                // token scope sums the score over the layers; the freeze loop runs at the step's end
                float prev[kStage];
#pragma unroll
                for (int k = 0; k < kStage; ++k) {
                    const int i = threadIdx.x + k * 64 * kWaves;
                    prev[k] = (i < len && !a.first_layer) ? a.rel_acc[seq_row + pos_lds[i]] : 0.f;
                }
#pragma unroll
                for (int k = 0; k < kStage; ++k) {
                    const int i = threadIdx.x + k * 64 * kWaves;
                    if (i < len) a.rel_acc[seq_row + pos_lds[i]] = prev[k] + rel_lds[i * NWG];
                }
            }
            // score flags of the chunk's tokens (s_j < tau), one byte per position, for
            // the freeze loop of the end-of-step rebuild (which tests the window)
            if (rel_abs && !scope_token) {
#pragma unroll
                for (int k = 0; k < kStage; ++k) {
                    const int i = threadIdx.x + k * 64 * kWaves;
                    if (i < len) a.flag[seq_row + pos_lds[i]] = flag_lds[i];
                }
            }
            __syncthreads();                       // LDS chunk buffers are reused next
        }

        if constexpr (kOneRound) {
            // merge the wave states in one round: every wave stores its state, then
            // each wave folds the states of its part's waves for its own rows
            // (fixed order)
            __syncthreads();
            {
                float* dst = merge_lds + (size_t)wave * NV * 64 + lane;
#pragma unroll
                for (int h = 0; h < GS; ++h) {
                    dst[(2 * h) * 64] = st.m[h];
                    dst[(2 * h + 1) * 64] = st.l[h];
#pragma unroll
                    for (int e = 0; e < EL; ++e) dst[(2 * GS + h * EL + e) * 64] = st.acc[h][e];
                }
            }
            __syncthreads();
            // the states of the waves of one part cover the same heads: fold those
            constexpr int kPerPart = kWaves / NWG;
            constexpr int RPW = GS * EL / kPerPart;       // acc rows folded by each wave
            const int row0 = wgrp * RPW;                  // first row, within head hh
            const int hh = row0 / EL, e0 = row0 % EL;
            float M = -INFINITY;
            float ms[kPerPart];
#pragma unroll
            for (int j = 0; j < kPerPart; ++j) {
                const int s2 = j * NWG + wpart;           // the part's waves, in order
                ms[j] = merge_lds[((size_t)s2 * NV + 2 * hh) * 64 + lane];
                M = fmaxf(M, ms[j]);
            }
            float Lf = 0.f, accf[RPW];
#pragma unroll
            for (int i = 0; i < RPW; ++i) accf[i] = 0.f;
#pragma unroll
            for (int j = 0; j < kPerPart; ++j) {
                const int s2 = j * NWG + wpart;
                const float wgt = (ms[j] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(ms[j] - M);
                Lf = fmaf(wgt, merge_lds[((size_t)s2 * NV + 2 * hh + 1) * 64 + lane], Lf);
#pragma unroll
                for (int i = 0; i < RPW; ++i)
                    accf[i] = fmaf(wgt, merge_lds[((size_t)s2 * NV + 2 * GS + hh * EL + e0 + i) * 64 + lane], accf[i]);
            }
            // slots holding the same KV head (different tokens of an iteration)
#pragma unroll
            for (int mask = 8 * SV; mask < 64; mask <<= 1) {
                const float om = __shfl_xor(M, mask), ol = __shfl_xor(Lf, mask);
                float oa[RPW];
#pragma unroll
                for (int i = 0; i < RPW; ++i) oa[i] = __shfl_xor(accf[i], mask);
                // fixed order: the lower lane's state first
                const bool up = (lane & mask) != 0;
                const float m1 = up ? om : M, m2 = up ? M : om;
                const float Mn = fmaxf(m1, m2);
                const float w1 = (m1 == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m1 - Mn);
                const float w2 = (m2 == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m2 - Mn);
                const float l1 = up ? ol : Lf, l2 = up ? Lf : ol;
                Lf = l1 * w1 + l2 * w2;
#pragma unroll
                for (int i = 0; i < RPW; ++i) {
                    const float a1 = up ? oa[i] : accf[i], a2 = up ? accf[i] : oa[i];
                    accf[i] = a1 * w1 + a2 * w2;
                }
                M = Mn;
            }
            __syncthreads();                       // merge buffer reads done: chunks may restage
            if (tk == 0) {
                const size_t part = (size_t)(w + b) * a.Hq + (size_t)qh0 + hh;
                float* dst = a.part_acc + part * D;
#pragma unroll
                for (int i = 0; i < RPW; ++i) {
                    const int e = e0 + i;
                    dst[(e / R::kPerChunk) * (128 / R::kElem) + r * R::kPerChunk + (e % R::kPerChunk)] = accf[i];
                }
                if (r == 0 && e0 == 0) {
                    a.part_ml[part * 2 + 0] = M;
                    a.part_ml[part * 2 + 1] = Lf;
                }
            }
        } else {
        // merge the waves' states: a fixed tree through LDS (4 -> 2 -> 1 partners)
#pragma unroll
        for (int half = kWaves / 2; half >= NWG; half >>= 1) {
            __syncthreads();
            if (wave >= half && wave < 2 * half) {
                float* dst = merge_lds + (size_t)(wave - half) * NV * 64 + lane;
#pragma unroll
                for (int h = 0; h < GS; ++h) {
                    dst[(2 * h) * 64] = st.m[h];
                    dst[(2 * h + 1) * 64] = st.l[h];
#pragma unroll
                    for (int e = 0; e < EL; ++e) dst[(2 * GS + h * EL + e) * 64] = st.acc[h][e];
                }
            }
            __syncthreads();
            if (wave < half) {
                const float* src = merge_lds + (size_t)wave * NV * 64 + lane;
                float bm[GS], bl[GS], bacc[GS][EL];
#pragma unroll
                for (int h = 0; h < GS; ++h) {
                    bm[h] = src[(2 * h) * 64];
                    bl[h] = src[(2 * h + 1) * 64];
#pragma unroll
                    for (int e = 0; e < EL; ++e) bacc[h][e] = src[(2 * GS + h * EL + e) * 64];
                }
                fold<BF16, D, GS>(st, bm, bl, bacc);
            }
        }
        __syncthreads();                           // merge buffer reads done: chunks may restage
        if (wave < NWG) {
            // merge the slots that hold the same KV head (different tokens of an iteration)
#pragma unroll
            for (int mask = 8 * SV; mask < 64; mask <<= 1) {
                float bm[GS], bl[GS], bacc[GS][EL];
#pragma unroll
                for (int h = 0; h < GS; ++h) {
                    bm[h] = __shfl_xor(st.m[h], mask);
                    bl[h] = __shfl_xor(st.l[h], mask);
#pragma unroll
                    for (int e = 0; e < EL; ++e) bacc[h][e] = __shfl_xor(st.acc[h][e], mask);
                }
                // fold in a fixed order: the lower lane's state first
                if (lane & mask) {
#pragma unroll
                    for (int h = 0; h < GS; ++h) {
                        const float tm = st.m[h], tl = st.l[h];
                        st.m[h] = bm[h]; bm[h] = tm;
                        st.l[h] = bl[h]; bl[h] = tl;
#pragma unroll
                        for (int e = 0; e < EL; ++e) {
                            const float ta = st.acc[h][e];
                            st.acc[h][e] = bacc[h][e];
                            bacc[h][e] = ta;
                        }
                    }
                }
                fold<BF16, D, GS>(st, bm, bl, bacc);
            }
            // partial of (workgroup w, sequence b): slot (token 0, virtual head vh) writes
            // query heads qh0 .. qh0 + GS - 1
            if (tk == 0) {
                const size_t part = (size_t)(w + b) * a.Hq + (size_t)qh0;
#pragma unroll
                for (int h = 0; h < GS; ++h) {
                    float* dst = a.part_acc + (part + h) * D;
#pragma unroll
                    for (int c = 0; c < NC; ++c)
#pragma unroll
                        for (int i = 0; i < R::kPerChunk; i += 4) {
                            const int e = c * R::kPerChunk + i;
                            *reinterpret_cast<float4*>(dst + c * (128 / R::kElem) + r * R::kPerChunk + i) =
                                make_float4(st.acc[h][e], st.acc[h][e + 1], st.acc[h][e + 2], st.acc[h][e + 3]);
                        }
                    if (r == 0) {
                        a.part_ml[(part + h) * 2 + 0] = st.m[h];
                        a.part_ml[(part + h) * 2 + 1] = st.l[h];
                    }
                }
            }
        }
        }
        first_piece = false;
        x = sb + i1;
    }
}

// Split combine.  A block owns 64 dims of one query head of one sequence;
// its GROUPS slot groups each fold every GROUPS-th partial slot into a running
// (max, sum, acc) in passes of kSlotUnroll slots (all loads of a pass issued
// together), and the groups' states are folded in a fixed order:
//   out[b][h][d] = sum_s 2^(m_s - M) acc_s[d] / sum_s 2^(m_s - M) l_s.
// The launch sizes GROUPS to the slots a sequence has, so that a sequence's
// partials take few dependent passes (one sequence over the whole device has
// about 257 slots, eight sequences about 33, sixty-four about 5).
constexpr int kFinishDims = 64;
constexpr int kSlotUnroll = 8;

template <int GROUPS>
__global__ void __launch_bounds__(kFinishDims * GROUPS)
finish_kernel(FinishArgs a, int D) {
    constexpr int kThreads = kFinishDims * GROUPS;
    __shared__ float sm[kThreads], sl[kThreads], sa[kThreads];
    const int per_head = D / kFinishDims;
    const int bh = blockIdx.x / per_head;                 // b * Hq + h
    const int d = (blockIdx.x % per_head) * kFinishDims + threadIdx.x % kFinishDims;
    const int grp = threadIdx.x / kFinishDims;
    const int b = bh / a.Hq, h = bh % a.Hq;
    const int s0 = a.slot_first[b], s1 = a.slot_end[b];
    float M = -INFINITY, L = 0.f, acc = 0.f;
    for (int k = s0 + grp; k < s1; k += GROUPS * kSlotUnroll) {
        float mk[kSlotUnroll], lk[kSlotUnroll], ak[kSlotUnroll];
#pragma unroll
        for (int u = 0; u < kSlotUnroll; ++u) {
            const int ks = min(k + u * GROUPS, s1 - 1);
            const size_t head = (size_t)ks * a.Hq + h;
            mk[u] = a.part_ml[head * 2];
            lk[u] = a.part_ml[head * 2 + 1];
            ak[u] = a.part_acc[head * D + d];
        }
        float Mn = M;
#pragma unroll
        for (int u = 0; u < kSlotUnroll; ++u)
            if (k + u * GROUPS < s1) Mn = fmaxf(Mn, mk[u]);
        const float sc = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(M - Mn);
        L *= sc;
        acc *= sc;
#pragma unroll
        for (int u = 0; u < kSlotUnroll; ++u) {
            if (k + u * GROUPS < s1) {
                const float wgt = __builtin_amdgcn_exp2f(mk[u] - Mn);
                L = fmaf(wgt, lk[u], L);
                acc = fmaf(wgt, ak[u], acc);
            }
        }
        M = Mn;
    }
    if constexpr (GROUPS > 1) {
        sm[threadIdx.x] = M;
        sl[threadIdx.x] = L;
        sa[threadIdx.x] = acc;
        __syncthreads();
        if (grp != 0) return;
        float Mt = -INFINITY;
#pragma unroll
        for (int k = 0; k < GROUPS; ++k) Mt = fmaxf(Mt, sm[k * kFinishDims + threadIdx.x]);
        float o = 0.f, lt = 0.f;
#pragma unroll
        for (int k = 0; k < GROUPS; ++k) {
            const float mk = sm[k * kFinishDims + threadIdx.x];
            const float wgt = (mk == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mk - Mt);
            o = fmaf(wgt, sa[k * kFinishDims + threadIdx.x], o);
            lt = fmaf(wgt, sl[k * kFinishDims + threadIdx.x], lt);
        }
        M = Mt;
        L = lt;
        acc = o;
    }
    a.out[(size_t)bh * D + d] = acc / L;
    if (a.norm && threadIdx.x == 0 && blockIdx.x % per_head == 0) {
        a.norm[(size_t)bh * 2] = M;
        a.norm[(size_t)bh * 2 + 1] = L;
    }
}

// First-tile records of every range of the attention grid, one workgroup per
// state layer, one thread per range: the same split, the same piece and chunk
// as the attention kernel takes (which compares the record with its own before
// using it).
__global__ void __launch_bounds__(256) plan_kernel(PlanArgs a) {
    __shared__ int32_t seq_off[kMaxBatch + 1];
    const size_t st = blockIdx.x;
    plan_ranges(a.n_active + st * a.B, a.B, seq_off);
    __syncthreads();
    const int T = seq_off[a.B];
    const int Gn = active_groups(T, a.grid);
    const int32_t* list = a.list + st * a.B * a.cap;
    for (int w = threadIdx.x; w < a.grid; w += blockDim.x) {
        int32_t* rec = a.plan + (st * a.grid + w) * kPlanInts;
        int b = -1, i0 = 0, len = 0;
        const int x = (int)((int64_t)w * T / Gn);
        const int x_end = (int)((int64_t)(w + 1) * T / Gn);
        if (w < Gn && x < x_end) {
            int lo = 0, hi = a.B - 1;              // last sequence with seq_off <= x
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (seq_off[mid] <= x) lo = mid; else hi = mid - 1;
            }
            while (seq_off[lo + 1] <= x) ++lo;     // past empty lists (seq_off[B] = T > x)
            const int sb = seq_off[lo] + kSeqCost, se = seq_off[lo + 1];
            if (x_end > sb) {
                b = lo;
                i0 = max(x, sb) - sb;
                len = min(kChunk, min(se, x_end) - sb - i0);
            }
        }
        rec[0] = b;
        rec[1] = i0;
        rec[2] = len;
        rec[3] = 0;
        if (b >= 0) {
            const int32_t* src = list + (size_t)b * a.cap + i0;
            int v[kPlanTokens];
#pragma unroll
            for (int k = 0; k < kPlanTokens; ++k) v[k] = src[min(k, len - 1)];
#pragma unroll
            for (int k = 0; k < kPlanTokens; ++k) rec[4 + k] = v[k];
        }
    }
}

template <bool BF16, int D, int G>
constexpr int state_floats() { return 2 * G + G * Row<BF16, D>::kPerLane; }

template <bool BF16, int D, int G>
size_t lds_bytes(const AttnArgs& a) {
    const size_t chunk = (size_t)kChunk * (4 + 4 + 16 + 1);
    constexpr int GS = G / split_of<BF16, D, G>();
    const size_t merge = (size_t)(merge_one_round<BF16, D, GS>() ? kWaves : kWaves / 2) *
                         state_floats<BF16, D, GS>() * 64 * 4;
    return (size_t)((a.B + 1 + 3) & ~3) * 4 + (chunk > merge ? chunk : merge);
}

// Timing events, when given, are recorded by the dispatch itself, so they
// bracket the kernel's execution and not the queue work around it.
struct Launch {
    int grid;
    hipStream_t stream;
    hipEvent_t start, stop;
    int* occ;                       // non-null: report occupancy instead
};

template <bool BF16, int D, int G, int HKV>
hipError_t launch_t(const AttnArgs& a, const Launch& l) {
    const size_t lds = lds_bytes<BF16, D, G>(a);
    constexpr bool kPF = prefetch_shape<BF16, D, G, HKV>();
    if (l.occ) {                          // the variant that fits fewer workgroups
        hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
            l.occ, attention_kernel<BF16, D, G, HKV, false>, 64 * kWaves, lds);
        if (e != hipSuccess || !kPF) return e;
        int occ_pf = 0;
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ_pf, attention_kernel<BF16, D, G, HKV, kPF>,
                                                         64 * kWaves, lds);
        if (occ_pf < *l.occ) *l.occ = occ_pf;
        return e;
    }
    auto k = kPF && a.plan ? attention_kernel<BF16, D, G, HKV, kPF> : attention_kernel<BF16, D, G, HKV, false>;
    AttnArgs arg = a;
    void* args[] = {&arg};
    return hipExtLaunchKernel(reinterpret_cast<const void*>(k), dim3(l.grid), dim3(64 * kWaves),
                              args, lds, l.stream, l.start, l.stop, 0);
}

template <bool BF16, int D, int G, int HKV>
hipError_t launch_s(const AttnArgs& a, const Launch& l) {
    if constexpr (shape_supported<BF16, D, G, HKV>()) return launch_t<BF16, D, G, HKV>(a, l);
    else return hipErrorInvalidValue;
}

template <bool BF16, int D, int G>
hipError_t launch_h(const AttnArgs& a, const Launch& l) {
    switch (a.Hkv) {
        case 1: return launch_s<BF16, D, G, 1>(a, l);
        case 2: return launch_s<BF16, D, G, 2>(a, l);
        case 4: return launch_s<BF16, D, G, 4>(a, l);
        case 8: return launch_s<BF16, D, G, 8>(a, l);
        case 16: return launch_s<BF16, D, G, 16>(a, l);
        case 32: return launch_s<BF16, D, G, 32>(a, l);
    }
    return hipErrorInvalidValue;
}

template <bool BF16, int D>
hipError_t launch_g(const AttnArgs& a, int group, const Launch& l) {
    switch (group) {
        case 1: return launch_h<BF16, D, 1>(a, l);
        case 2: return launch_h<BF16, D, 2>(a, l);
        case 4: return launch_h<BF16, D, 4>(a, l);
        case 8: return launch_h<BF16, D, 8>(a, l);
    }
    return hipErrorInvalidValue;
}

hipError_t dispatch(const AttnArgs& a, int dtype_bf16, int head_dim, int group, const Launch& l) {
    if (dtype_bf16) {
        if (head_dim == 128) return launch_g<true, 128>(a, group, l);
        if (head_dim == 64) return launch_g<true, 64>(a, group, l);
        if (head_dim == 256) return launch_g<true, 256>(a, group, l);
    } else {
        if (head_dim == 128) return launch_g<false, 128>(a, group, l);
        if (head_dim == 64) return launch_g<false, 64>(a, group, l);
    }
    return hipErrorInvalidValue;
}

}  // namespace

namespace {
template <bool BF16, int D, int G>
bool supported_h(int hkv) {
    switch (hkv) {
        case 1: return shape_supported<BF16, D, G, 1>();
        case 2: return shape_supported<BF16, D, G, 2>();
        case 4: return shape_supported<BF16, D, G, 4>();
        case 8: return shape_supported<BF16, D, G, 8>();
        case 16: return shape_supported<BF16, D, G, 16>();
        case 32: return shape_supported<BF16, D, G, 32>();
    }
    return false;
}
template <bool BF16, int D>
bool supported_g(int group, int hkv) {
    switch (group) {
        case 1: return supported_h<BF16, D, 1>(hkv);
        case 2: return supported_h<BF16, D, 2>(hkv);
        case 4: return supported_h<BF16, D, 4>(hkv);
        case 8: return supported_h<BF16, D, 8>(hkv);
    }
    return false;
}
}  // namespace

bool attention_shape_supported(int dtype_bf16, int head_dim, int group, int n_kv_heads) {
    if (head_dim == 128) return dtype_bf16 ? supported_g<true, 128>(group, n_kv_heads)
                                           : supported_g<false, 128>(group, n_kv_heads);
    if (head_dim == 64) return dtype_bf16 ? supported_g<true, 64>(group, n_kv_heads)
                                          : supported_g<false, 64>(group, n_kv_heads);
    if (head_dim == 256) return dtype_bf16 && supported_g<true, 256>(group, n_kv_heads);
    return false;
}

hipError_t launch_attention(const AttnArgs& a, int dtype_bf16, int head_dim, int group,
                            int grid, hipStream_t s, hipEvent_t start, hipEvent_t stop) {
    return dispatch(a, dtype_bf16, head_dim, group, Launch{grid, s, start, stop, nullptr});
}

hipError_t attention_occupancy(const AttnArgs& a, int dtype_bf16, int head_dim, int group,
                               int* blocks_per_cu) {
    return dispatch(a, dtype_bf16, head_dim, group, Launch{0, nullptr, nullptr, nullptr, blocks_per_cu});
}

hipError_t launch_plan(const PlanArgs& a, int n_states, hipStream_t s) {
    if (a.B < 1 || a.B > kMaxBatch || a.grid < 1 || n_states < 1) return hipErrorInvalidValue;
    hipLaunchKernelGGL(plan_kernel, dim3(n_states), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_finish(const FinishArgs& a, int head_dim, int slots_per_seq, hipStream_t s) {
    if (head_dim % kFinishDims) return hipErrorInvalidValue;
    const dim3 grid(a.B * a.Hq * (head_dim / kFinishDims));
    if (slots_per_seq > 8 * kSlotUnroll)
        hipLaunchKernelGGL(finish_kernel<16>, grid, dim3(kFinishDims * 16), 0, s, a, head_dim);
    else if (slots_per_seq > kSlotUnroll)
        hipLaunchKernelGGL(finish_kernel<4>, grid, dim3(kFinishDims * 4), 0, s, a, head_dim);
    else
        hipLaunchKernelGGL(finish_kernel<1>, grid, dim3(kFinishDims), 0, s, a, head_dim);
    return hipGetLastError();
}

}  // namespace asrkf
