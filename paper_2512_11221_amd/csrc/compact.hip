// End-of-step rebuild of every active cache, with staged recovery fused in.
//
// One workgroup per (layer, sequence), or per sequence when the token states
// are shared by all layers.  It streams the unfreeze steps U_p, detection
// counts c_p and score flags of the n_t positions and:
//   0. runs the step's freeze loop (Algorithm 1): a position that attended
//      step t (U_p <= t), is a freeze candidate and scored below tau gets
//      c_p += 1 and, when d = floor(sqrt(c_p)/k) >= 1, U_p = t + d.  The
//      verdict "below tau" is the flag byte the attention kernel wrote for
//      the position at step t (layer scope), or in token scope the relevance
//      summed over every layer, which no single layer's kernel can form;
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
// Spill mode (Sec. 3.2: frozen KV leaves the GPU) adds device-row bookkeeping
// to the same pass structure, all of it on the device:
//   pass 1  a token frozen at step t for d >= spill_min_D steps gives its
//           device row back to the sequence's free stack; if the host store
//           does not hold its rows yet (K and V never change, so they are
//           copied out once), the (position, row) pair goes to the out-list;
//   pass 2  every position of the new active list that has no device row
//           (its timer ran out, or recovery released it) takes one from the
//           stack and goes to the in-list; the next token takes one too.
// Rows are pushed and popped in ascending position order, so the assignment
// is the same on every run.  The copies themselves are made by the transfer
// kernel (out-list first, so a row is read before it is handed out again).
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

__device__ __forceinline__ void load4(const int32_t* src, int p, int n, int (&v)[4], int fill) {
    // p is a multiple of 4 and every array row starts 16-byte aligned
    if (p + 3 < n) {
        const int4 x = *reinterpret_cast<const int4*>(src + p);
        v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) v[k] = (p + k < n) ? src[p + k] : fill;
    }
}

struct Ladder {
    bool sr, wr, fr;
    int t1, wr_from;
};

__device__ __forceinline__ Ladder make_ladder(const CompactArgs& a, int b, int n) {
    const int level = a.forced_level >= 0 ? a.forced_level : (a.level ? a.level[b] : 0);
    return Ladder{level == 1, level == 2, level == 3, a.t + 1, n - a.wr_last_N};
}

// The freeze loop of step t over the 4 positions p .. p+3 of a thread (those
// below hi): u, cnt are their U and c, flags their score flags (one byte
// each, layer scope).  With a cumulative count (history_W = 0) the counts come
// in with U and only changed entries are stored; a finite history window
// updates the detection bits of a flagged position.  Returns whether u changed.
__device__ __forceinline__ bool freeze4(const CompactArgs& a, size_t base, int p, int hi, int n,
                                        int (&u)[4], const int (&cnt)[4], uint32_t flags) {
    if (!a.freeze) return false;
    bool dirty = false;
    const bool inside = a.cand_inside != 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int q = p + k;
        bool low;
        if (a.scope_token) low = q < hi && a.rel_acc[base + q] < a.tau_LH;
        else low = ((flags >> (8 * k)) & 0xFFu) != 0;
        if (q < hi && u[k] <= a.t && low && freeze_candidate(q, n - a.window_K, inside)) {
            int c;
            if (a.history_W == 0) {
                c = cnt[k] + 1;
                a.count[base + q] = c;
            } else {
                c = detect(a.count, a.hmask, a.hlast, base + q, a.t, a.history_W);
            }
            const int d = a.dur[min(c, a.dur_len - 1)];
            if (d >= 1) {
                u[k] = a.t + d;
                dirty = true;
            }
        }
    }
    return dirty;
}

// U, counts and flags of the 4 positions p .. p+3 (those below hi), as the
// freeze loop reads them; counts and flags only when the step freezes.
struct Tile4 {
    int u[4], c[4];
    uint32_t f;
};

__device__ __forceinline__ void load_tile(const CompactArgs& a, size_t base, int p, int hi, Tile4& x) {
    load4(a.unfreeze + base, p, hi, x.u, 0);
    x.f = 0;
    if (a.freeze) {
        if (a.history_W == 0) load4(a.count + base, p, hi, x.c, 0);
        if (!a.scope_token) {
            if (p + 3 < hi) {
                x.f = *reinterpret_cast<const uint32_t*>(a.flag + base + p);
            } else {
#pragma unroll
                for (int k = 0; k < 4; ++k) x.f |= (p + k < hi ? (uint32_t)a.flag[base + p + k] : 0u) << (8 * k);
            }
        }
    }
}

// Every rebuild kernel starts here: the step index t comes from the device
// counter that the step's first attention launch advanced (so a step captured
// in a graph replays with the right index), the freeze loop runs from step 1
// on, and the rebuild after a step that took a sequence past max_ctx positions
// (a replayed step; the host refuses such a step otherwise) is refused: flag
// for the host, nothing read or written, so every access stays below
// max_ctx + 1 <= cap.  Returns n_t of sequence b, or -1 when refused.
// Uniform over the workgroup.
__device__ __forceinline__ int begin_rebuild(CompactArgs& a, int b, bool first_pass) {
    a.t = *a.t_dev;
    a.freeze = a.t > 0 ? 1 : 0;
    const int n = a.plen[b] + a.t;
    if (n > a.max_ctx) {
        if (threadIdx.x == 0) a.flags[1] = 1;
        return -1;
    }
    // a forced recovery level (no logits) is counted once per rebuild, by its first pass
    if (first_pass && a.count_forced && a.forced_level > 0 && blockIdx.x == 0 && blockIdx.y == 0 &&
        threadIdx.x == 0)
        atomicAdd(a.recoveries + a.forced_level, (unsigned long long)a.B);
    return n;
}

// Recovery select of one position.  Written with bitwise operators only: one
// select per position, no short-circuit control flow.
__device__ __forceinline__ int recover(const Ladder& r, int u, int q, bool live, bool& hit) {
    const bool frozen_now = live & (u > r.t1);
    hit = frozen_now & ((r.sr & (u > r.t1 + 1)) | (r.wr & (q >= r.wr_from)) | r.fr);
    return hit ? r.t1 : u;
}

// Exclusive offsets inside the tile of up to two per-thread item counts, and
// the tile totals.  Every thread of the block must call it.
struct Scan {
    int off0, off1, tot0, tot1;
};

__device__ __forceinline__ Scan tile_scan(int before0, int mine0, int before1, int mine1,
                                          int* tot0, int* tot1) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 63) {
        tot0[wave] = before0 + mine0;
        tot1[wave] = before1 + mine1;
    }
    __syncthreads();
    Scan s{before0, before1, 0, 0};
    for (int w = 0; w < kWaves; ++w) {
        const int c0 = tot0[w], c1 = tot1[w];
        s.off0 += (w < wave) ? c0 : 0;
        s.off1 += (w < wave) ? c1 : 0;
        s.tot0 += c0;
        s.tot1 += c1;
    }
    __syncthreads();                          // tot0/tot1 are rewritten by the next tile
    return s;
}

// Ballot prefix of 4 per-position flags: items of lower lanes, own items.
__device__ __forceinline__ void ballot4(const bool (&f)[4], int& before, int& mine) {
    before = 0;
    mine = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        before += lanes_below(__ballot(f[k]));
        mine += f[k];
    }
}

// The rebuild of positions [lo, hi) of one instance.  MODE 0 applies the
// step's updates (freeze loop, recovery) and writes the list;
// MODE 1 applies the updates and only counts; MODE 2 writes the list from
// the already updated U.  List entries start at list + out_base.  Returns
// the number of listed positions (the same value in every thread).
template <int MODE>
__device__ int compact_range(const CompactArgs& a, const Ladder& r, size_t base, int n, int lo,
                             int hi, int out_base, int* tot0, int* tot1) {
    int32_t* U = a.unfreeze + base;
    int32_t* list = a.list + base;
    const int tid = threadIdx.x;
    int listed = 0;
    Tile4 next;
    if constexpr (MODE != 2) load_tile(a, base, lo + 4 * tid, hi, next);
    else load4(U, lo + 4 * tid, hi, next.u, 0);
    for (int p0 = lo; p0 < hi; p0 += 4 * kThreads) {
        const int p = p0 + 4 * tid;
        Tile4 cur = next;
        int (&u)[4] = cur.u;
        if (p0 + 4 * kThreads < hi) {                                            // next tile in flight
            if constexpr (MODE != 2) load_tile(a, base, p + 4 * kThreads, hi, next);
            else load4(U, p + 4 * kThreads, hi, next.u, 0);
        }
        bool flag[4];
        if constexpr (MODE != 2) {
            bool dirty = freeze4(a, base, p, hi, n, u, cur.c, cur.f);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                bool hit;
                const bool live = p + k < hi;
                u[k] = recover(r, u[k], p + k, live, hit);
                dirty |= hit;
                flag[k] = live & (u[k] <= r.t1);
            }
            if (dirty) {
                for (int k = 0; k < 4; ++k) if (p + k < hi) U[p + k] = u[k];
            }
        } else {
#pragma unroll
            for (int k = 0; k < 4; ++k) flag[k] = (p + k < hi) & (u[k] <= r.t1);
        }
        int before, mine;
        ballot4(flag, before, mine);
        const Scan sc = tile_scan(before, mine, 0, 0, tot0, tot1);
        if constexpr (MODE != 1) {
            int out = out_base + listed + sc.off0;
#pragma unroll
            for (int k = 0; k < 4; ++k) if (flag[k]) list[out++] = p + k;
        }
        listed += sc.tot0;
    }
    return listed;
}

// List tail of an instance: the position n that the next token will take.
__device__ __forceinline__ void finish_list(const CompactArgs& a, int inst, size_t base, int n, int listed) {
    a.list[base + listed] = n;
    a.n_active[inst] = listed + 1;
    atomicAdd(a.listed_total, (unsigned long long)(listed + 1));
}

// One workgroup per instance.
__global__ void __launch_bounds__(kThreads)
compact_kernel(CompactArgs a) {
    __shared__ int tot0[kWaves], tot1[kWaves];
    const int inst = blockIdx.x;
    const int b = inst % a.B;
    const int n = begin_rebuild(a, b, true);        // positions after step t
    if (n < 0) return;
    const Ladder r = make_ladder(a, b, n);
    const size_t base = (size_t)inst * a.cap;
    const int listed = compact_range<0>(a, r, base, n, 0, n, 0, tot0, tot1);
    if (threadIdx.x == 0) finish_list(a, inst, base, n, listed);
}

// Few, long instances: each instance is cut into segments of seg_len
// positions, one workgroup each.  Pass A applies the updates and counts each
// segment; pass B adds the counts of the segments before it and writes.
__global__ void __launch_bounds__(kThreads)
compact_count_kernel(CompactArgs a) {
    __shared__ int tot0[kWaves], tot1[kWaves];
    const int seg = blockIdx.x, inst = blockIdx.y;
    const int b = inst % a.B;
    const int n = begin_rebuild(a, b, true);
    if (n < 0) return;
    const int lo = seg * a.seg_len, hi = min(n, lo + a.seg_len);
    int cnt = 0;
    if (lo < hi) {
        const Ladder r = make_ladder(a, b, n);
        cnt = compact_range<1>(a, r, (size_t)inst * a.cap, n, lo, hi, 0, tot0, tot1);
    }
    if (threadIdx.x == 0) a.seg_count[(size_t)inst * gridDim.x + seg] = cnt;
}

__global__ void __launch_bounds__(kThreads)
compact_write_kernel(CompactArgs a) {
    __shared__ int tot0[kWaves], tot1[kWaves];
    __shared__ int prefix;
    const int seg = blockIdx.x, inst = blockIdx.y;
    const int b = inst % a.B;
    const int n = begin_rebuild(a, b, false);
    if (n < 0) return;
    const int lo = seg * a.seg_len, hi = min(n, lo + a.seg_len);
    const int last = n > 0 ? (n - 1) / a.seg_len : 0;
    if (seg > last) return;
    if (threadIdx.x == 0) {
        int s = 0;
        for (int k = 0; k < seg; ++k) s += a.seg_count[(size_t)inst * gridDim.x + k];
        prefix = s;
    }
    __syncthreads();
    const size_t base = (size_t)inst * a.cap;
    int cnt = 0;
    if (lo < hi) {
        const Ladder r = make_ladder(a, b, n);
        cnt = compact_range<2>(a, r, base, n, lo, hi, prefix, tot0, tot1);
    }
    if (seg == last && threadIdx.x == 0) finish_list(a, inst, base, n, prefix + cnt);
}

__global__ void __launch_bounds__(kThreads)
compact_spill_kernel(CompactArgs a) {
    __shared__ int tot0[kWaves], tot1[kWaves];

    const int inst = blockIdx.x;
    const int b = inst % a.B;
    const int n = begin_rebuild(a, b, true);
    if (n < 0) return;
    const Ladder r = make_ladder(a, b, n);
    const size_t base = (size_t)inst * a.cap;
    int32_t* U = a.unfreeze + base;
    int32_t* list = a.list + base;
    int32_t* lrow = a.list_row + base;
    int32_t* row_of = a.row_of + base;
    uint8_t* on_host = a.on_host + base;
    int32_t* stack = a.free_rows + (size_t)inst * a.pool_rows;
    int32_t* out_pos = a.out_pos + base;
    int32_t* out_row = a.out_row + base;
    int32_t* in_pos = a.in_pos + base;
    int32_t* in_row = a.in_row + base;
    const int tid = threadIdx.x;
    const int top0 = a.free_top[inst];

    // pass 1: the freeze loop and recovery, then release the rows of tokens
    // frozen now for d >= spill_min_D
    int pushed = 0, n_out = 0;
    for (int p0 = 0; p0 < n; p0 += 4 * kThreads) {
        const int p = p0 + 4 * tid;
        Tile4 cur;
        load_tile(a, base, p, n, cur);
        int (&u)[4] = cur.u;
        int row[4];
        load4(row_of, p, n, row, -1);
        bool spill[4], first[4];
        bool dirty = freeze4(a, base, p, n, n, u, cur.c, cur.f);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            bool hit;
            const bool live = p + k < n;
            u[k] = recover(r, u[k], p + k, live, hit);
            dirty |= hit;
            // frozen at step t (U = t + d) for d >= spill_min_D, and still in a device row
            spill[k] = live & (row[k] >= 0) & (u[k] > r.t1) & (u[k] - a.t >= a.spill_min_D);
            const bool stored = live ? on_host[p + k] != 0 : true;
            first[k] = spill[k] & !stored;
        }
        if (dirty) {
            for (int k = 0; k < 4; ++k) if (p + k < n) U[p + k] = u[k];
        }
        int b0, m0, b1, m1;
        ballot4(spill, b0, m0);
        ballot4(first, b1, m1);
        const Scan sc = tile_scan(b0, m0, b1, m1, tot0, tot1);
        int ps = top0 + pushed + sc.off0, po = n_out + sc.off1;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (first[k]) {
                out_pos[po] = p + k;
                out_row[po] = row[k];
                on_host[p + k] = 1;
                ++po;
            }
            if (spill[k]) {
                if (ps < a.pool_rows) stack[ps] = row[k];
                row_of[p + k] = -1;
                ++ps;
            }
        }
        pushed += sc.tot0;
        n_out += sc.tot1;
    }
    __syncthreads();                          // stack and row_of writes are read below
    const int top = min(a.pool_rows, top0 + pushed);

    // pass 2: the active list of step t+1, device rows for positions that lack one
    int listed = 0, popped = 0;
    bool short_of_rows = false;
    for (int p0 = 0; p0 < n; p0 += 4 * kThreads) {
        const int p = p0 + 4 * tid;
        int u[4], row[4];
        load4(U, p, n, u, 0);
        load4(row_of, p, n, row, -1);
        bool flag[4], need[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            flag[k] = (p + k < n) & (u[k] <= r.t1);
            need[k] = flag[k] & (row[k] < 0);
        }
        int b0, m0, b1, m1;
        ballot4(flag, b0, m0);
        ballot4(need, b1, m1);
        const Scan sc = tile_scan(b0, m0, b1, m1, tot0, tot1);
        int pl = listed + sc.off0, pn = popped + sc.off1;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (!flag[k]) continue;
            int dev = row[k];
            if (need[k]) {
                const int idx = top - 1 - pn;
                if (idx >= 0) {
                    dev = stack[idx];
                    row_of[p + k] = dev;
                    in_pos[pn] = p + k;
                    in_row[pn] = dev;
                } else {
                    dev = 0;                  // no row left: results are void, the host is told
                    short_of_rows = true;
                }
                ++pn;
            }
            list[pl] = p + k;
            lrow[pl] = dev;
            ++pl;
        }
        listed += sc.tot0;
        popped += sc.tot1;
    }
    if (short_of_rows) a.flags[0] = 1;
    __syncthreads();
    if (tid == 0) {
        const int restored = min(popped, top);
        const int idx = top - 1 - popped;     // the next token's row
        int dev = 0;
        if (idx >= 0) {
            dev = stack[idx];
            row_of[n] = dev;
        } else {
            a.flags[0] = 1;
        }
        list[listed] = n;
        lrow[listed] = dev;
        a.free_top[inst] = max(0, idx);
        a.n_out[inst] = n_out;
        a.n_in[inst] = restored;
        a.n_active[inst] = listed + 1;
        atomicAdd(a.listed_total, (unsigned long long)(listed + 1));
        if (n_out) atomicAdd(a.xfer + 0, (unsigned long long)n_out);
        if (restored) atomicAdd(a.xfer + 1, (unsigned long long)restored);
        if (pushed) atomicAdd(a.xfer + 2, (unsigned long long)pushed);
    }
}

// Spill mode for few, long instances: the same two passes cut into segments,
// as three launches (pass 1 must push every released row before pass 2 pops).
//   S1  recovery, then per segment: released rows, rows to copy out, positions
//       that need a row back, listed positions;
//   S2  releases (pushes in position order after the counts of the segments
//       before), out-list entries;
//   S3  the list and the rows it needs (pops in position order), and the tail.
struct SegCounts {
    int spill, first, need, flag;
};

// seg_count holds, per instance, n_seg count records and one more whose first
// field is the stack height at the start of the rebuild (the last segment of
// S3 overwrites free_top while other segments may still read it).
__device__ __forceinline__ SegCounts seg_prefix(const CompactArgs& a, int inst, int seg) {
    const int4* c = reinterpret_cast<const int4*>(a.seg_count) + (size_t)inst * (a.n_seg + 1);
    SegCounts s{0, 0, 0, 0};
    for (int k = 0; k < seg; ++k) {
        const int4 v = c[k];
        s.spill += v.x; s.first += v.y; s.need += v.z; s.flag += v.w;
    }
    return s;
}

__global__ void __launch_bounds__(kThreads)
spill_count_kernel(CompactArgs a) {
    __shared__ int tot0[kWaves], tot1[kWaves];
    const int seg = blockIdx.x, inst = blockIdx.y;
    const int b = inst % a.B;
    const int n = begin_rebuild(a, b, true);
    if (n < 0) return;
    const int lo = seg * a.seg_len, hi = min(n, lo + a.seg_len);
    const Ladder r = make_ladder(a, b, n);
    const size_t base = (size_t)inst * a.cap;
    int32_t* U = a.unfreeze + base;
    const int32_t* row_of = a.row_of + base;
    const uint8_t* on_host = a.on_host + base;
    int ns = 0, nf = 0, nn = 0, nl = 0;
    for (int p0 = lo; p0 < hi; p0 += 4 * kThreads) {
        const int p = p0 + 4 * threadIdx.x;
        Tile4 cur;
        load_tile(a, base, p, hi, cur);
        int (&u)[4] = cur.u;
        int row[4];
        load4(row_of, p, hi, row, -1);
        bool spill[4], first[4], need[4], flag[4];
        bool dirty = freeze4(a, base, p, hi, n, u, cur.c, cur.f);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            bool hit;
            const bool live = p + k < hi;
            u[k] = recover(r, u[k], p + k, live, hit);
            dirty |= hit;
            spill[k] = live & (row[k] >= 0) & (u[k] > r.t1) & (u[k] - a.t >= a.spill_min_D);
            const bool stored = live ? on_host[p + k] != 0 : true;
            first[k] = spill[k] & !stored;
            flag[k] = live & (u[k] <= r.t1);
            need[k] = flag[k] & (row[k] < 0);
        }
        if (dirty) {
            for (int k = 0; k < 4; ++k) if (p + k < hi) U[p + k] = u[k];
        }
        int b0, m0, b1, m1;
        ballot4(spill, b0, m0);
        ballot4(first, b1, m1);
        const Scan s1 = tile_scan(b0, m0, b1, m1, tot0, tot1);
        ballot4(need, b0, m0);
        ballot4(flag, b1, m1);
        const Scan s2 = tile_scan(b0, m0, b1, m1, tot0, tot1);
        ns += s1.tot0; nf += s1.tot1; nn += s2.tot0; nl += s2.tot1;
    }
    if (threadIdx.x == 0) {
        int4* rec = reinterpret_cast<int4*>(a.seg_count) + (size_t)inst * (a.n_seg + 1);
        rec[seg] = make_int4(ns, nf, nn, nl);
        if (seg == 0) rec[a.n_seg] = make_int4(a.free_top[inst], 0, 0, 0);
    }
}

__global__ void __launch_bounds__(kThreads)
spill_push_kernel(CompactArgs a) {
    __shared__ int tot0[kWaves], tot1[kWaves];
    __shared__ SegCounts pre;
    const int seg = blockIdx.x, inst = blockIdx.y;
    const int b = inst % a.B;
    const int n = begin_rebuild(a, b, false);
    if (n < 0) return;
    const int lo = seg * a.seg_len, hi = min(n, lo + a.seg_len);
    if (lo >= hi) return;
    if (threadIdx.x == 0) pre = seg_prefix(a, inst, seg);
    __syncthreads();
    const Ladder r = make_ladder(a, b, n);
    const size_t base = (size_t)inst * a.cap;
    const int32_t* U = a.unfreeze + base;
    int32_t* row_of = a.row_of + base;
    uint8_t* on_host = a.on_host + base;
    int32_t* stack = a.free_rows + (size_t)inst * a.pool_rows;
    const int top0 = reinterpret_cast<const int4*>(a.seg_count)[(size_t)inst * (a.n_seg + 1) + a.n_seg].x;
    int pushed = pre.spill, n_out = pre.first;
    for (int p0 = lo; p0 < hi; p0 += 4 * kThreads) {
        const int p = p0 + 4 * threadIdx.x;
        int u[4], row[4];
        load4(U, p, hi, u, 0);                // already recovered by S1
        load4(row_of, p, hi, row, -1);
        bool spill[4], first[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const bool live = p + k < hi;
            spill[k] = live & (row[k] >= 0) & (u[k] > r.t1) & (u[k] - a.t >= a.spill_min_D);
            const bool stored = live ? on_host[p + k] != 0 : true;
            first[k] = spill[k] & !stored;
        }
        int b0, m0, b1, m1;
        ballot4(spill, b0, m0);
        ballot4(first, b1, m1);
        const Scan sc = tile_scan(b0, m0, b1, m1, tot0, tot1);
        int ps = top0 + pushed + sc.off0, po = n_out + sc.off1;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (first[k]) {
                a.out_pos[base + po] = p + k;
                a.out_row[base + po] = row[k];
                on_host[p + k] = 1;
                ++po;
            }
            if (spill[k]) {
                if (ps < a.pool_rows) stack[ps] = row[k];
                row_of[p + k] = -1;
                ++ps;
            }
        }
        pushed += sc.tot0;
        n_out += sc.tot1;
    }
}

__global__ void __launch_bounds__(kThreads)
spill_list_kernel(CompactArgs a) {
    __shared__ int tot0[kWaves], tot1[kWaves];
    __shared__ SegCounts pre, all;
    const int seg = blockIdx.x, inst = blockIdx.y;
    const int b = inst % a.B;
    const int n = begin_rebuild(a, b, false);
    if (n < 0) return;
    const int lo = seg * a.seg_len, hi = min(n, lo + a.seg_len);
    const int last = n > 0 ? (n - 1) / a.seg_len : 0;
    if (seg > last) return;
    if (threadIdx.x == 0) {
        pre = seg_prefix(a, inst, seg);
        all = seg_prefix(a, inst, a.n_seg);
    }
    __syncthreads();
    const Ladder r = make_ladder(a, b, n);
    const size_t base = (size_t)inst * a.cap;
    const int32_t* U = a.unfreeze + base;
    int32_t* row_of = a.row_of + base;
    const int32_t* stack = a.free_rows + (size_t)inst * a.pool_rows;
    const int top0 = reinterpret_cast<const int4*>(a.seg_count)[(size_t)inst * (a.n_seg + 1) + a.n_seg].x;
    const int top = min(a.pool_rows, top0 + all.spill);
    int listed = pre.flag, popped = pre.need;
    bool short_of_rows = false;
    for (int p0 = lo; p0 < hi; p0 += 4 * kThreads) {
        const int p = p0 + 4 * threadIdx.x;
        int u[4], row[4];
        load4(U, p, hi, u, 0);
        load4(row_of, p, hi, row, -1);
        bool flag[4], need[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            flag[k] = (p + k < hi) & (u[k] <= r.t1);
            need[k] = flag[k] & (row[k] < 0);
        }
        int b0, m0, b1, m1;
        ballot4(flag, b0, m0);
        ballot4(need, b1, m1);
        const Scan sc = tile_scan(b0, m0, b1, m1, tot0, tot1);
        int pl = listed + sc.off0, pn = popped + sc.off1;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (!flag[k]) continue;
            int dev = row[k];
            if (need[k]) {
                const int idx = top - 1 - pn;
                if (idx >= 0) {
                    dev = stack[idx];
                    row_of[p + k] = dev;
                    a.in_pos[base + pn] = p + k;
                    a.in_row[base + pn] = dev;
                } else {
                    dev = 0;                  // no row left: results are void, the host is told
                    short_of_rows = true;
                }
                ++pn;
            }
            a.list[base + pl] = p + k;
            a.list_row[base + pl] = dev;
            ++pl;
        }
        listed += sc.tot0;
        popped += sc.tot1;
    }
    if (short_of_rows) a.flags[0] = 1;
    if (seg == last && threadIdx.x == 0) {
        const int idx = top - 1 - all.need;   // the next token's row
        int dev = 0;
        if (idx >= 0) {
            dev = stack[idx];
            row_of[n] = dev;
        } else {
            a.flags[0] = 1;
        }
        a.list[base + all.flag] = n;
        a.list_row[base + all.flag] = dev;
        a.free_top[inst] = max(0, idx);
        const int restored = min(all.need, top);
        a.n_out[inst] = all.first;
        a.n_in[inst] = restored;
        a.n_active[inst] = all.flag + 1;
        atomicAdd(a.listed_total, (unsigned long long)(all.flag + 1));
        if (all.first) atomicAdd(a.xfer + 0, (unsigned long long)all.first);
        if (restored) atomicAdd(a.xfer + 1, (unsigned long long)restored);
        if (all.spill) atomicAdd(a.xfer + 2, (unsigned long long)all.spill);
    }
}

__global__ void __launch_bounds__(256)
spill_init_kernel(SpillInitArgs a) {
    const int inst = blockIdx.x;
    const int P = a.plen[inst % a.B];
    const size_t base = (size_t)inst * a.cap;
    for (int p = threadIdx.x; p < a.cap; p += blockDim.x) {
        a.row_of[base + p] = p < P ? p : -1;
        a.on_host[base + p] = 0;
    }
    const int free_n = max(0, a.pool_rows - P);
    int32_t* stack = a.free_rows + (size_t)inst * a.pool_rows;
    for (int k = threadIdx.x; k < free_n; k += blockDim.x) stack[k] = a.pool_rows - 1 - k;
    if (threadIdx.x == 0) a.free_top[inst] = free_n;
}

}  // namespace

hipError_t launch_compact(const CompactArgs& a, int n_instances, hipStream_t s) {
    if (a.spill_min_D > 0 && a.n_seg > 1) {
        const dim3 grid(a.n_seg, n_instances);
        hipLaunchKernelGGL(spill_count_kernel, grid, dim3(kThreads), 0, s, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(spill_push_kernel, grid, dim3(kThreads), 0, s, a);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(spill_list_kernel, grid, dim3(kThreads), 0, s, a);
    } else if (a.spill_min_D > 0) {
        hipLaunchKernelGGL(compact_spill_kernel, dim3(n_instances), dim3(kThreads), 0, s, a);
    } else if (a.n_seg <= 1) {
        hipLaunchKernelGGL(compact_kernel, dim3(n_instances), dim3(kThreads), 0, s, a);
    } else {
        const dim3 grid(a.n_seg, n_instances);
        hipLaunchKernelGGL(compact_count_kernel, grid, dim3(kThreads), 0, s, a);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(compact_write_kernel, grid, dim3(kThreads), 0, s, a);
    }
    return hipGetLastError();
}

int compact_segments(int n_instances, int cap, int* seg_len) {
    // enough workgroups to spread a few long instances over the device
    constexpr int kTile = 4 * kThreads;
    const int tiles = (cap + kTile - 1) / kTile;
    if (n_instances >= 256) {                 // already one workgroup per CU: no second pass
        *seg_len = cap;
        return 1;
    }
    int n_seg = (512 + n_instances - 1) / n_instances;
    if (n_seg > tiles) n_seg = tiles;
    if (n_seg < 1) n_seg = 1;
    const int per = (tiles + n_seg - 1) / n_seg;
    *seg_len = per * kTile;
    return (cap + *seg_len - 1) / *seg_len;
}

hipError_t launch_spill_init(const SpillInitArgs& a, int n_instances, hipStream_t s) {
    hipLaunchKernelGGL(spill_init_kernel, dim3(n_instances), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace asrkf
