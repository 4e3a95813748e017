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
//   pass 1  a token frozen at step t for d >= spill_min_D steps gives up its
//           device row; if the host store does not hold its rows yet (K and V
//           never change, so they are copied out once), the (position, row)
//           pair goes to the out-list.  A position of the new active list
//           without a device row takes its last row back when that row still
//           holds its K/V;
//   rows    the positions still without a row, and the next token, take free
//           rows found by a search that wraps around the rows;
//   pass 2  the list of the next step and the row of every entry; positions
//           that took a found row go to the in-list.
// The copies themselves are made by the transfer kernel (out-list first, so a
// row is read before it is handed out again).
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
constexpr int kDurLds = 1024;                 // Eq. 3 durations cached in LDS

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
__device__ __forceinline__ bool freeze4(const CompactArgs& a, const int32_t* dur_lds, size_t base,
                                        int p, int hi, int n, int (&u)[4], const int (&cnt)[4],
                                        uint32_t flags, const float (&rel)[4], int& near) {
    if (!a.freeze) return false;
    bool dirty = false;
    const bool inside = a.cand_inside != 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int q = p + k;
        bool low, close;
        if (a.scope_token) {
            low = rel[k] < a.tau_LH;
            close = fabsf(rel[k] - a.tau_LH) < a.margin_LH;
        } else {
            low = ((flags >> (8 * k)) & 1u) != 0;
            close = ((flags >> (8 * k)) & 2u) != 0;
        }
        // debug margin: a freeze decision of step t (an attended candidate) on a
        // score near tau
        near += (q < hi && u[k] <= a.t && close && freeze_candidate(q, n - a.window_K, inside)) ? 1 : 0;
        if (q < hi && u[k] <= a.t && low && freeze_candidate(q, n - a.window_K, inside)) {
            int c;
            if (a.history_W == 0) {
                c = cnt[k] + 1;
                a.count[base + q] = c;
            } else {
                c = detect(a.count, a.hmask, a.hlast, base + q, a.t, a.history_W);
            }
            // the LDS read is unconditional and the rare global read stays in a
            // branch of its own (volatile: not merged into a select between the two
            // addresses, a generic load whose wait also waits for every load in flight)
            int d = dur_lds[min(c, kDurLds - 1)];
            if (c >= kDurLds) d = *reinterpret_cast<const volatile int32_t*>(a.dur + min(c, a.dur_len - 1));
            if (d >= 1) {
                u[k] = a.t + d;
                dirty = true;
            }
        }
    }
    return dirty;
}

// Debug margin: the decisions near tau a thread counted, added to the
// context's counter (one atomic per wave).  Every thread of the wave calls it.
__device__ __forceinline__ void add_margin_hits(const CompactArgs& a, int near) {
    if (!a.margin_hits) return;               // uniform
    for (int o = 32; o > 0; o >>= 1) near += __shfl_xor(near, o);
    if ((threadIdx.x & 63) == 0 && near) atomicAdd(a.margin_hits, (unsigned long long)near);
}

// Eq. 3 durations of the counts below kDurLds, staged in LDS by every
// workgroup that runs the freeze loop (one load per thread, before its tiles).
__device__ __forceinline__ void load_durations(const CompactArgs& a, int32_t* dur_lds) {
    if (!a.freeze) return;                    // uniform over the workgroup
    for (int c = threadIdx.x; c < kDurLds; c += kThreads) dur_lds[c] = a.dur[min(c, a.dur_len - 1)];
    __syncthreads();
}

// U, counts and flags of the 4 positions p .. p+3, loaded as they are: the
// entries at or past the range end hold whatever the rows hold there, and
// every use checks the position first.  Counts and flags are loaded in every
// mode (the arrays always exist), so the loads sit in straight-line code:
// a load inside a branch makes the compiler wait for it, and for everything
// in flight before it, before the branches join.  State rows hold cap
// entries, a multiple of 64, and start 16-byte aligned, so the load at
// min(p, cap - 4) stays inside the row for any p.
struct Tile4 {
    int u[4], c[4];
    uint32_t f;
    float r[4];                               // token scope: relevance summed over layers
};

__device__ __forceinline__ void load_tile(const CompactArgs& a, size_t base, int p, Tile4& x) {
    const size_t q = base + (size_t)min(p, a.cap - 4);
    const int4 u = *reinterpret_cast<const int4*>(a.unfreeze + q);
    const int4 c = *reinterpret_cast<const int4*>(a.count + q);
    x.f = *reinterpret_cast<const uint32_t*>(a.flag + q);
    if (a.scope_token) {                      // uniform; the sums exist in token scope only
        const float4 r = *reinterpret_cast<const float4*>(a.rel_acc + q);
        x.r[0] = r.x; x.r[1] = r.y; x.r[2] = r.z; x.r[3] = r.w;
    }
    x.u[0] = u.x; x.u[1] = u.y; x.u[2] = u.z; x.u[3] = u.w;
    x.c[0] = c.x; x.c[1] = c.y; x.c[2] = c.z; x.c[3] = c.w;
}

__device__ __forceinline__ void load_u(const int32_t* U, int p, int cap, int (&u)[4]) {
    const int4 x = *reinterpret_cast<const int4*>(U + min(p, cap - 4));
    u[0] = x.x; u[1] = x.y; u[2] = x.z; u[3] = x.w;
}

// The entries of a loaded tile at or past hi set to their neutral values
// (U 0, count 0, flag 0), for code that reads them without checking.
__device__ __forceinline__ void mask_tile(Tile4& x, int p, int hi) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        if (p + k >= hi) {
            x.u[k] = 0;
            x.c[k] = 0;
            x.f &= ~(0xFFu << (8 * k));
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
// the already updated U.  List entries start at list + out_base.  The next
// tile's loads are in flight while a tile is processed.  Returns the number
// of listed positions (the same value in every thread).
template <int MODE>
__device__ int compact_range(const CompactArgs& a, const Ladder& r, const int32_t* dur_lds, size_t base,
                             int n, int lo, int hi, int out_base, int* tot0, int* tot1) {
    int32_t* U = a.unfreeze + base;
    int32_t* list = a.list + base;
    const int tid = threadIdx.x;
    int listed = 0, near = 0;
    Tile4 next;
    if constexpr (MODE != 2) load_tile(a, base, lo + 4 * tid, next);
    else load_u(U, lo + 4 * tid, a.cap, next.u);
    for (int p0 = lo; p0 < hi; p0 += 4 * kThreads) {
        const int p = p0 + 4 * tid;
        Tile4 cur = next;
        int (&u)[4] = cur.u;
        if (p0 + 4 * kThreads < hi) {                                            // next tile in flight
            if constexpr (MODE != 2) load_tile(a, base, p + 4 * kThreads, next);
            else load_u(U, p + 4 * kThreads, a.cap, next.u);
        }
        bool flag[4];
        if constexpr (MODE != 2) {
            bool dirty = freeze4(a, dur_lds, base, p, hi, n, u, cur.c, cur.f, cur.r, near);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                bool hit;
                const bool live = p + k < hi;
                u[k] = recover(r, u[k], p + k, live, hit);
                dirty |= hit;
                flag[k] = live & (u[k] <= r.t1);
            }
            if (dirty) {
                if (p + 3 < hi) *reinterpret_cast<int4*>(U + p) = make_int4(u[0], u[1], u[2], u[3]);
                else for (int k = 0; k < 4; ++k) if (p + k < hi) U[p + k] = u[k];
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
    if constexpr (MODE != 2) add_margin_hits(a, near);
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
    __shared__ int32_t dur_lds[kDurLds];
    const int inst = blockIdx.x;
    const int b = inst % a.B;
    const int n = begin_rebuild(a, b, true);        // positions after step t
    if (n < 0) return;
    const Ladder r = make_ladder(a, b, n);
    const size_t base = (size_t)inst * a.cap;
    load_durations(a, dur_lds);
    const int listed = compact_range<0>(a, r, dur_lds, base, n, 0, n, 0, tot0, tot1);
    if (threadIdx.x == 0) finish_list(a, inst, base, n, listed);
}

// Few, long instances: each instance is cut into segments of seg_len
// positions, one workgroup each.  Pass A applies the updates and counts each
// segment; pass B adds the counts of the segments before it and writes.
__global__ void __launch_bounds__(kThreads)
compact_count_kernel(CompactArgs a) {
    __shared__ int tot0[kWaves], tot1[kWaves];
    __shared__ int32_t dur_lds[kDurLds];
    const int seg = blockIdx.x, inst = blockIdx.y;
    const int b = inst % a.B;
    const int n = begin_rebuild(a, b, true);
    if (n < 0) return;
    load_durations(a, dur_lds);
    const int lo = seg * a.seg_len, hi = min(n, lo + a.seg_len);
    int cnt = 0;
    if (lo < hi) {
        const Ladder r = make_ladder(a, b, n);
        cnt = compact_range<1>(a, r, dur_lds, (size_t)inst * a.cap, n, lo, hi, 0, tot0, tot1);
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
        cnt = compact_range<2>(a, r, nullptr, base, n, lo, hi, prefix, tot0, tot1);
    }
    if (seg == last && threadIdx.x == 0) finish_list(a, inst, base, n, prefix + cnt);
}

// ---- spill mode ----
// A token frozen at step t for d >= spill_min_D steps gives up its device row
// (row_of = -1; last_row remembers the row).  The row is then free, but it keeps
// the token's K/V until another position is written into it: every row records
// its owner, the position whose K/V it holds, and is free unless that owner
// currently sits in it,
//     free(r) = owner[r] < 0 || row_of[owner[r]] != r.
// A host-only position that attends again takes its last row back when the row
// still holds its K/V (no copy), else a free row that a search finds, and its
// K/V comes back from the host store.  The search starts where the previous
// one stopped and wraps around the rows, so a released row is handed out again
// as late as the free rows allow.  Every decision is taken in ascending
// position or row order, so the assignment is the same on every run.

__device__ __forceinline__ bool row_free(const int32_t* owner, const int32_t* row_of, int r) {
    const int o = owner[r];
    return o < 0 || row_of[o] != r;
}

// Releases, out-list entries and take-backs of the positions p .. p+3 of a
// thread (recovery already applied to u): released[k] for tokens frozen now
// for d >= spill_min_D that still hold a row (first[k]: the host store does not
// hold them yet), need[k] for listed positions without a row after the
// take-backs, back[k] for the take-backs.  Writes row_of, last_row, on_host.
struct SpillFlags {
    bool released[4], first[4], need[4], back[4], listed[4];
    int row[4];
};

__device__ __forceinline__ void spill_decide(const CompactArgs& a, const Ladder& r, size_t base,
                                             int p, int hi, const int (&u)[4], SpillFlags& f) {
    int32_t* row_of = a.row_of + base;
    int32_t* last_row = a.last_row + base;
    const int32_t* owner = a.row_owner + (base / a.cap) * a.pool_rows;
    int row[4];
    load4(row_of, p, hi, row, -1);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const bool live = p + k < hi;
        f.listed[k] = live & (u[k] <= r.t1);
        // frozen at step t (U = t + d) for d >= spill_min_D, and still in a device row
        f.released[k] = live & (row[k] >= 0) & (u[k] > r.t1) & (u[k] - a.t >= a.spill_min_D);
        const bool stored = live ? a.on_host[base + p + k] != 0 : true;
        f.first[k] = f.released[k] & !stored;
        f.back[k] = false;
        if (f.released[k]) {
            row_of[p + k] = -1;
            last_row[p + k] = row[k];
            if (f.first[k]) a.on_host[base + p + k] = 1;
            row[k] = -1;
        } else if (f.listed[k] && row[k] < 0) {
            const int lr = last_row[p + k];
            if (lr >= 0 && owner[lr] == p + k) {           // its K/V is still in its last row
                row_of[p + k] = lr;
                row[k] = lr;
                f.back[k] = true;
            }
        }
        f.need[k] = f.listed[k] & (row[k] < 0);
        f.row[k] = row[k];
    }
}

// The first `need` free rows from the instance's hand on, in cyclic row order,
// into pop_buf[0 .. need); returns how many there were (fewer when the rows ran
// out) and moves the hand past the last one taken.  Every thread of the block
// calls it.
__device__ int find_free_rows(const CompactArgs& a, int inst, int need, int* tot0, int* tot1,
                              int* last_idx) {
    const int R = a.pool_rows;
    const int32_t* owner = a.row_owner + (size_t)inst * R;
    const int32_t* row_of = a.row_of + (size_t)inst * a.cap;
    int32_t* pop = a.pop_buf + (size_t)inst * R;
    const int h0 = a.hand[inst];
    int found = 0;
    if (threadIdx.x == 0) *last_idx = -1;
    for (int s0 = 0; s0 < R && found < need; s0 += 4 * kThreads) {
        bool f[4];
        int rw[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int i = s0 + 4 * threadIdx.x + k;
            rw[k] = (h0 + i) % R;
            f[k] = i < R && row_free(owner, row_of, rw[k]);
        }
        int before, mine;
        ballot4(f, before, mine);
        const Scan sc = tile_scan(before, mine, 0, 0, tot0, tot1);
        int slot = found + sc.off0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (!f[k]) continue;
            if (slot < need) pop[slot] = rw[k];
            if (slot == need - 1) *last_idx = s0 + 4 * threadIdx.x + k;
            ++slot;
        }
        found += sc.tot0;
    }
    __syncthreads();                          // last_idx; every thread has read the hand
    if (threadIdx.x == 0 && *last_idx >= 0) a.hand[inst] = (h0 + *last_idx + 1) % R;
    return min(found, need);
}

// The list of step t+1 for positions p .. p+3, with the device row of each;
// listed positions that need a row take pop_buf[pn], pn counting up (their K/V
// comes back from the host store: in-list).
__device__ __forceinline__ void spill_list4(const CompactArgs& a, size_t base, int inst, int p,
                                            const SpillFlags& f, int pl, int pn, int popped,
                                            bool& short_of_rows) {
    int32_t* owner = a.row_owner + (size_t)inst * a.pool_rows;
    const int32_t* pop = a.pop_buf + (size_t)inst * a.pool_rows;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        if (!f.listed[k]) continue;
        int dev = f.row[k];
        if (f.need[k]) {
            if (pn < popped) {
                dev = pop[pn];
                a.row_of[base + p + k] = dev;
                owner[dev] = p + k;
                a.in_pos[base + pn] = p + k;
                a.in_row[base + pn] = dev;
            } else {
                dev = 0;                      // no row left: results are void, the host is told
                short_of_rows = true;
            }
            ++pn;
        }
        a.list[base + pl] = p + k;
        a.list_row[base + pl] = dev;
        ++pl;
    }
}

// The list tail: the next token's position n and the row it takes (the last
// row found); counts and counters of the rebuild.
__device__ __forceinline__ void spill_tail(const CompactArgs& a, int inst, size_t base, int n,
                                           int listed, int need, int popped, int n_out,
                                           int released, int back) {
    int dev = 0;
    if (need < popped) {
        dev = a.pop_buf[(size_t)inst * a.pool_rows + need];
        a.row_of[base + n] = dev;
        a.row_owner[(size_t)inst * a.pool_rows + dev] = n;
    } else {
        a.flags[0] = 1;
    }
    a.list[base + listed] = n;
    a.list_row[base + listed] = dev;
    const int restored = min(need, popped);
    a.n_out[inst] = n_out;
    a.n_in[inst] = restored;
    a.n_active[inst] = listed + 1;
    atomicAdd(a.listed_total, (unsigned long long)(listed + 1));
    if (n_out) atomicAdd(a.xfer + 0, (unsigned long long)n_out);
    if (restored) atomicAdd(a.xfer + 1, (unsigned long long)restored);
    if (released) atomicAdd(a.xfer + 2, (unsigned long long)released);
    if (back) atomicAdd(a.xfer + 3, (unsigned long long)back);
}

__global__ void __launch_bounds__(kThreads)
compact_spill_kernel(CompactArgs a) {
    __shared__ int tot0[kWaves], tot1[kWaves];
    __shared__ int last_idx;
    __shared__ int32_t dur_lds[kDurLds];

    const int inst = blockIdx.x;
    const int b = inst % a.B;
    const int n = begin_rebuild(a, b, true);
    if (n < 0) return;
    load_durations(a, dur_lds);
    const Ladder r = make_ladder(a, b, n);
    const size_t base = (size_t)inst * a.cap;
    int32_t* U = a.unfreeze + base;
    const int tid = threadIdx.x;

    // pass 1: the freeze loop, recovery, releases (out-list), take-backs, and the
    // number of positions that need a row
    int n_out = 0, released = 0, back = 0, need = 0, near = 0;
    for (int p0 = 0; p0 < n; p0 += 4 * kThreads) {
        const int p = p0 + 4 * tid;
        Tile4 cur;
        load_tile(a, base, p, cur);
        mask_tile(cur, p, n);
        int (&u)[4] = cur.u;
        bool dirty = freeze4(a, dur_lds, base, p, n, n, u, cur.c, cur.f, cur.r, near);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            bool hit;
            u[k] = recover(r, u[k], p + k, p + k < n, hit);
            dirty |= hit;
        }
        if (dirty) {
            for (int k = 0; k < 4; ++k) if (p + k < n) U[p + k] = u[k];
        }
        SpillFlags f;
        spill_decide(a, r, base, p, n, u, f);
        int b0, m0, b1, m1;
        ballot4(f.first, b0, m0);
        ballot4(f.released, b1, m1);
        const Scan s1 = tile_scan(b0, m0, b1, m1, tot0, tot1);
        int po = n_out + s1.off0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (!f.first[k]) continue;
            a.out_pos[base + po] = p + k;
            a.out_row[base + po] = a.last_row[base + p + k];
            ++po;
        }
        ballot4(f.need, b0, m0);
        ballot4(f.back, b1, m1);
        const Scan s2 = tile_scan(b0, m0, b1, m1, tot0, tot1);
        n_out += s1.tot0;
        released += s1.tot1;
        need += s2.tot0;
        back += s2.tot1;
    }
    __syncthreads();                          // row_of and last_row writes are read below

    // the rows for the positions that need one, and one for the next token
    const int popped = find_free_rows(a, inst, need + 1, tot0, tot1, &last_idx);

    add_margin_hits(a, near);

    // pass 2: the active list of step t+1 and the device row of every entry
    int listed = 0, pn_run = 0;
    bool short_of_rows = false;
    for (int p0 = 0; p0 < n; p0 += 4 * kThreads) {
        const int p = p0 + 4 * tid;
        int u[4];
        load4(U, p, n, u, 0);
        SpillFlags f;
        int row[4];
        load4(a.row_of + base, p, n, row, -1);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            f.listed[k] = (p + k < n) & (u[k] <= r.t1);
            f.need[k] = f.listed[k] & (row[k] < 0);
            f.row[k] = row[k];
        }
        int b0, m0, b1, m1;
        ballot4(f.listed, b0, m0);
        ballot4(f.need, b1, m1);
        const Scan sc = tile_scan(b0, m0, b1, m1, tot0, tot1);
        spill_list4(a, base, inst, p, f, listed + sc.off0, pn_run + sc.off1, popped, short_of_rows);
        listed += sc.tot0;
        pn_run += sc.tot1;
    }
    if (short_of_rows) a.flags[0] = 1;
    __syncthreads();
    if (tid == 0) spill_tail(a, inst, base, n, listed, need, popped, n_out, released, back);
}

// Spill mode for few, long instances: the same passes cut into segments of
// seg_len positions, as four launches:
//   S1  the freeze loop and recovery; per segment: positions listed
//   S2  releases, out-list entries (after the counts of the segments before),
//       take-backs; per segment: positions that need a row, releases, take-backs
//   S3  one workgroup per instance: the free rows for the positions that need
//       one and for the next token
//   S4  the list and the rows of its entries, and the tail.
struct SegCounts {
    int first, released, need, listed, back, pad0, pad1, pad2;
};

// seg_count holds, per instance, n_seg count records and one more whose first
// field is the number of free rows found (S3).
__device__ __forceinline__ SegCounts* seg_records(const CompactArgs& a, int inst) {
    return reinterpret_cast<SegCounts*>(a.seg_count) + (size_t)inst * (a.n_seg + 1);
}

__device__ __forceinline__ SegCounts seg_prefix(const CompactArgs& a, int inst, int seg) {
    const SegCounts* c = seg_records(a, inst);
    SegCounts s{0, 0, 0, 0, 0, 0, 0, 0};
    for (int k = 0; k < seg; ++k) {
        s.first += c[k].first; s.released += c[k].released; s.need += c[k].need;
        s.listed += c[k].listed; s.back += c[k].back;
    }
    return s;
}

__global__ void __launch_bounds__(kThreads)
spill_count_kernel(CompactArgs a) {
    __shared__ int tot0[kWaves], tot1[kWaves];
    __shared__ int32_t dur_lds[kDurLds];
    const int seg = blockIdx.x, inst = blockIdx.y;
    const int b = inst % a.B;
    const int n = begin_rebuild(a, b, true);
    if (n < 0) return;
    load_durations(a, dur_lds);
    const int lo = seg * a.seg_len, hi = min(n, lo + a.seg_len);
    const Ladder r = make_ladder(a, b, n);
    const size_t base = (size_t)inst * a.cap;
    int32_t* U = a.unfreeze + base;
    int nl = 0, nf = 0, near = 0;
    for (int p0 = lo; p0 < hi; p0 += 4 * kThreads) {
        const int p = p0 + 4 * threadIdx.x;
        Tile4 cur;
        load_tile(a, base, p, cur);
        mask_tile(cur, p, hi);
        int (&u)[4] = cur.u;
        int row[4];
        load4(a.row_of + base, p, hi, row, -1);
        bool dirty = freeze4(a, dur_lds, base, p, hi, n, u, cur.c, cur.f, cur.r, near);
        bool listed[4], first[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            bool hit;
            const bool live = p + k < hi;
            u[k] = recover(r, u[k], p + k, live, hit);
            dirty |= hit;
            listed[k] = live & (u[k] <= r.t1);
            const bool rel = live & (row[k] >= 0) & (u[k] > r.t1) & (u[k] - a.t >= a.spill_min_D);
            first[k] = rel & (live ? a.on_host[base + p + k] == 0 : false);
        }
        if (dirty) {
            for (int k = 0; k < 4; ++k) if (p + k < hi) U[p + k] = u[k];
        }
        int b0, m0, b1, m1;
        ballot4(listed, b0, m0);
        ballot4(first, b1, m1);
        const Scan sc = tile_scan(b0, m0, b1, m1, tot0, tot1);
        nl += sc.tot0;
        nf += sc.tot1;
    }
    add_margin_hits(a, near);
    if (threadIdx.x == 0) {
        SegCounts* rec = seg_records(a, inst);
        rec[seg].listed = nl;
        rec[seg].first = nf;
    }
}

__global__ void __launch_bounds__(kThreads)
spill_release_kernel(CompactArgs a) {
    __shared__ int tot0[kWaves], tot1[kWaves];
    __shared__ SegCounts pre;
    const int seg = blockIdx.x, inst = blockIdx.y;
    const int b = inst % a.B;
    const int n = begin_rebuild(a, b, false);
    if (n < 0) return;
    const int lo = seg * a.seg_len, hi = min(n, lo + a.seg_len);
    if (threadIdx.x == 0) pre = seg_prefix(a, inst, seg);
    __syncthreads();
    const Ladder r = make_ladder(a, b, n);
    const size_t base = (size_t)inst * a.cap;
    int n_out = pre.first, nr = 0, nn = 0, nb = 0;
    for (int p0 = lo; p0 < hi; p0 += 4 * kThreads) {
        const int p = p0 + 4 * threadIdx.x;
        int u[4];
        load4(a.unfreeze + base, p, hi, u, 0);      // already updated by S1
        SpillFlags f;
        spill_decide(a, r, base, p, hi, u, f);
        int b0, m0, b1, m1;
        ballot4(f.first, b0, m0);
        ballot4(f.released, b1, m1);
        const Scan s1 = tile_scan(b0, m0, b1, m1, tot0, tot1);
        int po = n_out + s1.off0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (!f.first[k]) continue;
            a.out_pos[base + po] = p + k;
            a.out_row[base + po] = a.last_row[base + p + k];
            ++po;
        }
        ballot4(f.need, b0, m0);
        ballot4(f.back, b1, m1);
        const Scan s2 = tile_scan(b0, m0, b1, m1, tot0, tot1);
        n_out += s1.tot0;
        nr += s1.tot1;
        nn += s2.tot0;
        nb += s2.tot1;
    }
    if (threadIdx.x == 0) {
        SegCounts* rec = seg_records(a, inst);
        rec[seg].released = nr;
        rec[seg].need = nn;
        rec[seg].back = nb;
    }
}

__global__ void __launch_bounds__(kThreads)
spill_rows_kernel(CompactArgs a) {
    __shared__ int tot0[kWaves], tot1[kWaves];
    __shared__ int last_idx, need;
    const int inst = blockIdx.x;
    const int b = inst % a.B;
    const int n = begin_rebuild(a, b, false);
    if (n < 0) return;
    if (threadIdx.x == 0) need = seg_prefix(a, inst, a.n_seg).need;
    __syncthreads();
    const int popped = find_free_rows(a, inst, need + 1, tot0, tot1, &last_idx);
    if (threadIdx.x == 0) seg_records(a, inst)[a.n_seg].first = popped;
}

__global__ void __launch_bounds__(kThreads)
spill_list_kernel(CompactArgs a) {
    __shared__ int tot0[kWaves], tot1[kWaves];
    __shared__ SegCounts pre, all;
    __shared__ int popped;
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
        popped = seg_records(a, inst)[a.n_seg].first;
    }
    __syncthreads();
    const Ladder r = make_ladder(a, b, n);
    const size_t base = (size_t)inst * a.cap;
    int listed = pre.listed, pn_run = pre.need;
    bool short_of_rows = false;
    for (int p0 = lo; p0 < hi; p0 += 4 * kThreads) {
        const int p = p0 + 4 * threadIdx.x;
        int u[4], row[4];
        load4(a.unfreeze + base, p, hi, u, 0);
        load4(a.row_of + base, p, hi, row, -1);
        SpillFlags f;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            f.listed[k] = (p + k < hi) & (u[k] <= r.t1);
            f.need[k] = f.listed[k] & (row[k] < 0);
            f.row[k] = row[k];
        }
        int b0, m0, b1, m1;
        ballot4(f.listed, b0, m0);
        ballot4(f.need, b1, m1);
        const Scan sc = tile_scan(b0, m0, b1, m1, tot0, tot1);
        spill_list4(a, base, inst, p, f, listed + sc.off0, pn_run + sc.off1, popped, short_of_rows);
        listed += sc.tot0;
        pn_run += sc.tot1;
    }
    if (short_of_rows) a.flags[0] = 1;
    if (seg == last && threadIdx.x == 0)
        spill_tail(a, inst, base, n, all.listed, all.need, popped, all.first, all.released, all.back);
}

__global__ void __launch_bounds__(256)
spill_init_kernel(SpillInitArgs a) {
    const int inst = blockIdx.x;
    const int P = a.plen[inst % a.B];
    const size_t base = (size_t)inst * a.cap;
    for (int p = threadIdx.x; p < a.cap; p += blockDim.x) {
        a.row_of[base + p] = p < P ? p : -1;
        a.last_row[base + p] = -1;
        a.on_host[base + p] = 0;
    }
    int32_t* owner = a.row_owner + (size_t)inst * a.pool_rows;
    for (int r = threadIdx.x; r < a.pool_rows; r += blockDim.x) owner[r] = r < P ? r : -1;
    if (threadIdx.x == 0) a.hand[inst] = a.pool_rows > P ? P : 0;
}

}  // namespace

hipError_t launch_compact(const CompactArgs& a, int n_instances, hipStream_t s) {
    if (a.spill_min_D > 0 && a.n_seg > 1) {
        const dim3 grid(a.n_seg, n_instances);
        hipLaunchKernelGGL(spill_count_kernel, grid, dim3(kThreads), 0, s, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(spill_release_kernel, grid, dim3(kThreads), 0, s, a);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(spill_rows_kernel, dim3(n_instances), dim3(kThreads), 0, s, a);
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
