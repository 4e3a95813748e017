// Internal interface between the runtime (runtime.hip) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stdint.h>

namespace asrkf {

// Split-K attention.  The concatenated active lists of all sequences are cut
// into one equal contiguous token range per workgroup of a fixed grid
// (derived on the device from the active counts, no host round trip); the
// workgroup leaves one partial (m, l, acc) of every query head per sequence
// its range touches, at slot (workgroup + sequence).
constexpr int kMaxBatch = 1024;

// A low-relevance detection of the token at state index o in step t: the new
// count c_j (Eq. 3).  W = 0 counts every detection; otherwise a bit mask of
// the detections of the last W steps (bit i = step t - i) gives the count.
__device__ __forceinline__ int detect(int32_t* count, uint64_t* hmask, int32_t* hlast, size_t o,
                                      int t, int W) {
    int c;
    if (W == 0) {
        c = count[o] + 1;
    } else {
        const int gap = t - hlast[o];
        uint64_t m = gap >= 64 ? 0ull : (hmask[o] << gap);
        m |= 1ull;
        if (W < 64) m &= (1ull << W) - 1ull;
        hmask[o] = m;
        hlast[o] = t;
        c = __popcll(m);
    }
    count[o] = c;
    return c;
}

// Whether the token at position pos may be frozen.  wedge = n_t - K: positions
// >= wedge form the window of the K most recent positions (Sec. 3.2), which
// includes the token appended this step.  Algorithm 1 takes the candidates
// outside the window; inside = true takes those inside it instead.
__device__ __forceinline__ bool freeze_candidate(int pos, int wedge, bool inside) {
    return (pos < wedge) != inside;
}

struct AttnArgs {
    const void* kpool;        // layer base, [B][pool_rows][Hkv][D]
    const void* vpool;
    const void* q;            // [B][Hq][D]
    const void* knew;         // [B][Hkv][D]
    const void* vnew;
    void* kpool_w;            // same as kpool, writable (append)
    void* vpool_w;
    const int32_t* list;      // layer base, [B][cap] ascending positions
    const int32_t* list_row;  // layer base, [B][cap] device row of each listed position
                              // (spill mode only; in resident mode the row is the position)
    const int32_t* n_active;  // layer base, [B]
    uint8_t* flag;            // layer base, [B][cap]: bit 0 set where the attended position
                              // scores below tau (Eq. 2), bit 1 where the score lies within
                              // the debug margin of tau; read by the freeze loop at the
                              // end of the step
    int32_t* t_dev;           // first layer of a step: advanced by one (steps started), else null
    float* part_acc;          // [grid + B][Hq][D]
    float* part_ml;           // [grid + B][Hq][2]: (max in log2 units, sum)
    int32_t* slot_first;      // [B] first partial slot of each sequence (written)
    int32_t* slot_end;        // [B] one past its last slot (written)
    int32_t B, cap, Hq, Hkv;
    int32_t pool_rows;        // device rows per sequence (cap in resident mode)
    int32_t spill;            // 1: rows come from list_row
    float tau_H;              // tau * Hq: compared against sum_h |q_h . k_j|
    float margin_H;           // debug margin * Hq (0: off): a score this close to tau_H
                              // also sets bit 1 of the position's flag
    float scale_log2;         // log2(e) / sqrt(D)
    // relevance reading and state scope
    int32_t rel_mode;         // 0: Eq. 2 |q.k| scored here; 1: softmax weights (weight_relevance_kernel)
    int32_t scope_token;      // 1: one token state per sequence, scored by the sum over layers
    int32_t first_layer;      // token scope: this launch starts the per-token sums
    float* rel_acc;           // token scope, [B][cap]: sum over layers and heads of the relevance
    float* xlog;              // softmax relevance, [B][cap][Hq]: q.k * log2(e)/sqrt(D) per listed token
    const int32_t* plan;      // state base, [grid][kPlanInts] first-tile records of the ranges
                              // (plan_kernel), or null
};

// The first positions of every attention range, staged after each list
// rebuild, so that an attention workgroup can request its first K/V rows
// before its chunk's positions and q arrive.  Record of range w:
//   [0] sequence of the range's first piece, -1: the range has no real token
//   [1] the piece's first list index  [2] its first chunk's length  [3] unused
//   [4 .. 4 + kPlanTokens) list entries from the first list index on (the
//   last entry of the chunk repeated past its end)
constexpr int kPlanTokens = 32;
constexpr int kPlanInts = 4 + kPlanTokens;
constexpr int kPlanMinLayers = 4;   // fewer layers per step: no records (the launch costs more)

struct PlanArgs {
    const int32_t* list;      // [states][B][cap]
    const int32_t* n_active;  // [states][B]
    int32_t* plan;            // [states][grid][kPlanInts]
    int32_t B, cap, grid;
};

// Per layer, after the attention: the split combine of Eq. 1.
struct FinishArgs {
    const float* part_acc;
    const float* part_ml;
    const int32_t* slot_first;
    const int32_t* slot_end;
    float* out;               // [B][Hq][D]
    float* norm;              // softmax relevance: [B][Hq][2] (max, sum) of the sequence (written), or null
    int32_t B, Hq;
};

// Relevance by attention weight, after the split combine of a layer:
// s_j = sum_h 2^(y_hj - M_h) / L_h over the heads (compared with tau * Hq),
// then the score flag (layer scope) or the per-token sum (token scope).
struct RelevanceArgs {
    const float* xlog;        // [B][cap][Hq]
    const float* norm;        // [B][Hq][2]
    const int32_t* list;      // state base [B][cap]
    const int32_t* n_active;  // state base [B]
    uint8_t* flag;            // state base [B][cap]
    float* rel_acc;           // token scope [B][cap]
    int32_t B, cap, Hq, scope_token, first_layer;
    float tau_H, margin_H;
};

struct CompactArgs {
    int32_t* unfreeze;        // [L][B][cap]
    int32_t* list;            // [L][B][cap]
    int32_t* n_active;        // [L][B]
    const int32_t* plen;      // [B]
    const int32_t* level;     // [B] recovery level per sequence (may be null)
    unsigned long long* listed_total;  // running sum of list lengths
    int32_t forced_level;     // -1: read level[]; 0: none; 1..3 forced SR/WR/FR
    int32_t count_forced;     // 1: count a forced level (no logits) in recoveries[]
    unsigned long long* recoveries;  // [4], indexed by level 1..3
    const int32_t* t_dev;     // steps started (advanced by each step's first attention launch)
    int32_t t;                // completed step, read from t_dev; lists are built for step t+1
    int32_t max_ctx;          // positions per sequence; a rebuild that would pass it is refused
    int32_t* flags;           // [0] a sequence ran out of device rows (spill mode),
                              // [1] a step would pass max_ctx positions
    int32_t B, cap, wr_last_N;
    // spill mode only (spill_min_D > 0)
    int32_t spill_min_D;
    int32_t pool_rows;        // device rows per (layer, sequence)
    int32_t* row_of;          // [L][B][cap] device row of a position, -1: host store only
    uint8_t* on_host;         // [L][B][cap] 1: the host store holds the position's rows
    int32_t* list_row;        // [L][B][cap] device row of each listed position
    int32_t* last_row;        // [L][B][cap] the device row a host-only position held last
    int32_t* row_owner;       // [L][B][pool_rows] position whose K/V a row holds, -1: none
    int32_t* hand;            // [L][B] where the next search for free rows starts
    int32_t* pop_buf;         // [L][B][pool_rows] the free rows found for this rebuild
    int32_t* out_pos;         // [L][B][cap] rows to copy to the host store: position ...
    int32_t* out_row;         //   ... and the device row it leaves
    int32_t* n_out;           // [L][B]
    int32_t* in_pos;          // [L][B][cap] rows to copy back: position ...
    int32_t* in_row;          //   ... and the device row it takes
    int32_t* n_in;            // [L][B]
    unsigned long long* xfer; // [0] rows to host, [1] rows from host, [2] device rows released,
                              // [3] rows taken back intact (no copy)
    // the freeze loop of step t runs here, before recovery (not before step 1)
    int32_t freeze;           // 1: apply the step's freeze loop (set on the device: t > 0)
    const uint8_t* flag;      // [L][B][cap] layer scope: 1 where the position scored below tau at step t
    int32_t scope_token;      // 1: one state per sequence, scored by the sum over layers
    const float* rel_acc;     // [B][cap] token scope: relevance summed over layers and heads
    float tau_LH;             // tau * n_layers * Hq
    float margin_LH;          // token scope: debug margin * n_layers * Hq
    unsigned long long* margin_hits;  // debug margin on: decisions near tau are counted here
    int32_t* count;           // [L][B][cap] (or [B][cap] in token scope): c_j
    uint64_t* hmask;
    int32_t* hlast;
    const int32_t* dur;
    int32_t dur_len, history_W, window_K;
    int32_t cand_inside;      // 1: freeze candidates inside the window, 0: outside
    // segmented rebuild of few, long instances (n_seg > 1)
    int32_t n_seg, seg_len;
    int32_t* seg_count;       // [instances][n_seg] counts ([instances][n_seg + 1][4] in spill mode)
};

// First decode step in spill mode: prompt positions p < P sit in device rows
// p, the other rows are free (the search for free rows starts at row P),
// nothing is on the host.
struct SpillInitArgs {
    int32_t* row_of;
    uint8_t* on_host;
    int32_t* last_row;
    int32_t* row_owner;
    int32_t* hand;
    const int32_t* plen;
    int32_t B, cap, pool_rows;
};

// Row copies between the device cache and the host store (spill mode).
struct XferArgs {
    char* kpool;              // [L][B][pool_rows][row_bytes]
    char* vpool;
    char* khost;              // device-visible pointer of the pinned store, [L][B][cap][row_bytes]
    char* vhost;
    const int32_t* pos;       // [L][B][cap] per-instance lists of positions ...
    const int32_t* row;       //   ... and device rows
    const int32_t* count;     // [L][B] list lengths
    int32_t inst0;            // first (layer, sequence) instance of the launch
    int32_t cap, pool_rows, row_bytes;
    int32_t to_host;          // 1: device -> host store, 0: host store -> device
};

// Workgroups per sequence in the entropy pass: about 512 in all (measured: at
// batch 64, 8 per sequence take 12.8 us per step against 20.2 us for 32; more
// blocks per sequence wait longer on the sequence's ticket), 4 .. 32 each.
constexpr int kEntropySplitMax = 32;
constexpr int entropy_split(int B) {
    int s = kEntropySplitMax;
    while (s > 4 && s * B > 512) s >>= 1;
    return s;
}

struct EntropyArgs {
    const float* logits;      // [B][V]
    float* partial;           // [B][split][3] block triples (m, S, T)
    int32_t split;            // workgroups per sequence, 4 .. kEntropySplitMax
    int32_t* ticket;          // [B] blocks finished; reset by the last one
    int32_t V, B;
    float theta_H, theta_p;
    int32_t mode;             // 0 AUTO, 1..3 forced, 4 none
    int32_t* escalation;      // [B]
    int32_t* level;           // [B] (written)
    float* entropy;           // [B]
    float* pmax;              // [B]
    unsigned long long* recoveries;  // [4], indexed by level 1..3
    unsigned long long* rr_requests;
};

// start/stop (may be null) are recorded by the kernel's own dispatch.
hipError_t launch_attention(const AttnArgs& a, int dtype_bf16, int head_dim, int group,
                            int grid, hipStream_t s, hipEvent_t start, hipEvent_t stop);
hipError_t attention_occupancy(const AttnArgs& a, int dtype_bf16, int head_dim, int group,
                               int* blocks_per_cu);
// slots_per_seq: about how many partial slots a sequence has (grid / B + 1).
hipError_t launch_finish(const FinishArgs& a, int head_dim, int slots_per_seq, hipStream_t s);
hipError_t launch_compact(const CompactArgs& a, int n_instances, hipStream_t s);
// The first-tile records of every (state layer, range) after a list rebuild.
hipError_t launch_plan(const PlanArgs& a, int n_states, hipStream_t s);
// Segments per instance (and their length) for the rebuild; 1 = one workgroup per instance.
int compact_segments(int n_instances, int cap, int* seg_len);
hipError_t launch_weight_relevance(const RelevanceArgs& a, hipStream_t s);
hipError_t launch_spill_init(const SpillInitArgs& a, int n_instances, hipStream_t s);
hipError_t launch_xfer(const XferArgs& a, int n_instances, hipStream_t s);
// Whether the attention kernel handles this (dtype, head_dim, q heads per KV head, KV heads).
bool attention_shape_supported(int dtype_bf16, int head_dim, int group, int n_kv_heads);
hipError_t launch_delay(int microseconds, hipStream_t s);
hipError_t launch_entropy(const EntropyArgs& a, hipStream_t s);

}  // namespace asrkf
