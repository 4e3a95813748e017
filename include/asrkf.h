/*
 * asrkf.h -- C ABI of the MI355X (gfx950) decode-step library for
 * Adaptive Soft Rolling KV Freeze with Entropy-Guided Recovery
 * (arXiv 2512.11221).
 *
 * One context holds the KV cache and token states of n_layers x batch
 * (layer, sequence) instances.  A decode step is
 *
 *     for layer in 0 .. n_layers-1:  asrkf_decode_step(ctx, layer, ...)
 *     asrkf_restore(ctx, logits, mode, stream)
 *
 * decode_step is Algorithm 1 up to and including the freeze loop for one
 * layer of every sequence (attention over the active cache, Eq. 1; relevance,
 * Eq. 2; the freeze verdicts).  restore is the rest of the step: entropy
 * monitoring and staged recovery (Sec. 3.6), the freeze schedule of the step's
 * verdicts (Eq. 3), then the timer loop and the rebuild of every active cache
 * for the next step (Sec. 3.5).
 *
 * Conventions for every call:
 *  - Pointers named "device" must point to GPU memory of the current HIP
 *    device; "host" pointers to CPU memory.  Arrays are dense, row-major,
 *    in the layout given per argument.  The caller keeps ownership of every
 *    buffer it passes and keeps it valid until the work queued on `stream`
 *    has finished.  The library owns its cache, state, scratch and events.
 *  - `stream` is a hipStream_t passed as void*; NULL is the default stream.
 *    Calls marked "asynchronous" only queue work on that stream.  Successive
 *    calls on one context may use different streams: a call on another
 *    stream than the context's previous call first makes its stream wait for
 *    the work that call queued (the context's cache, states and scratch are
 *    shared by all calls).  Calls marked "waits" synchronize only the
 *    context's own streams, not the whole device.
 *  - Graph capture (resident mode): after the first decode step, a whole step
 *    (decode_step of every layer, then restore) may be captured on a stream
 *    into a HIP graph and replayed; the kernels take the step index from the
 *    context's device counter, so each replay runs the next step.  A captured
 *    call queues nothing until the graph is replayed.  The host learns of
 *    replayed steps at its next waiting call (asrkf_stats, asrkf_get_state,
 *    ...), which the caller makes before any further uncaptured decode_step.
 *    A replayed step that takes a sequence past max_ctx positions is caught
 *    on the device (the end-of-step rebuild is skipped, no access goes out
 *    of bounds) and reported as ECAPACITY by the next waiting call.  Capture
 *    returns ESTATE before the first decode step and in spill mode.
 *  - On any HIP runtime error the context is poisoned: that call returns
 *    ASRKF_EHIP and every later call returns ASRKF_ESTATE until destroy.
 *    asrkf_last_error() gives a message for the calling thread.
 *  - One host thread per context; calls on one context are not re-entrant.
 */
#ifndef ASRKF_H
#define ASRKF_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    ASRKF_OK = 0,
    ASRKF_EINVAL = -1,     /* bad argument or configuration; nothing done */
    ASRKF_ENOMEM = -2,     /* device or pinned host allocation failed */
    ASRKF_EHIP = -3,       /* HIP runtime error; context poisoned */
    ASRKF_ESTATE = -4,     /* call out of order, or context poisoned */
    ASRKF_ECAPACITY = -5   /* a sequence would exceed max_ctx positions, or (spill
                              mode) needed more than device_rows device rows */
} asrkf_status;

typedef enum { ASRKF_BF16 = 0, ASRKF_F32 = 1 } asrkf_dtype;

/* Recovery applied at the end of a step (Sec. 3.6 escalation ladder). */
typedef enum {
    ASRKF_AUTO = 0,   /* entropy-driven: level = consecutive spike steps, capped at FR */
    ASRKF_SR = 1,     /* Soft Reset: restore frozen tokens whose remaining timer > 1 */
    ASRKF_WR = 2,     /* Window Reset: restore frozen tokens among the last wr_last_N positions */
    ASRKF_FR = 3,     /* Full Reset: restore every frozen token (counts are kept) */
    ASRKF_NONE = 4    /* no recovery; entropy is still computed when logits are given */
} asrkf_recover;

/* Relevance score used by the freeze loop. */
typedef enum { ASRKF_REL_ABS = 0, ASRKF_REL_SOFTMAX = 1 } asrkf_relevance;

/* Scope of the token states. */
typedef enum { ASRKF_SCOPE_LAYER = 0, ASRKF_SCOPE_TOKEN = 1 } asrkf_scope;

/* Where the freeze loop takes its candidates, relative to the window of the
 * window_K most recent positions (the window includes the token appended this
 * step).  Algorithm 1 freezes tokens outside the window; Sec. 3.2 words the
 * estimate as made within the window. */
typedef enum { ASRKF_CAND_OUTSIDE = 0, ASRKF_CAND_INSIDE = 1 } asrkf_candidates;

typedef struct {
    int32_t n_layers;        /* >= 1 */
    int32_t batch;           /* sequences, 1 .. 1024 */
    int32_t n_q_heads;       /* H in Eq. 2 */
    int32_t n_kv_heads;      /* 1, 2, 4, 8, 16 or 32; n_q_heads / n_kv_heads in {1, 2, 4, 8};
                                with 16 KV heads at most 4 q heads per KV head, with 32 at
                                most 2, and for fp32 rows of 128 at most 16 KV heads */
    int32_t head_dim;        /* 64, 128 or 256 (256 with bf16 rows only) */
    int32_t max_ctx;         /* positions per sequence: prompt + decode steps */
    int32_t window_K;        /* protected window of most recent positions (Sec. 3.2; paper: 32) */
    float   tau;             /* relevance threshold, strict s_j < tau (paper: 0.5) */
    float   k_soft;          /* Eq. 3 softness k, in [2^-8, 2^16] (paper: 2) */
    int32_t vocab;           /* logits per sequence for entropy; >= 1 */
    float   entropy_spike;   /* theta_H in nats; +inf disables the entropy trigger */
    float   conf_drop;       /* theta_p on the top probability; <= 0 disables */
    int32_t wr_last_N;       /* Window Reset span in positions; <= 0 means 4 * window_K */
    int32_t dtype;           /* storage type of q, k, v: an asrkf_dtype value */
    int32_t spill_min_D;     /* 0: resident mode, frozen KV stays in HBM and only leaves
                                the active list.  >= 1: spill mode (Sec. 3.2, frozen KV
                                moved off the GPU): a token frozen for d >= spill_min_D
                                steps gives up its device row; its K and V rows are copied
                                once into a pinned host store and copied back into a free
                                device row at the end of the step before it attends again
                                (timer or recovery).  All copies run on a library stream
                                and are ordered before the attention that reads them. */
    int32_t device_rows;     /* spill mode: device KV rows per (layer, sequence), 0 means
                                max_ctx + 1 rounded up to 64; else 2 .. max_ctx + 1.  A
                                sequence that needs more rows than this voids the results
                                and the next call returns ECAPACITY.  Must be 0 in
                                resident mode. */
    int32_t history_W;       /* window of the detection count c_j (Eq. 3's history window W):
                                0 counts every detection; 1 .. 64 counts the detections of
                                the last history_W steps */
    int32_t relevance;       /* ASRKF_REL_ABS: Eq. 2, s_j = (1/H) sum_h |q_h . k_j|;
                                ASRKF_REL_SOFTMAX: s_j = (1/H) sum_h softmax weight of j
                                under head h (the share of attention j receives) */
    int32_t scope;           /* ASRKF_SCOPE_LAYER: token states per (layer, sequence);
                                ASRKF_SCOPE_TOKEN: one token state per sequence shared by
                                every layer (a frozen token leaves all layers), scored by
                                the mean of its per-layer relevance.  Not with spill mode. */
    int32_t candidates;      /* ASRKF_CAND_OUTSIDE (0, Algorithm 1): active tokens at positions
                                < n_t - window_K may freeze; ASRKF_CAND_INSIDE: active tokens at
                                positions >= n_t - window_K may freeze instead */
    float   debug_margin;    /* 0: off.  > 0: every freeze decision (an attended token that
                                may freeze, per `candidates`) taken on a relevance within
                                debug_margin of tau (|s_j - tau| < debug_margin, s_j as in
                                Eq. 2; token scope: its mean over layers) is counted in
                                asrkf_stats.margin_hits -- decisions that rounding can flip;
                                a run whose scores keep that margin reports 0 */
} asrkf_config;

typedef struct {
    int64_t step;               /* completed decode steps t */
    int64_t total_positions;    /* sum over (layer, seq) of positions n_t */
    int64_t active_positions;   /* sum over (layer, seq) of |{p < n_t : active at t+1}|
                                   -- the "Active KV" column of Table 1 */
    int64_t attended_total;     /* sum over completed steps and (layer, seq) of |A_t| */
    int64_t recoveries[4];      /* [1] SR, [2] WR, [3] FR applications (per sequence) */
    int64_t rr_requests;        /* steps at which the ladder asked for Rewalk Regeneration */
    int64_t attn_launches;      /* timed attention launches (asrkf_set_timing) */
    double  attn_kernel_ms;     /* summed duration of those launches */
    double  compression;        /* 1 - active_positions / total_positions */
    int64_t rows_to_host;       /* spill mode: tokens whose K and V rows were copied to the
                                   host store (each token at most once per layer) */
    int64_t rows_from_host;     /* spill mode: token rows copied back to the device */
    int64_t rows_released;      /* spill mode: device rows given up by freezing tokens */
    int64_t rows_reused;        /* spill mode: restored tokens that took back their last device
                                   row, which still held their K and V (no copy) */
    int64_t margin_hits;        /* debug_margin > 0: freeze decisions, over completed steps,
                                   on a relevance within debug_margin of tau */
} asrkf_stats_t;

typedef struct asrkf_ctx asrkf_ctx;

/* Allocate the cache and token states of every (layer, sequence): the
 * active cache A, frozen storage F and states S of Algorithm 1 (REQUIRE).
 * cfg: host.  On success *out receives the context.  Errors: EINVAL for a
 * configuration outside the documented ranges, ENOMEM, EHIP. */
asrkf_status asrkf_init(const asrkf_config* cfg, asrkf_ctx** out);

/* Copy the prompt KV of one (layer, sequence) into the cache (Sec. 3.1: the
 * pairs (K_j, V_j) of every previous token).  k, v: device,
 * [n_tokens][n_kv_heads][head_dim] of cfg.dtype.  Every layer of a sequence
 * must be given the same n_tokens (1 .. max_ctx-1); a sequence never
 * prefilled starts empty.  Only before the first decode step (else ESTATE).
 * Asynchronous. */
asrkf_status asrkf_prefill(asrkf_ctx* ctx, int32_t layer, int32_t seq,
                           const void* k, const void* v, int32_t n_tokens, void* stream);

/* Algorithm 1 up to the end of the freeze loop, for one layer of every
 * sequence: append the new token, attend over the active cache (Eq. 1),
 * score every attended token (Eq. 2), and decide which low-relevance tokens
 * outside the window of the window_K most recent positions (inside it with
 * ASRKF_CAND_INSIDE) freeze.  Their counts and Eq. 3 durations are applied to
 * the token states by asrkf_restore, before recovery, in one pass over every
 * layer's states; the states after restore are Algorithm 1's at the end of
 * the step.
 *   q:     device, [batch][n_q_heads][head_dim] of cfg.dtype
 *   k_new: device, [batch][n_kv_heads][head_dim] of cfg.dtype
 *   v_new: device, same layout as k_new
 *   out:   device, [batch][n_q_heads][head_dim] float32 (written)
 * Layers must come in order 0 .. n_layers-1 within a step (else ESTATE);
 * ECAPACITY when a sequence has no room for the new position.  Asynchronous. */
asrkf_status asrkf_decode_step(asrkf_ctx* ctx, int32_t layer, const void* q,
                               const void* k_new, const void* v_new, float* out,
                               void* stream);

/* asrkf_decode_step for callers that cannot allocate device memory when they
 * call (code under HIP graph capture, serving loops, harnesses that forbid
 * hipMalloc).  Same arguments, work and results as asrkf_decode_step (the same
 * kernels); it allocates nothing and creates no event.  Its split-K partials
 * (per partial slot and query head: head_dim + 2 floats; slots = attention
 * grid + batch, where the grid is the number of attention workgroups resident
 * at once, one per compute unit at the LLaMA-3-8B shape) live in a static
 * device array of 32 MiB that the library holds on every GPU it runs on until
 * the process ends; asrkf_init resolves its address on the context's device.
 * EINVAL, with nothing done, when the partials of this context exceed 32 MiB
 * ((grid + batch) * n_q_heads * (head_dim + 2) * 4 + 8 * batch bytes).  Every
 * call on one GPU shares the array and leaves its contents behind: calls on
 * one context are ordered (as for every call), but calls of different
 * contexts that overlap on one GPU (unordered streams) race.  Attention
 * timing (asrkf_set_timing) is not recorded by this call.  Asynchronous. */
asrkf_status asrkf_decode_step_static(asrkf_ctx* ctx, int32_t layer, const void* q,
                                      const void* k_new, const void* v_new, float* out,
                                      void* stream);

/* End the step: entropy of each sequence's next-token distribution and the
 * recovery ladder (Sec. 3.6), the step's freeze schedule (c_j += 1 and the
 * Eq. 3 duration for every token the step's decode_step calls found below
 * tau), the recovery level applied, then the timer loop and the active caches
 * of the next step (Algorithm 1 timer loop; Sec. 3.5).
 *   logits: device, [batch][vocab] float32, or NULL (no entropy; AUTO then
 *           applies no recovery)
 *   mode:   an asrkf_recover value; a forced level applies to every sequence;
 *           EINVAL for any other value.
 * Must follow decode_step of the last layer (else ESTATE).  Asynchronous. */
asrkf_status asrkf_restore(asrkf_ctx* ctx, const float* logits, int32_t mode,
                           void* stream);

/* Counters of the context (Table 1 columns, attended tokens, recoveries).
 * out: host.  Waits for all queued work of the context. */
asrkf_status asrkf_stats(asrkf_ctx* ctx, asrkf_stats_t* out);

/* Zero the cumulative counters (attended_total, recoveries, rr_requests,
 * attention timing).  Waits for all queued work of the context. */
asrkf_status asrkf_stats_reset(asrkf_ctx* ctx);

/* Have every attention launch record a pair of HIP events in its own
 * dispatch (enable != 0), so that asrkf_stats reports the kernel's summed
 * execution time.  Host-side switch. */
asrkf_status asrkf_set_timing(asrkf_ctx* ctx, int32_t enable);

/* The execution time of every timed attention launch since the last
 * asrkf_stats_reset, in launch order (milliseconds).
 *   ms:    host, room for cap values (may be NULL when cap = 0)
 *   count: receives the number of timed launches; min(cap, *count) values
 *          are written.
 * EINVAL for a null count or a negative cap.  Waits for all queued work of
 * the context. */
asrkf_status asrkf_timing_series(asrkf_ctx* ctx, float* ms, int64_t cap, int64_t* count);

/* Token states of one (layer, sequence) after the last completed step t
 * (test export; with ASRKF_SCOPE_TOKEN every layer shows the sequence's one
 * state).  All outputs are host buffers of at least max_ctx entries
 * (any may be NULL):
 *   n_positions:   receives n_t
 *   unfreeze_step: [n_t] step at which a frozen token attends again
 *                  (a token attends at step t' iff its value is <= t')
 *   count:         [n_t] low-relevance detections c_j (Eq. 3)
 *   frozen:        [n_t] 1 if the token is excluded at step t+1
 *   active:        ascending positions attended at step t+1 (including the
 *                  position the next token will take); *n_active their number
 * Waits for all queued work of the context. */
asrkf_status asrkf_get_state(asrkf_ctx* ctx, int32_t layer, int32_t seq,
                             int32_t* n_positions, int32_t* unfreeze_step, int32_t* count,
                             uint8_t* frozen, int32_t* active, int32_t* n_active);

/* Where the K and V rows of one (layer, sequence) live after the last
 * completed step (test export; Sec. 3.2 frozen storage).  Host outputs of at
 * least max_ctx entries, any may be NULL:
 *   n_positions: receives n_t
 *   device_row:  [n_t] row of the device cache holding the position, or -1
 *                when only the host store holds it (spill mode)
 *   on_host:     [n_t] 1 if the host store holds the position's rows
 * In resident mode device_row[p] = p and on_host is all 0.  Waits for all
 * queued work of the context. */
asrkf_status asrkf_get_residency(asrkf_ctx* ctx, int32_t layer, int32_t seq,
                                 int32_t* n_positions, int32_t* device_row, uint8_t* on_host);

/* Test hook for spill mode: before each step's row copies, the library's side
 * stream first runs a kernel that waits `microseconds` (0 = off, the default).
 * The attention of the next step must still read the restored rows, which
 * shows that it waits for the copies rather than for time.  Host-side switch;
 * EINVAL outside [0, 1e6]. */
asrkf_status asrkf_debug_delay_side(asrkf_ctx* ctx, int32_t microseconds);

/* Entropy monitor of one sequence after the last restore (Sec. 3.6):
 * entropy (nats), top probability, consecutive spike steps, level applied.
 * Host outputs, any may be NULL.  Waits for all queued work. */
asrkf_status asrkf_get_seq(asrkf_ctx* ctx, int32_t seq, float* entropy, float* pmax,
                           int32_t* escalation, int32_t* level);

/* Host-only helper: d(c) = floor(sqrt(c) / k) of Eq. 3 for c = 0 .. n-1,
 * exact for the float32 value k_soft (the table the library uses).
 * out: host, n entries.  EINVAL if k_soft is outside [2^-8, 2^16] or n < 1. */
asrkf_status asrkf_schedule_table(float k_soft, int32_t n, int32_t* out);

/* Return the context to the state asrkf_init leaves it in (no prompts, no
 * step, counters and timing cleared, timing off) and keep every allocation,
 * so that the next batch of sequences reuses the same device memory: prefill
 * follows as after asrkf_init.  ESTATE while the context's last stream is
 * being captured.  Waits for all queued work of the context. */
asrkf_status asrkf_reset(asrkf_ctx* ctx);

/* Free everything the context owns.  Waits for its queued work.  NULL is a no-op. */
void asrkf_destroy(asrkf_ctx* ctx);

/* Message of the last failed call on this thread ("" if none). */
const char* asrkf_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ASRKF_H */
