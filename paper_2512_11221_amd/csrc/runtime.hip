// Context, memory layout and the C ABI declared in include/asrkf.h.
//
// HBM layout of a context (cap = max_ctx + 1 rounded up to 64 positions;
// pool_rows = cap in resident mode, the configured device rows in spill mode):
//   K, V cache      [L][B][pool_rows][Hkv][D]   dtype   token-major rows
//   unfreeze U      [L][B][cap]           int32   token attends at step t iff U <= t
//   count c         [L][B][cap]           int32   low-relevance detections (Eq. 3)
//   score flag      [L][B][cap]           uint8   s_j < tau at the current step (Eq. 2)
//   active list     [L][B][cap]           int32   ascending positions for the step
//   n_active        [L][B]                int32
//   partials        [grid+B][Hq][D+2]     fp32    split-K attention partials
//   plan records    [L][grid][36]         int32   first tile of every attention range
//                                                 (resident mode, four or more layers)
//   per sequence    prompt length, escalation, level, entropy, p_max
//   duration table  [max_ctx + 2]         int32   d(c) of Eq. 3, built exactly on the host
// Spill mode adds, per (layer, sequence): the device row of every position,
// a host-store flag, the device row of every listed position, a stack of
// free rows and the out/in copy lists; and a pinned host store
// [L][B][cap][Hkv][D] for K and V, written once per token.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include <rocprofiler-sdk-roctx/roctx.h>

#include "../../include/asrkf.h"
#include "kernels.h"

using namespace asrkf;

namespace {

thread_local std::string g_last_error;

constexpr int kCounters = 16;   // device counters of a context (see asrkf_ctx::counters)

asrkf_status fail(asrkf_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

// d(c) = floor(sqrt(c) / k) for the exact binary value of k: the largest
// integer d with (d k)^2 <= c.  k = M 2^E with M < 2^24 an integer.
int32_t exact_duration(uint64_t c, float k) {
    int e2;
    const float fr = frexpf(k, &e2);                  // k = fr * 2^e2, fr in [0.5, 1)
    const uint64_t M = (uint64_t)ldexpf(fr, 24);      // exact 24-bit mantissa
    const int E = e2 - 24;                            // k = M * 2^E
    // test (d M)^2 2^(2E) <= c  <=>  (d M)^2 <= c 2^(-2E)   (E < 0)
    //                           <=>  (d M)^2 2^(2E) <= c     (E >= 0)
    auto fits = [&](uint64_t d) -> bool {
        const unsigned __int128 lhs = (unsigned __int128)(d * M) * (d * M);
        if (E >= 0) {
            if (2 * E >= 100) return d == 0;
            return (lhs << (2 * E)) <= (unsigned __int128)c;
        }
        return lhs <= ((unsigned __int128)c << (-2 * E));
    };
    // initial guess from floating point, then fix up exactly
    double g = floor(sqrt((double)c) / (double)k);
    uint64_t d = g > 0 ? (uint64_t)g : 0;
    while (d > 0 && !fits(d)) --d;
    while (fits(d + 1)) ++d;
    return (int32_t)d;
}

bool valid_k(float k) { return isfinite(k) && k >= 0x1p-8f && k <= 0x1p16f; }

// Split-K partials of asrkf_decode_step_static: a fixed device array, so that
// the call allocates nothing.  Every GPU the library runs on holds its own
// copy until the process ends.  Host code never uses the array's name as an
// address: each device's address is looked up once (asrkf_init) and kept.
constexpr size_t kStaticScratchBytes = (size_t)32 << 20;
__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

}  // namespace

struct asrkf_ctx {
    asrkf_config cfg{};
    int cap = 0;                 // positions per (layer, seq) array
    int group = 0;
    size_t esz = 0;
    size_t row_bytes = 0;        // one token, all KV heads
    int grid = 0;                // attention grid (resident workgroups)
    int n_slots = 0;             // partial slots: grid + batch
    int dur_len = 0;

    // device memory
    void* kpool = nullptr;
    void* vpool = nullptr;
    int32_t* unfreeze = nullptr;
    int32_t* count = nullptr;
    uint8_t* flag = nullptr;
    int32_t* list = nullptr;
    int32_t* n_active = nullptr;
    int32_t* plen = nullptr;
    int32_t* dur = nullptr;
    int32_t* escalation = nullptr;
    int32_t* level = nullptr;
    float* entropy = nullptr;
    float* pmax = nullptr;
    float* part_acc = nullptr;
    float* part_ml = nullptr;
    int32_t* slot_info = nullptr;   // [2B]: first slot, end slot per sequence
    int32_t* plan = nullptr;        // [state_layers][grid][kPlanInts] first-tile records of the
                                    // attention ranges (resident mode, several layers), or null
    float* ent_partial = nullptr;   // [B][kEntropySplitMax][3]
    int32_t* ent_ticket = nullptr;  // [B]
    unsigned long long* counters = nullptr;   // [0] listed_total, [1..3] recoveries, [5] rr,
                                              // [8] rows to host, [9] rows from host, [10] released,
                                              // [11] rows taken back, [12] margin hits

    // relevance reading and state scope
    bool token_scope = false;     // one token state per sequence (state_layers = 1)
    int state_layers = 0;         // layers that own token states: n_layers, or 1
    uint64_t* hmask = nullptr;    // [state_layers][B][cap] (history window)
    int32_t* hlast = nullptr;
    float* rel_acc = nullptr;     // [B][cap] (token scope)
    float* xlog = nullptr;        // [B][cap][Hq] (relevance by attention weight)
    float* norm = nullptr;        // [B][Hq][2]
    int n_seg = 1, seg_len = 0;   // segmented list rebuild (few, long instances)
    int32_t* seg_count = nullptr; // [state instances][n_seg]

    // spill mode
    bool spill = false;
    int pool_rows = 0;            // device rows per (layer, seq)
    int32_t* row_of = nullptr;
    uint8_t* on_host = nullptr;
    int32_t* list_row = nullptr;
    int32_t* last_row = nullptr;  // [L][B][cap] row a host-only position held last
    int32_t* row_owner = nullptr; // [L][B][pool_rows] position whose K/V a row holds
    int32_t* hand = nullptr;      // [L][B] start of the next free-row search
    int32_t* pop_buf = nullptr;   // [L][B][pool_rows] free rows found by a rebuild
    int32_t* out_pos = nullptr;
    int32_t* out_row = nullptr;
    int32_t* n_out = nullptr;
    int32_t* in_pos = nullptr;
    int32_t* in_row = nullptr;
    int32_t* n_in = nullptr;
    int32_t* flags = nullptr;     // [0] out of device rows (spill), [1] past max_ctx (device check)
    int32_t* t_dev = nullptr;     // steps started, advanced by each step's first attention launch
    void* khost = nullptr;        // pinned host store (host pointers)
    void* vhost = nullptr;
    void* khost_dev = nullptr;    // the same memory as seen by kernels
    void* vhost_dev = nullptr;
    int32_t* flags_host = nullptr;      // pinned copy of flags (spill mode, read without a wait)
    hipStream_t side = nullptr;   // copies to and from the host store
    hipEvent_t ev_lists = nullptr;      // compaction done (main stream)
    hipEvent_t ev_flag = nullptr;       // flags copied to the host
    std::vector<hipEvent_t> ev_in;      // per layer: its restores are in the device cache
    bool xfer_recorded = false;
    bool flag_recorded = false;

    std::vector<int32_t> plen_host;
    std::vector<char> prefilled;   // per sequence
    int t = 0;                     // completed steps
    int next_layer = 0;            // next layer expected by decode_step
    bool lists_ready = false;
    bool poisoned = false;
    bool timing = false;
    hipStream_t last_stream = nullptr;  // stream of the last call that queued work
    bool queued = false;                // some call has queued work on last_stream
    hipEvent_t ev_switch = nullptr;     // orders a call on a new stream after last_stream
    std::vector<std::pair<hipEvent_t, hipEvent_t>> ev_used, ev_free;
    double attn_ms_done = 0.0;
    int64_t attn_launches = 0;
    std::vector<float> launch_ms;             // every timed launch, in launch order
    int side_delay_us = 0;              // test hook: side stream waits before its copies
    int device = 0;
    void* static_scratch = nullptr;     // this device's address of the static partials array
};

namespace {

asrkf_status hip_fail(asrkf_ctx* ctx, hipError_t e, const char* what) {
    if (ctx) ctx->poisoned = true;
    return fail(ASRKF_EHIP, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_OK(ctx, expr)                                              \
    do {                                                               \
        hipError_t e_ = (expr);                                        \
        if (e_ != hipSuccess) return hip_fail((ctx), e_, #expr);       \
    } while (0)

// A roctx range over one host call of the ABI, so that a marker trace
// (rocprofv3 --marker-trace) shows the step's phases next to its kernels.
struct TraceRange {
    explicit TraceRange(const char* name) { roctxRangePushA(name); }
    ~TraceRange() { roctxRangePop(); }
    TraceRange(const TraceRange&) = delete;
    TraceRange& operator=(const TraceRange&) = delete;
};

asrkf_status check_ctx(asrkf_ctx* ctx) {
    if (!ctx) return fail(ASRKF_EINVAL, "null context");
    if (ctx->poisoned) return fail(ASRKF_ESTATE, "context poisoned by an earlier HIP error");
    return ASRKF_OK;
}

template <typename T>
asrkf_status dev_alloc(asrkf_ctx* ctx, T** p, size_t bytes) {
    void* q = nullptr;
    hipError_t e = hipMalloc(&q, bytes ? bytes : 16);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(ASRKF_ENOMEM, "hipMalloc of %zu bytes failed: %s", bytes, hipGetErrorString(e));
    }
    *p = static_cast<T*>(q);
    (void)ctx;
    return ASRKF_OK;
}

void free_all(asrkf_ctx* ctx) {
    void* ptrs[] = {ctx->kpool, ctx->vpool, ctx->unfreeze, ctx->count, ctx->flag, ctx->list,
                    ctx->n_active, ctx->plen, ctx->dur, ctx->escalation, ctx->level,
                    ctx->entropy, ctx->pmax, ctx->part_acc, ctx->part_ml, ctx->slot_info, ctx->ent_partial, ctx->ent_ticket,
                    ctx->counters, ctx->row_of, ctx->on_host, ctx->list_row, ctx->last_row,
                    ctx->row_owner, ctx->hand, ctx->pop_buf, ctx->out_pos, ctx->out_row, ctx->n_out, ctx->in_pos, ctx->in_row,
                    ctx->n_in, ctx->flags, ctx->t_dev, ctx->hmask, ctx->hlast, ctx->rel_acc, ctx->xlog,
                    ctx->norm, ctx->seg_count, ctx->plan};
    for (void* p : ptrs) if (p) (void)hipFree(p);
    void* host[] = {ctx->khost, ctx->vhost, ctx->flags_host};
    for (void* p : host) if (p) (void)hipHostFree(p);
    if (ctx->side) (void)hipStreamDestroy(ctx->side);
    if (ctx->ev_lists) (void)hipEventDestroy(ctx->ev_lists);
    if (ctx->ev_flag) (void)hipEventDestroy(ctx->ev_flag);
    if (ctx->ev_switch) (void)hipEventDestroy(ctx->ev_switch);
    for (hipEvent_t e : ctx->ev_in) if (e) (void)hipEventDestroy(e);
    for (auto& ev : ctx->ev_used) { (void)hipEventDestroy(ev.first); (void)hipEventDestroy(ev.second); }
    for (auto& ev : ctx->ev_free) { (void)hipEventDestroy(ev.first); (void)hipEventDestroy(ev.second); }
}

asrkf_status validate(const asrkf_config* c) {
    if (!c) return fail(ASRKF_EINVAL, "null config");
    if (c->n_layers < 1) return fail(ASRKF_EINVAL, "n_layers must be >= 1");
    if (c->batch < 1 || c->batch > kMaxBatch) return fail(ASRKF_EINVAL, "batch must be in 1..%d", kMaxBatch);
    if (c->n_kv_heads != 1 && c->n_kv_heads != 2 && c->n_kv_heads != 4 && c->n_kv_heads != 8 &&
        c->n_kv_heads != 16 && c->n_kv_heads != 32)
        return fail(ASRKF_EINVAL, "n_kv_heads must be 1, 2, 4, 8, 16 or 32");
    if (c->n_q_heads < c->n_kv_heads || c->n_q_heads % c->n_kv_heads)
        return fail(ASRKF_EINVAL, "n_q_heads must be a multiple of n_kv_heads");
    const int g = c->n_q_heads / c->n_kv_heads;
    if (g != 1 && g != 2 && g != 4 && g != 8) return fail(ASRKF_EINVAL, "n_q_heads / n_kv_heads must be 1, 2, 4 or 8");
    if (c->head_dim != 64 && c->head_dim != 128 && c->head_dim != 256)
        return fail(ASRKF_EINVAL, "head_dim must be 64, 128 or 256");
    if (c->dtype == ASRKF_BF16 || c->dtype == ASRKF_F32) {
        if (!attention_shape_supported(c->dtype == ASRKF_BF16, c->head_dim, g, c->n_kv_heads))
            return fail(ASRKF_EINVAL, "unsupported head layout: %d q heads over %d KV heads of %d %s",
                        c->n_q_heads, c->n_kv_heads, c->head_dim,
                        c->dtype == ASRKF_BF16 ? "bf16" : "fp32");
    }
    if (c->max_ctx < 2 || c->max_ctx > (1 << 28)) return fail(ASRKF_EINVAL, "max_ctx must be in 2..2^28");
    if (c->window_K < 0) return fail(ASRKF_EINVAL, "window_K must be >= 0");
    if (isnan(c->tau)) return fail(ASRKF_EINVAL, "tau is NaN");
    if (!valid_k(c->k_soft)) return fail(ASRKF_EINVAL, "k_soft must be in [2^-8, 2^16]");
    if (c->vocab < 1) return fail(ASRKF_EINVAL, "vocab must be >= 1");
    if (isnan(c->entropy_spike) || isnan(c->conf_drop)) return fail(ASRKF_EINVAL, "NaN threshold");
    if (!(c->debug_margin >= 0.f) || isinf(c->debug_margin))
        return fail(ASRKF_EINVAL, "debug_margin must be finite and >= 0");
    if (c->dtype != ASRKF_BF16 && c->dtype != ASRKF_F32) return fail(ASRKF_EINVAL, "unknown dtype");
    if (c->spill_min_D < 0) return fail(ASRKF_EINVAL, "spill_min_D must be >= 0");
    if (c->history_W < 0 || c->history_W > 64) return fail(ASRKF_EINVAL, "history_W must be in 0..64");
    if (c->relevance != ASRKF_REL_ABS && c->relevance != ASRKF_REL_SOFTMAX)
        return fail(ASRKF_EINVAL, "unknown relevance kind");
    if (c->scope != ASRKF_SCOPE_LAYER && c->scope != ASRKF_SCOPE_TOKEN)
        return fail(ASRKF_EINVAL, "unknown state scope");
    if (c->candidates != ASRKF_CAND_OUTSIDE && c->candidates != ASRKF_CAND_INSIDE)
        return fail(ASRKF_EINVAL, "unknown freeze candidates");
    if (c->scope == ASRKF_SCOPE_TOKEN && c->spill_min_D != 0)
        return fail(ASRKF_EINVAL, "spill mode needs per-layer token states (ASRKF_SCOPE_LAYER)");
    if (c->spill_min_D == 0 && c->device_rows != 0)
        return fail(ASRKF_EINVAL, "device_rows applies to spill mode only (spill_min_D > 0)");
    if (c->device_rows != 0 && (c->device_rows < 2 || c->device_rows > c->max_ctx + 1))
        return fail(ASRKF_EINVAL, "device_rows must be 0 or in 2..max_ctx+1");
    {
        const int64_t row = (int64_t)c->n_kv_heads * c->head_dim * (c->dtype == ASRKF_BF16 ? 2 : 4);
        const int64_t cap = ((int64_t)c->max_ctx + 1 + 63) / 64 * 64;
        if (cap * row >= ((int64_t)1 << 31))
            return fail(ASRKF_EINVAL, "max_ctx too large: one sequence's cache must stay below 2 GiB per layer");
    }
    return ASRKF_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// The context's arrays (cache, token states, lists, split partials) are shared
// by every call, so a call on another stream than the previous one first waits
// for everything that call queued.
bool capturing(hipStream_t s) {
    hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
    return hipStreamIsCapturing(s, &st) == hipSuccess && st == hipStreamCaptureStatusActive;
}

hipError_t follow_last_stream(asrkf_ctx* ctx, hipStream_t s) {
    // under stream capture the caller orders the capture after earlier work
    if (!ctx->queued || s == ctx->last_stream || capturing(s)) return hipSuccess;
    hipError_t e = hipEventRecord(ctx->ev_switch, ctx->last_stream);
    if (e == hipSuccess) e = hipStreamWaitEvent(s, ctx->ev_switch, 0);
    return e;
}

void mark_queued(asrkf_ctx* ctx, hipStream_t s) {
    ctx->last_stream = s;
    ctx->queued = true;
}

}  // namespace

extern "C" {

const char* asrkf_last_error(void) { return g_last_error.c_str(); }

asrkf_status asrkf_schedule_table(float k_soft, int32_t n, int32_t* out) {
    if (!valid_k(k_soft)) return fail(ASRKF_EINVAL, "k_soft must be in [2^-8, 2^16]");
    if (n < 1 || !out) return fail(ASRKF_EINVAL, "bad table size or null output");
    for (int32_t c = 0; c < n; ++c) out[c] = exact_duration((uint64_t)c, k_soft);
    return ASRKF_OK;
}

asrkf_status asrkf_init(const asrkf_config* cfg, asrkf_ctx** out) {
    if (!out) return fail(ASRKF_EINVAL, "null output pointer");
    *out = nullptr;
    asrkf_status st = validate(cfg);
    if (st != ASRKF_OK) return st;

    asrkf_ctx* ctx = new asrkf_ctx();
    ctx->cfg = *cfg;
    if (ctx->cfg.wr_last_N <= 0) ctx->cfg.wr_last_N = 4 * ctx->cfg.window_K;
    const asrkf_config& c = ctx->cfg;
    ctx->cap = (c.max_ctx + 1 + 63) / 64 * 64;
    ctx->group = c.n_q_heads / c.n_kv_heads;
    ctx->esz = c.dtype == ASRKF_BF16 ? 2 : 4;
    ctx->row_bytes = (size_t)c.n_kv_heads * c.head_dim * ctx->esz;
    ctx->plen_host.assign(c.batch, 0);
    ctx->prefilled.assign(c.batch, 0);

    hipError_t e = hipGetDevice(&ctx->device);
    if (e != hipSuccess) { delete ctx; return hip_fail(nullptr, e, "hipGetDevice"); }
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, ctx->device);
    if (e != hipSuccess) { delete ctx; return hip_fail(nullptr, e, "hipGetDeviceProperties"); }
    if (ctx->device >= 0 && ctx->device < kMaxDevices) {
        // the static partials' address on this device (it is current here), once per device
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        if (!g_scratch[ctx->device]) {
            void* p = nullptr;
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess) { delete ctx; return hip_fail(nullptr, e, "hipGetSymbolAddress(scratch)"); }
            g_scratch[ctx->device] = p;
        }
        ctx->static_scratch = g_scratch[ctx->device];
    }
    // persistent grid: as many attention workgroups as can be resident at once
    {
        AttnArgs probe{};
        probe.B = c.batch;
        probe.Hkv = c.n_kv_heads;
        int per_cu = 0;
        e = attention_occupancy(probe, c.dtype == ASRKF_BF16, c.head_dim, ctx->group, &per_cu);
        if (e != hipSuccess) { delete ctx; return hip_fail(nullptr, e, "hipOccupancyMaxActiveBlocksPerMultiprocessor"); }
        if (per_cu < 1) {
            delete ctx;
            return fail(ASRKF_EINVAL, "attention workgroup does not fit on a CU for this shape");
        }
        ctx->grid = per_cu * prop.multiProcessorCount;
    }
    ctx->n_slots = ctx->grid + c.batch;
    ctx->dur_len = c.max_ctx + 2;
    ctx->spill = c.spill_min_D > 0;
    ctx->pool_rows = ctx->spill && c.device_rows > 0 ? c.device_rows : ctx->cap;

    ctx->token_scope = c.scope == ASRKF_SCOPE_TOKEN;
    ctx->state_layers = ctx->token_scope ? 1 : c.n_layers;
    const size_t inst = (size_t)c.n_layers * c.batch;          // (layer, sequence) caches
    const size_t per_pos = inst * ctx->cap;
    const size_t st_inst = (size_t)ctx->state_layers * c.batch; // token-state instances
    const size_t st_pos = st_inst * ctx->cap;
#define ALLOC(field, bytes)                                       \
    do {                                                          \
        st = dev_alloc(ctx, &ctx->field, (bytes));                \
        if (st != ASRKF_OK) { free_all(ctx); delete ctx; return st; } \
    } while (0)
    const size_t pool_bytes = inst * ctx->pool_rows * ctx->row_bytes;
    ALLOC(kpool, pool_bytes);
    ALLOC(vpool, pool_bytes);
    ALLOC(unfreeze, st_pos * 4);
    ALLOC(count, st_pos * 4);
    ALLOC(flag, st_pos);
    ALLOC(list, st_pos * 4);
    if (c.history_W > 0) {
        ALLOC(hmask, st_pos * 8);
        ALLOC(hlast, st_pos * 4);
    }
    if (ctx->token_scope) ALLOC(rel_acc, (size_t)c.batch * ctx->cap * 4);
    ctx->n_seg = compact_segments((int)st_inst, ctx->cap, &ctx->seg_len);
    if (ctx->n_seg > 1) ALLOC(seg_count, st_inst * (ctx->n_seg + 1) * 32);   // spill mode: 8 counts per segment
    if (c.relevance == ASRKF_REL_SOFTMAX) {
        ALLOC(xlog, (size_t)c.batch * ctx->cap * c.n_q_heads * 4);
        ALLOC(norm, (size_t)c.batch * c.n_q_heads * 2 * 4);
    }
    ALLOC(n_active, inst * 4);
    ALLOC(plen, (size_t)c.batch * 4);
    ALLOC(dur, (size_t)ctx->dur_len * 4);
    ALLOC(escalation, (size_t)c.batch * 4);
    ALLOC(level, (size_t)c.batch * 4);
    ALLOC(entropy, (size_t)c.batch * 4);
    ALLOC(pmax, (size_t)c.batch * 4);
    ALLOC(part_acc, (size_t)ctx->n_slots * c.n_q_heads * c.head_dim * 4);
    ALLOC(part_ml, (size_t)ctx->n_slots * c.n_q_heads * 2 * 4);
    ALLOC(slot_info, (size_t)c.batch * 2 * 4);
    // The first-tile records cost a launch per step and save about a memory round
    // trip per attention launch: worth it from a few layers on.
    if (!ctx->spill && c.n_layers >= kPlanMinLayers)
        ALLOC(plan, (size_t)ctx->state_layers * ctx->grid * kPlanInts * 4);
    ALLOC(ent_partial, (size_t)c.batch * kEntropySplitMax * 3 * 4);
    ALLOC(ent_ticket, (size_t)c.batch * 4);
    ALLOC(counters, kCounters * sizeof(unsigned long long));
    ALLOC(flags, 8);
    ALLOC(t_dev, 4);
    if (ctx->spill) {
        ALLOC(row_of, per_pos * 4);
        ALLOC(on_host, per_pos);
        ALLOC(list_row, per_pos * 4);
        ALLOC(last_row, per_pos * 4);
        ALLOC(row_owner, inst * ctx->pool_rows * 4);
        ALLOC(hand, inst * 4);
        ALLOC(pop_buf, inst * ctx->pool_rows * 4);
        ALLOC(out_pos, per_pos * 4);
        ALLOC(out_row, per_pos * 4);
        ALLOC(n_out, inst * 4);
        ALLOC(in_pos, per_pos * 4);
        ALLOC(in_row, per_pos * 4);
        ALLOC(n_in, inst * 4);
        // host store: pinned, mapped, coarse-grained (only the GPU reads and writes it)
        const size_t store = per_pos * ctx->row_bytes;
        const unsigned flags = hipHostMallocMapped | hipHostMallocNonCoherent;
        hipError_t he = hipHostMalloc(&ctx->khost, store, flags);
        if (he == hipSuccess) he = hipHostMalloc(&ctx->vhost, store, flags);
        if (he == hipSuccess) he = hipHostMalloc((void**)&ctx->flags_host, 64, hipHostMallocDefault);
        if (he != hipSuccess) {
            (void)hipGetLastError();
            free_all(ctx);
            delete ctx;
            return fail(ASRKF_ENOMEM, "pinned host store of 2 x %zu bytes: %s", store, hipGetErrorString(he));
        }
        ctx->flags_host[0] = ctx->flags_host[1] = 0;
        he = hipHostGetDevicePointer(&ctx->khost_dev, ctx->khost, 0);
        if (he == hipSuccess) he = hipHostGetDevicePointer(&ctx->vhost_dev, ctx->vhost, 0);
        if (he == hipSuccess) he = hipStreamCreateWithFlags(&ctx->side, hipStreamNonBlocking);
        if (he == hipSuccess) he = hipEventCreateWithFlags(&ctx->ev_lists, hipEventDisableTiming);
        if (he == hipSuccess) he = hipEventCreateWithFlags(&ctx->ev_flag, hipEventDisableTiming);
        ctx->ev_in.assign(c.n_layers, nullptr);
        for (int l = 0; l < c.n_layers && he == hipSuccess; ++l)
            he = hipEventCreateWithFlags(&ctx->ev_in[l], hipEventDisableTiming);
        if (he != hipSuccess) {
            st = hip_fail(nullptr, he, "spill-mode stream, events or mapping");
            free_all(ctx);
            delete ctx;
            return st;
        }
    }
#undef ALLOC

    {
        const hipError_t he = hipEventCreateWithFlags(&ctx->ev_switch, hipEventDisableTiming);
        if (he != hipSuccess) {
            st = hip_fail(nullptr, he, "hipEventCreateWithFlags");
            free_all(ctx);
            delete ctx;
            return st;
        }
    }

    std::vector<int32_t> table(ctx->dur_len);
    for (int i = 0; i < ctx->dur_len; ++i) table[i] = exact_duration((uint64_t)i, c.k_soft);
#define INIT(expr)                                                              \
    do {                                                                        \
        hipError_t e_ = (expr);                                                 \
        if (e_ != hipSuccess) { st = hip_fail(nullptr, e_, #expr); free_all(ctx); delete ctx; return st; } \
    } while (0)
    INIT(hipMemset(ctx->unfreeze, 0, st_pos * 4));
    INIT(hipMemset(ctx->count, 0, st_pos * 4));
    INIT(hipMemset(ctx->n_active, 0, st_inst * 4));
    if (ctx->hmask) INIT(hipMemset(ctx->hmask, 0, st_pos * 8));
    if (ctx->hlast) INIT(hipMemset(ctx->hlast, 0, st_pos * 4));
    INIT(hipMemset(ctx->plen, 0, (size_t)c.batch * 4));
    INIT(hipMemset(ctx->escalation, 0, (size_t)c.batch * 4));
    INIT(hipMemset(ctx->level, 0, (size_t)c.batch * 4));
    INIT(hipMemset(ctx->entropy, 0, (size_t)c.batch * 4));
    INIT(hipMemset(ctx->pmax, 0, (size_t)c.batch * 4));
    INIT(hipMemset(ctx->ent_ticket, 0, (size_t)c.batch * 4));
    INIT(hipMemset(ctx->counters, 0, kCounters * sizeof(unsigned long long)));
    INIT(hipMemset(ctx->flags, 0, 8));
    INIT(hipMemset(ctx->t_dev, 0, 4));
    INIT(hipMemcpy(ctx->dur, table.data(), table.size() * 4, hipMemcpyHostToDevice));
    INIT(hipDeviceSynchronize());
#undef INIT
    *out = ctx;
    return ASRKF_OK;
}

asrkf_status asrkf_prefill(asrkf_ctx* ctx, int32_t layer, int32_t seq, const void* k,
                           const void* v, int32_t n_tokens, void* stream) {
    asrkf_status st = check_ctx(ctx);
    if (st != ASRKF_OK) return st;
    const asrkf_config& c = ctx->cfg;
    if (ctx->t > 0 || ctx->next_layer != 0 || ctx->lists_ready)
        return fail(ASRKF_ESTATE, "prefill after the first decode step");
    if (layer < 0 || layer >= c.n_layers || seq < 0 || seq >= c.batch)
        return fail(ASRKF_EINVAL, "layer or sequence out of range");
    if (n_tokens < 1 || n_tokens > c.max_ctx - 1)
        return fail(ASRKF_EINVAL, "n_tokens must be in 1..max_ctx-1");
    if (n_tokens > ctx->pool_rows - 1)
        return fail(ASRKF_EINVAL, "n_tokens must leave one device row free (device_rows = %d)",
                    ctx->pool_rows);
    if (!k || !v) return fail(ASRKF_EINVAL, "null k or v");
    if (ctx->prefilled[seq] && ctx->plen_host[seq] != n_tokens)
        return fail(ASRKF_EINVAL, "sequence %d was prefilled with %d tokens in another layer",
                    seq, ctx->plen_host[seq]);
    hipStream_t s = static_cast<hipStream_t>(stream);
    HIP_OK(ctx, follow_last_stream(ctx, s));
    const size_t off = ((size_t)layer * c.batch + seq) * ctx->pool_rows * ctx->row_bytes;
    const size_t bytes = (size_t)n_tokens * ctx->row_bytes;
    HIP_OK(ctx, hipMemcpyAsync((char*)ctx->kpool + off, k, bytes, hipMemcpyDeviceToDevice, s));
    HIP_OK(ctx, hipMemcpyAsync((char*)ctx->vpool + off, v, bytes, hipMemcpyDeviceToDevice, s));
    if (!ctx->prefilled[seq]) {
        ctx->prefilled[seq] = 1;
        ctx->plen_host[seq] = n_tokens;
        HIP_OK(ctx, hipMemcpyAsync(ctx->plen + seq, &ctx->plen_host[seq], 4,
                                   hipMemcpyHostToDevice, s));
    }
    mark_queued(ctx, s);
    return ASRKF_OK;
}

}  // extern "C"

namespace {

asrkf_status build_lists(asrkf_ctx* ctx, int forced_level, hipStream_t s) {
    const int n_inst = ctx->state_layers * ctx->cfg.batch;
    if (ctx->spill && ctx->t == 0) {
        SpillInitArgs z{};
        z.row_of = ctx->row_of;
        z.on_host = ctx->on_host;
        z.last_row = ctx->last_row;
        z.row_owner = ctx->row_owner;
        z.hand = ctx->hand;
        z.plen = ctx->plen;
        z.B = ctx->cfg.batch;
        z.cap = ctx->cap;
        z.pool_rows = ctx->pool_rows;
        HIP_OK(ctx, launch_spill_init(z, n_inst, s));
    }
    CompactArgs a{};
    a.unfreeze = ctx->unfreeze;
    a.list = ctx->list;
    a.n_active = ctx->n_active;
    a.plen = ctx->plen;
    a.level = ctx->level;
    a.listed_total = ctx->counters;
    a.forced_level = forced_level;
    a.count_forced = forced_level > 0 ? 1 : 0;       // no logits: the entropy kernel counts none
    a.recoveries = ctx->counters;
    a.t_dev = ctx->t_dev;
    a.max_ctx = ctx->cfg.max_ctx;
    a.flags = ctx->flags;
    a.B = ctx->cfg.batch;
    a.cap = ctx->cap;
    a.wr_last_N = ctx->cfg.wr_last_N;
    a.n_seg = ctx->n_seg;
    a.seg_len = ctx->seg_len;
    a.seg_count = ctx->seg_count;
    // the freeze loop of the step that ends here (the kernels skip it before step 1)
    a.flag = ctx->flag;
    a.scope_token = ctx->token_scope ? 1 : 0;
    a.rel_acc = ctx->rel_acc;
    a.tau_LH = ctx->cfg.tau * (float)ctx->cfg.n_layers * (float)ctx->cfg.n_q_heads;
    a.margin_LH = ctx->cfg.debug_margin * (float)ctx->cfg.n_layers * (float)ctx->cfg.n_q_heads;
    a.margin_hits = ctx->cfg.debug_margin > 0.f ? ctx->counters + 12 : nullptr;
    a.count = ctx->count;
    a.hmask = ctx->hmask;
    a.hlast = ctx->hlast;
    a.dur = ctx->dur;
    a.dur_len = ctx->dur_len;
    a.history_W = ctx->cfg.history_W;
    a.window_K = ctx->cfg.window_K;
    a.cand_inside = ctx->cfg.candidates == ASRKF_CAND_INSIDE;
    if (ctx->spill) {
        a.spill_min_D = ctx->cfg.spill_min_D;
        a.pool_rows = ctx->pool_rows;
        a.row_of = ctx->row_of;
        a.on_host = ctx->on_host;
        a.list_row = ctx->list_row;
        a.last_row = ctx->last_row;
        a.row_owner = ctx->row_owner;
        a.hand = ctx->hand;
        a.pop_buf = ctx->pop_buf;
        a.out_pos = ctx->out_pos;
        a.out_row = ctx->out_row;
        a.n_out = ctx->n_out;
        a.in_pos = ctx->in_pos;
        a.in_row = ctx->in_row;
        a.n_in = ctx->n_in;
        a.xfer = ctx->counters + 8;
    }
    HIP_OK(ctx, launch_compact(a, n_inst, s));
    if (!ctx->spill) {
        if (ctx->plan) {
            PlanArgs p{};
            p.list = ctx->list;
            p.n_active = ctx->n_active;
            p.plan = ctx->plan;
            p.B = ctx->cfg.batch;
            p.cap = ctx->cap;
            p.grid = ctx->grid;
            HIP_OK(ctx, launch_plan(p, ctx->state_layers, s));
        }
        return ASRKF_OK;
    }

    // the flag tells the host (one step late, without a wait) that rows ran out
    HIP_OK(ctx, hipMemcpyAsync(ctx->flags_host, ctx->flags, 8, hipMemcpyDeviceToHost, s));
    HIP_OK(ctx, hipEventRecord(ctx->ev_flag, s));
    ctx->flag_recorded = true;

    // copies on the side stream: every out-list first (its rows may be handed
    // out again below), then each layer's in-list, which that layer's next
    // attention launch waits for
    HIP_OK(ctx, hipEventRecord(ctx->ev_lists, s));
    HIP_OK(ctx, hipStreamWaitEvent(ctx->side, ctx->ev_lists, 0));
    if (ctx->side_delay_us > 0) HIP_OK(ctx, launch_delay(ctx->side_delay_us, ctx->side));
    XferArgs x{};
    x.kpool = static_cast<char*>(ctx->kpool);
    x.vpool = static_cast<char*>(ctx->vpool);
    x.khost = static_cast<char*>(ctx->khost_dev);
    x.vhost = static_cast<char*>(ctx->vhost_dev);
    x.cap = ctx->cap;
    x.pool_rows = ctx->pool_rows;
    x.row_bytes = (int32_t)ctx->row_bytes;
    x.pos = ctx->out_pos;
    x.row = ctx->out_row;
    x.count = ctx->n_out;
    x.inst0 = 0;
    x.to_host = 1;
    HIP_OK(ctx, launch_xfer(x, n_inst, ctx->side));
    x.pos = ctx->in_pos;
    x.row = ctx->in_row;
    x.count = ctx->n_in;
    x.to_host = 0;
    for (int l = 0; l < ctx->cfg.n_layers; ++l) {
        x.inst0 = l * ctx->cfg.batch;
        HIP_OK(ctx, launch_xfer(x, ctx->cfg.batch, ctx->side));
        HIP_OK(ctx, hipEventRecord(ctx->ev_in[l], ctx->side));
    }
    ctx->xfer_recorded = true;
    return ASRKF_OK;
}

// The device flags of earlier rebuilds: a sequence ran out of device rows
// (spill mode), or a step would have passed max_ctx positions (a step replayed
// from a graph, which the host checks do not see).  Without waiting, only spill
// mode's flag copy is read, if it has arrived; the synchronizing calls read the
// flags themselves after their wait.
asrkf_status check_overflow(asrkf_ctx* ctx, bool synced) {
    int32_t f[2] = {0, 0};
    if (synced) {
        HIP_OK(ctx, hipMemcpy(f, ctx->flags, 8, hipMemcpyDeviceToHost));
    } else {
        if (!ctx->spill || !ctx->flag_recorded) return ASRKF_OK;
        const hipError_t q = hipEventQuery(ctx->ev_flag);
        if (q == hipErrorNotReady) return ASRKF_OK;
        if (q != hipSuccess) return hip_fail(ctx, q, "hipEventQuery");
        f[0] = ((volatile int32_t*)ctx->flags_host)[0];
        f[1] = ((volatile int32_t*)ctx->flags_host)[1];
    }
    if (f[0]) {
        ctx->poisoned = true;
        return fail(ASRKF_ECAPACITY, "a sequence needed more than device_rows = %d device rows; "
                    "results since then are void", ctx->pool_rows);
    }
    if (f[1]) {
        ctx->poisoned = true;
        return fail(ASRKF_ECAPACITY, "a replayed step would pass max_ctx = %d positions; the "
                    "active caches were not rebuilt since then", ctx->cfg.max_ctx);
    }
    return ASRKF_OK;
}

}  // namespace

namespace {

// Bytes of the split partials (acc, (m, l), slot range per sequence).
size_t partial_bytes(const asrkf_ctx* ctx) {
    const asrkf_config& c = ctx->cfg;
    return (size_t)ctx->n_slots * c.n_q_heads * (c.head_dim + 2) * 4 + (size_t)c.batch * 2 * 4;
}

// decode_step with its split partials in the context's scratch, or (use_static)
// in the static array, with no event of its own.
asrkf_status decode_step_impl(asrkf_ctx* ctx, int32_t layer, const void* q, const void* k_new,
                              const void* v_new, float* out, void* stream, bool use_static) {
    asrkf_status st = check_ctx(ctx);
    if (st != ASRKF_OK) return st;
    const asrkf_config& c = ctx->cfg;
    if (use_static) {
        if (!ctx->static_scratch)
            return fail(ASRKF_EINVAL, "no static scratch on device %d (devices 0..%d only)",
                        ctx->device, kMaxDevices - 1);
        if (partial_bytes(ctx) > kStaticScratchBytes)
            return fail(ASRKF_EINVAL, "split partials of %zu bytes exceed the static scratch of %zu "
                        "bytes; use asrkf_decode_step", partial_bytes(ctx), kStaticScratchBytes);
    }
    if (layer != ctx->next_layer)
        return fail(ASRKF_ESTATE, "decode_step expected layer %d, got %d", ctx->next_layer, layer);
    if (!q || !k_new || !v_new || !out) return fail(ASRKF_EINVAL, "null argument");
    if (!aligned16(q) || !aligned16(k_new) || !aligned16(v_new) || !aligned16(out))
        return fail(ASRKF_EINVAL, "q, k_new, v_new and out must be 16-byte aligned");
    const int t = ctx->t + 1;
    for (int b = 0; b < c.batch; ++b)
        if (ctx->plen_host[b] + t > c.max_ctx)
            return fail(ASRKF_ECAPACITY, "sequence %d would exceed max_ctx=%d", b, c.max_ctx);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool capture = capturing(s);
    if (capture && (ctx->spill || !ctx->lists_ready))
        return fail(ASRKF_ESTATE, ctx->spill ? "spill-mode steps cannot be captured in a graph"
                                             : "capture a step only after the first decode step");
    st = check_overflow(ctx, false);
    if (st != ASRKF_OK) return st;
    HIP_OK(ctx, follow_last_stream(ctx, s));
    mark_queued(ctx, s);
    if (!ctx->lists_ready) {
        if (ctx->spill)
            for (int b = 0; b < c.batch; ++b)
                if (ctx->plen_host[b] + 1 > ctx->pool_rows)
                    return fail(ASRKF_ECAPACITY, "sequence %d: prompt leaves no free device row", b);
        st = build_lists(ctx, 0, s);          // step 1 attends every prompt position
        if (st != ASRKF_OK) return st;
        ctx->lists_ready = true;
    }
    if (ctx->spill && ctx->xfer_recorded)    // this layer's restored rows are in place
        HIP_OK(ctx, hipStreamWaitEvent(s, ctx->ev_in[layer], 0));

    const size_t inst0 = (size_t)layer * c.batch;              // this layer's caches
    const size_t st0 = ctx->token_scope ? 0 : inst0;           // its token states
    AttnArgs a{};
    const size_t pool_off = inst0 * ctx->pool_rows * ctx->row_bytes;
    a.kpool = (const char*)ctx->kpool + pool_off;
    a.vpool = (const char*)ctx->vpool + pool_off;
    a.kpool_w = (char*)ctx->kpool + pool_off;
    a.vpool_w = (char*)ctx->vpool + pool_off;
    a.q = q;
    a.knew = k_new;
    a.vnew = v_new;
    a.list = ctx->list + st0 * ctx->cap;
    a.list_row = ctx->spill ? ctx->list_row + inst0 * ctx->cap : a.list;
    a.pool_rows = ctx->pool_rows;
    a.spill = ctx->spill ? 1 : 0;
    a.n_active = ctx->n_active + st0;
    a.flag = ctx->flag + st0 * ctx->cap;
    a.t_dev = layer == 0 ? ctx->t_dev : nullptr;
    a.rel_mode = c.relevance;
    a.scope_token = ctx->token_scope ? 1 : 0;
    a.first_layer = layer == 0 ? 1 : 0;
    a.rel_acc = ctx->rel_acc;
    a.xlog = ctx->xlog;
    a.part_acc = ctx->part_acc;
    a.part_ml = ctx->part_ml;
    a.slot_first = ctx->slot_info;
    a.slot_end = ctx->slot_info + c.batch;
    a.plan = ctx->plan ? ctx->plan + (ctx->token_scope ? 0 : (size_t)layer) * ctx->grid * kPlanInts : nullptr;
    if (use_static) {
        float* base = static_cast<float*>(ctx->static_scratch);
        a.part_acc = base;
        a.part_ml = base + (size_t)ctx->n_slots * c.n_q_heads * c.head_dim;
        a.slot_first = reinterpret_cast<int32_t*>(a.part_ml + (size_t)ctx->n_slots * c.n_q_heads * 2);
        a.slot_end = a.slot_first + c.batch;
    }
    a.B = c.batch;
    a.cap = ctx->cap;
    a.Hq = c.n_q_heads;
    a.Hkv = c.n_kv_heads;
    a.tau_H = c.tau * (float)c.n_q_heads;
    a.margin_H = c.debug_margin * (float)c.n_q_heads;
    a.scale_log2 = (float)(1.4426950408889634 / sqrt((double)c.head_dim));

    std::pair<hipEvent_t, hipEvent_t> ev{nullptr, nullptr};
    if (ctx->timing && !use_static && !capture) {
        if (!ctx->ev_free.empty()) {
            ev = ctx->ev_free.back();
            ctx->ev_free.pop_back();
        } else {
            // timing only: no system-scope fence (no cache write-back or invalidate)
            // when the events complete, so they do not perturb the work they measure
            HIP_OK(ctx, hipEventCreateWithFlags(&ev.first, hipEventDisableSystemFence));
            HIP_OK(ctx, hipEventCreateWithFlags(&ev.second, hipEventDisableSystemFence));
        }
    }
    HIP_OK(ctx, launch_attention(a, c.dtype == ASRKF_BF16, c.head_dim, ctx->group, ctx->grid, s,
                                 ev.first, ev.second));
    if (ev.first) ctx->ev_used.push_back(ev);

    FinishArgs f{};
    f.part_acc = a.part_acc;
    f.part_ml = a.part_ml;
    f.slot_first = a.slot_first;
    f.slot_end = a.slot_end;
    f.out = out;
    f.norm = ctx->norm;
    f.B = c.batch;
    f.Hq = c.n_q_heads;
    HIP_OK(ctx, launch_finish(f, c.head_dim, ctx->grid / c.batch + 1, s));
    if (c.relevance == ASRKF_REL_SOFTMAX) {
        RelevanceArgs r{};
        r.xlog = ctx->xlog;
        r.norm = ctx->norm;
        r.list = a.list;
        r.n_active = a.n_active;
        r.flag = a.flag;
        r.rel_acc = ctx->rel_acc;
        r.B = c.batch;
        r.cap = ctx->cap;
        r.Hq = c.n_q_heads;
        r.scope_token = a.scope_token;
        r.first_layer = a.first_layer;
        r.tau_H = a.tau_H;
        r.margin_H = a.margin_H;
        HIP_OK(ctx, launch_weight_relevance(r, s));
    }

    ctx->next_layer = layer + 1;
    return ASRKF_OK;
}

}  // namespace

extern "C" {

asrkf_status asrkf_decode_step(asrkf_ctx* ctx, int32_t layer, const void* q, const void* k_new,
                               const void* v_new, float* out, void* stream) {
    TraceRange range("asrkf_decode_step");
    return decode_step_impl(ctx, layer, q, k_new, v_new, out, stream, false);
}

asrkf_status asrkf_decode_step_static(asrkf_ctx* ctx, int32_t layer, const void* q,
                                      const void* k_new, const void* v_new, float* out,
                                      void* stream) {
    TraceRange range("asrkf_decode_step_static");
    return decode_step_impl(ctx, layer, q, k_new, v_new, out, stream, true);
}

asrkf_status asrkf_restore(asrkf_ctx* ctx, const float* logits, int32_t mode, void* stream) {
    TraceRange range("asrkf_restore");
    asrkf_status st = check_ctx(ctx);
    if (st != ASRKF_OK) return st;
    const asrkf_config& c = ctx->cfg;
    if ((int)mode < ASRKF_AUTO || (int)mode > ASRKF_NONE) return fail(ASRKF_EINVAL, "unknown recovery mode");
    if (ctx->next_layer != c.n_layers)
        return fail(ASRKF_ESTATE, "restore before decode_step of every layer (next layer %d of %d)",
                    ctx->next_layer, c.n_layers);
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (ctx->spill && capturing(s)) return fail(ASRKF_ESTATE, "spill-mode steps cannot be captured in a graph");
    st = check_overflow(ctx, false);
    if (st != ASRKF_OK) return st;
    HIP_OK(ctx, follow_last_stream(ctx, s));
    mark_queued(ctx, s);
    int forced;
    if (logits) {
        EntropyArgs e{};
        e.logits = logits;
        e.partial = ctx->ent_partial;
        e.split = entropy_split(c.batch);
        e.ticket = ctx->ent_ticket;
        e.V = c.vocab;
        e.B = c.batch;
        e.theta_H = c.entropy_spike;
        e.theta_p = c.conf_drop;
        e.mode = (int)mode;
        e.escalation = ctx->escalation;
        e.level = ctx->level;
        e.entropy = ctx->entropy;
        e.pmax = ctx->pmax;
        e.recoveries = ctx->counters;       // [level] for level 1..3
        e.rr_requests = ctx->counters + 5;
        HIP_OK(ctx, launch_entropy(e, s));
        forced = -1;                           // level[] written by the entropy kernel
    } else {
        forced = (mode >= ASRKF_SR && mode <= ASRKF_FR) ? (int)mode : 0;
    }
    // a captured step runs only when replayed: the host learns of it from the
    // device step counter at its next wait
    if (!capturing(s)) ctx->t += 1;
    ctx->next_layer = 0;
    return build_lists(ctx, forced, s);
}

}  // extern "C"

namespace {

// Everything the context queued: its calls are ordered on last_stream (a call
// on a new stream waits for the previous one), except the spill-mode copies
// on the side stream, which the next decode_step waits for.
// Steps replayed from a captured graph advance only the device's step
// counter: after the wait the host adopts it (the counter counts steps
// started, so a step in progress is not yet complete).
asrkf_status sync_ctx(asrkf_ctx* ctx) {
    HIP_OK(ctx, hipStreamSynchronize(ctx->last_stream));
    if (ctx->side) HIP_OK(ctx, hipStreamSynchronize(ctx->side));
    int32_t started = 0;
    HIP_OK(ctx, hipMemcpy(&started, ctx->t_dev, 4, hipMemcpyDeviceToHost));
    const int completed = started - (ctx->next_layer != 0 ? 1 : 0);
    if (completed > ctx->t) ctx->t = completed;
    return ASRKF_OK;
}

asrkf_status collect_timing(asrkf_ctx* ctx) {
    for (auto& ev : ctx->ev_used) {
        float ms = 0.f;
        HIP_OK(ctx, hipEventElapsedTime(&ms, ev.first, ev.second));
        ctx->attn_ms_done += ms;
        ctx->attn_launches += 1;
        ctx->launch_ms.push_back(ms);
        ctx->ev_free.push_back(ev);
    }
    ctx->ev_used.clear();
    return ASRKF_OK;
}

}  // namespace

extern "C" {

asrkf_status asrkf_stats(asrkf_ctx* ctx, asrkf_stats_t* out) {
    asrkf_status st = check_ctx(ctx);
    if (st != ASRKF_OK) return st;
    if (!out) return fail(ASRKF_EINVAL, "null output");
    st = sync_ctx(ctx);
    if (st != ASRKF_OK) return st;
    st = collect_timing(ctx);
    if (st != ASRKF_OK) return st;
    st = check_overflow(ctx, true);
    if (st != ASRKF_OK) return st;
    const asrkf_config& c = ctx->cfg;
    const size_t inst = (size_t)ctx->state_layers * c.batch;
    // with token scope one list serves every layer: count it once per layer
    const int64_t per_list = ctx->token_scope ? c.n_layers : 1;
    unsigned long long cnt[kCounters];
    std::vector<int32_t> na(inst);
    HIP_OK(ctx, hipMemcpy(cnt, ctx->counters, sizeof cnt, hipMemcpyDeviceToHost));
    HIP_OK(ctx, hipMemcpy(na.data(), ctx->n_active, inst * 4, hipMemcpyDeviceToHost));
    memset(out, 0, sizeof *out);
    out->step = ctx->t;
    int64_t total = 0, active = 0, current = 0;
    for (int b = 0; b < c.batch; ++b) total += (int64_t)(ctx->plen_host[b] + ctx->t) * c.n_layers;
    if (ctx->lists_ready) {
        for (size_t i = 0; i < inst; ++i) { current += na[i]; active += na[i] - 1; }
        current *= per_list;
        active *= per_list;
    } else {
        active = total;
    }
    out->total_positions = total;
    out->active_positions = active;
    out->attended_total = ctx->lists_ready ? (int64_t)cnt[0] * per_list - current : 0;
    for (int i = 1; i < 4; ++i) out->recoveries[i] = (int64_t)cnt[i];
    out->rr_requests = (int64_t)cnt[5];
    out->attn_launches = ctx->attn_launches;
    out->attn_kernel_ms = ctx->attn_ms_done;
    out->compression = total > 0 ? 1.0 - (double)active / (double)total : 0.0;
    out->rows_to_host = (int64_t)cnt[8];
    out->rows_from_host = (int64_t)cnt[9];
    out->rows_released = (int64_t)cnt[10];
    out->rows_reused = (int64_t)cnt[11];
    out->margin_hits = (int64_t)cnt[12];
    return ASRKF_OK;
}

asrkf_status asrkf_stats_reset(asrkf_ctx* ctx) {
    asrkf_status st = check_ctx(ctx);
    if (st != ASRKF_OK) return st;
    st = sync_ctx(ctx);
    if (st != ASRKF_OK) return st;
    st = collect_timing(ctx);
    if (st != ASRKF_OK) return st;
    const asrkf_config& c = ctx->cfg;
    const size_t inst = (size_t)ctx->state_layers * c.batch;
    std::vector<int32_t> na(inst);
    HIP_OK(ctx, hipMemcpy(na.data(), ctx->n_active, inst * 4, hipMemcpyDeviceToHost));
    // keep the lists of the coming step counted, drop everything before it
    unsigned long long cnt[kCounters] = {};
    if (ctx->lists_ready)
        for (size_t i = 0; i < inst; ++i) cnt[0] += (unsigned long long)na[i];
    HIP_OK(ctx, hipMemcpy(ctx->counters, cnt, sizeof cnt, hipMemcpyHostToDevice));
    ctx->attn_ms_done = 0.0;
    ctx->attn_launches = 0;
    ctx->launch_ms.clear();
    return ASRKF_OK;
}

asrkf_status asrkf_debug_delay_side(asrkf_ctx* ctx, int32_t microseconds) {
    asrkf_status st = check_ctx(ctx);
    if (st != ASRKF_OK) return st;
    if (microseconds < 0 || microseconds > 1000000)
        return fail(ASRKF_EINVAL, "side-stream delay must be in [0, 1e6] us, got %d", microseconds);
    ctx->side_delay_us = microseconds;
    return ASRKF_OK;
}

asrkf_status asrkf_set_timing(asrkf_ctx* ctx, int32_t enable) {
    asrkf_status st = check_ctx(ctx);
    if (st != ASRKF_OK) return st;
    ctx->timing = enable != 0;
    return ASRKF_OK;
}

asrkf_status asrkf_timing_series(asrkf_ctx* ctx, float* ms, int64_t cap, int64_t* count) {
    asrkf_status st = check_ctx(ctx);
    if (st != ASRKF_OK) return st;
    if (!count || cap < 0 || (cap > 0 && !ms)) return fail(ASRKF_EINVAL, "bad timing series buffer");
    st = sync_ctx(ctx);
    if (st != ASRKF_OK) return st;
    st = collect_timing(ctx);
    if (st != ASRKF_OK) return st;
    const int64_t n = (int64_t)ctx->launch_ms.size();
    for (int64_t i = 0; i < n && i < cap; ++i) ms[i] = ctx->launch_ms[i];
    *count = n;
    return ASRKF_OK;
}

asrkf_status asrkf_get_state(asrkf_ctx* ctx, int32_t layer, int32_t seq, int32_t* n_positions,
                             int32_t* unfreeze_step, int32_t* count, uint8_t* frozen,
                             int32_t* active, int32_t* n_active) {
    asrkf_status st = check_ctx(ctx);
    if (st != ASRKF_OK) return st;
    const asrkf_config& c = ctx->cfg;
    if (layer < 0 || layer >= c.n_layers || seq < 0 || seq >= c.batch)
        return fail(ASRKF_EINVAL, "layer or sequence out of range");
    st = sync_ctx(ctx);
    if (st != ASRKF_OK) return st;
    st = check_overflow(ctx, true);
    if (st != ASRKF_OK) return st;
    const int n = ctx->plen_host[seq] + ctx->t;
    const size_t sidx = (size_t)(ctx->token_scope ? 0 : layer) * c.batch + seq;
    const size_t off = sidx * ctx->cap;
    std::vector<int32_t> U(n > 0 ? n : 1);
    if (n > 0) HIP_OK(ctx, hipMemcpy(U.data(), ctx->unfreeze + off, (size_t)n * 4, hipMemcpyDeviceToHost));
    if (n_positions) *n_positions = n;
    if (unfreeze_step && n > 0) memcpy(unfreeze_step, U.data(), (size_t)n * 4);
    if (count && n > 0) HIP_OK(ctx, hipMemcpy(count, ctx->count + off, (size_t)n * 4, hipMemcpyDeviceToHost));
    if (frozen)
        for (int p = 0; p < n; ++p) frozen[p] = U[p] > ctx->t + 1 ? 1 : 0;
    if (active || n_active) {
        int32_t na = 0;
        if (ctx->lists_ready) {
            HIP_OK(ctx, hipMemcpy(&na, ctx->n_active + sidx, 4,
                                  hipMemcpyDeviceToHost));
            if (active && na > 0)
                HIP_OK(ctx, hipMemcpy(active, ctx->list + off, (size_t)na * 4, hipMemcpyDeviceToHost));
        } else {
            // before the first step every prompt position attends, then the new token
            na = n + 1;
            if (active) for (int p = 0; p <= n; ++p) active[p] = p;
        }
        if (n_active) *n_active = na;
    }
    return ASRKF_OK;
}

asrkf_status asrkf_get_residency(asrkf_ctx* ctx, int32_t layer, int32_t seq, int32_t* n_positions,
                                 int32_t* device_row, uint8_t* on_host) {
    asrkf_status st = check_ctx(ctx);
    if (st != ASRKF_OK) return st;
    const asrkf_config& c = ctx->cfg;
    if (layer < 0 || layer >= c.n_layers || seq < 0 || seq >= c.batch)
        return fail(ASRKF_EINVAL, "layer or sequence out of range");
    st = sync_ctx(ctx);
    if (st != ASRKF_OK) return st;
    st = check_overflow(ctx, true);
    if (st != ASRKF_OK) return st;
    const int n = ctx->plen_host[seq] + ctx->t;
    if (n_positions) *n_positions = n;
    if (n <= 0) return ASRKF_OK;
    const size_t off = ((size_t)layer * c.batch + seq) * ctx->cap;
    if (!ctx->spill || !ctx->lists_ready) {
        // resident mode, or before the first step: every position in its own row
        if (device_row) for (int p = 0; p < n; ++p) device_row[p] = p;
        if (on_host) memset(on_host, 0, (size_t)n);
        return ASRKF_OK;
    }
    if (device_row) HIP_OK(ctx, hipMemcpy(device_row, ctx->row_of + off, (size_t)n * 4, hipMemcpyDeviceToHost));
    if (on_host) HIP_OK(ctx, hipMemcpy(on_host, ctx->on_host + off, (size_t)n, hipMemcpyDeviceToHost));
    return ASRKF_OK;
}

asrkf_status asrkf_get_seq(asrkf_ctx* ctx, int32_t seq, float* entropy, float* pmax,
                           int32_t* escalation, int32_t* level) {
    asrkf_status st = check_ctx(ctx);
    if (st != ASRKF_OK) return st;
    if (seq < 0 || seq >= ctx->cfg.batch) return fail(ASRKF_EINVAL, "sequence out of range");
    st = sync_ctx(ctx);
    if (st != ASRKF_OK) return st;
    if (entropy) HIP_OK(ctx, hipMemcpy(entropy, ctx->entropy + seq, 4, hipMemcpyDeviceToHost));
    if (pmax) HIP_OK(ctx, hipMemcpy(pmax, ctx->pmax + seq, 4, hipMemcpyDeviceToHost));
    if (escalation) HIP_OK(ctx, hipMemcpy(escalation, ctx->escalation + seq, 4, hipMemcpyDeviceToHost));
    if (level) HIP_OK(ctx, hipMemcpy(level, ctx->level + seq, 4, hipMemcpyDeviceToHost));
    return ASRKF_OK;
}

asrkf_status asrkf_reset(asrkf_ctx* ctx) {
    asrkf_status st = check_ctx(ctx);
    if (st != ASRKF_OK) return st;
    if (ctx->queued && capturing(ctx->last_stream))
        return fail(ASRKF_ESTATE, "reset while the context's stream is being captured");
    st = sync_ctx(ctx);
    if (st != ASRKF_OK) return st;
    st = collect_timing(ctx);
    if (st != ASRKF_OK) return st;
    const asrkf_config& c = ctx->cfg;
    const size_t st_inst = (size_t)ctx->state_layers * c.batch;
    const size_t st_pos = st_inst * ctx->cap;
    // the device state of a context that has run no step: the same values asrkf_init
    // writes (every other array is written before it is read again), on the stream
    // of the context's last work, which has just drained
    hipStream_t s = ctx->last_stream;
    HIP_OK(ctx, hipMemsetAsync(ctx->unfreeze, 0, st_pos * 4, s));
    HIP_OK(ctx, hipMemsetAsync(ctx->count, 0, st_pos * 4, s));
    HIP_OK(ctx, hipMemsetAsync(ctx->n_active, 0, st_inst * 4, s));
    if (ctx->hmask) HIP_OK(ctx, hipMemsetAsync(ctx->hmask, 0, st_pos * 8, s));
    if (ctx->hlast) HIP_OK(ctx, hipMemsetAsync(ctx->hlast, 0, st_pos * 4, s));
    HIP_OK(ctx, hipMemsetAsync(ctx->plen, 0, (size_t)c.batch * 4, s));
    HIP_OK(ctx, hipMemsetAsync(ctx->escalation, 0, (size_t)c.batch * 4, s));
    HIP_OK(ctx, hipMemsetAsync(ctx->level, 0, (size_t)c.batch * 4, s));
    HIP_OK(ctx, hipMemsetAsync(ctx->entropy, 0, (size_t)c.batch * 4, s));
    HIP_OK(ctx, hipMemsetAsync(ctx->pmax, 0, (size_t)c.batch * 4, s));
    HIP_OK(ctx, hipMemsetAsync(ctx->ent_ticket, 0, (size_t)c.batch * 4, s));
    HIP_OK(ctx, hipMemsetAsync(ctx->counters, 0, kCounters * sizeof(unsigned long long), s));
    HIP_OK(ctx, hipMemsetAsync(ctx->flags, 0, 8, s));
    HIP_OK(ctx, hipMemsetAsync(ctx->t_dev, 0, 4, s));
    HIP_OK(ctx, hipStreamSynchronize(s));
    if (ctx->flags_host) ctx->flags_host[0] = ctx->flags_host[1] = 0;
    ctx->plen_host.assign(c.batch, 0);
    ctx->prefilled.assign(c.batch, 0);
    ctx->t = 0;
    ctx->next_layer = 0;
    ctx->lists_ready = false;
    ctx->xfer_recorded = false;
    ctx->flag_recorded = false;
    ctx->timing = false;
    ctx->attn_ms_done = 0.0;
    ctx->attn_launches = 0;
    ctx->launch_ms.clear();
    ctx->queued = false;
    return ASRKF_OK;
}

void asrkf_destroy(asrkf_ctx* ctx) {
    if (!ctx) return;
    (void)hipStreamSynchronize(ctx->last_stream);
    if (ctx->side) (void)hipStreamSynchronize(ctx->side);
    free_all(ctx);
    delete ctx;
}

}  // extern "C"
