/* A plain C program that runs the decode step through the C ABI on the GPU,
 * with HIP device buffers and no Python.  Exit status 0 when every check holds.
 *
 * Workload: 1 layer, 2 sequences (prompts of 40 and 0 tokens), 8 q / 2 KV
 * heads, head_dim 64, fp32, 12 steps, tau = -inf so that no score is below
 * the threshold and nothing ever freezes: every step is dense attention over
 * all positions, which the program recomputes here in double precision,
 *     out_h = sum_j softmax_j(q_h . k_{g(h), j} / sqrt(D)) v_{g(h), j},  g(h) = h / 4,
 * and compares element by element (2e-4 absolute).  It also checks the step
 * counter, the attended-token total and the active positions reported by
 * asrkf_stats, and that a forced Full Reset leaves the dense path unchanged. */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "asrkf.h"

enum { L = 1, B = 2, HQ = 8, HKV = 2, D = 64, STEPS = 12, P0 = 40, P1 = 0, CAP = 64 };

#define CHECK(cond)                                                            \
    do {                                                                       \
        if (!(cond)) {                                                         \
            fprintf(stderr, "check failed: %s (line %d): %s\n", #cond, __LINE__, \
                    asrkf_last_error());                                       \
            return 1;                                                          \
        }                                                                      \
    } while (0)

static unsigned long long rng = 0x2512112211ull;
static float uniform_pm1(void) {               /* xorshift64*, values in [-1, 1) */
    rng ^= rng >> 12;
    rng ^= rng << 25;
    rng ^= rng >> 27;
    const unsigned long long x = rng * 2685821657736338717ull;
    return (float)((double)(x >> 11) / 9007199254740992.0 * 2.0 - 1.0);
}

/* keys and values of every position of every sequence, [b][pos][HKV][D] */
static float kall[B][CAP][HKV][D], vall[B][CAP][HKV][D];

int main(void) {
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) {
        fprintf(stderr, "no GPU\n");
        return 2;
    }
    asrkf_config cfg;
    memset(&cfg, 0, sizeof cfg);
    cfg.n_layers = L;
    cfg.batch = B;
    cfg.n_q_heads = HQ;
    cfg.n_kv_heads = HKV;
    cfg.head_dim = D;
    cfg.max_ctx = CAP;
    cfg.window_K = 4;
    cfg.tau = -INFINITY;
    cfg.k_soft = 2.0f;
    cfg.vocab = 8;
    cfg.entropy_spike = INFINITY;
    cfg.dtype = ASRKF_F32;
    asrkf_ctx* ctx = NULL;
    CHECK(asrkf_init(&cfg, &ctx) == ASRKF_OK);

    for (int b = 0; b < B; ++b)
        for (int p = 0; p < CAP; ++p)
            for (int g = 0; g < HKV; ++g)
                for (int e = 0; e < D; ++e) {
                    kall[b][p][g][e] = uniform_pm1();
                    vall[b][p][g][e] = uniform_pm1();
                }
    float *dk, *dv, *dq, *dout;
    const size_t row = (size_t)HKV * D * sizeof(float);
    CHECK(hipMalloc((void**)&dk, CAP * row) == hipSuccess);
    CHECK(hipMalloc((void**)&dv, CAP * row) == hipSuccess);
    CHECK(hipMalloc((void**)&dq, (size_t)B * HQ * D * sizeof(float)) == hipSuccess);
    CHECK(hipMalloc((void**)&dout, (size_t)B * HQ * D * sizeof(float)) == hipSuccess);
    const int plen[B] = {P0, P1};
    for (int b = 0; b < B; ++b) {
        if (!plen[b]) continue;
        CHECK(hipMemcpy(dk, kall[b], plen[b] * row, hipMemcpyHostToDevice) == hipSuccess);
        CHECK(hipMemcpy(dv, vall[b], plen[b] * row, hipMemcpyHostToDevice) == hipSuccess);
        CHECK(asrkf_prefill(ctx, 0, b, dk, dv, plen[b], NULL) == ASRKF_OK);
        CHECK(hipDeviceSynchronize() == hipSuccess);
    }

    static float q[B][HQ][D], knew[B][HKV][D], vnew[B][HKV][D], out[B][HQ][D];
    long long attended = 0;
    for (int t = 1; t <= STEPS; ++t) {
        for (int b = 0; b < B; ++b) {
            const int p = plen[b] + t - 1;              /* position of the new token */
            memcpy(knew[b], kall[b][p], row);
            memcpy(vnew[b], vall[b][p], row);
            for (int h = 0; h < HQ; ++h)
                for (int e = 0; e < D; ++e) q[b][h][e] = uniform_pm1();
        }
        CHECK(hipMemcpy(dq, q, sizeof q, hipMemcpyHostToDevice) == hipSuccess);
        CHECK(hipMemcpy(dk, knew, sizeof knew, hipMemcpyHostToDevice) == hipSuccess);
        CHECK(hipMemcpy(dv, vnew, sizeof vnew, hipMemcpyHostToDevice) == hipSuccess);
        CHECK(asrkf_decode_step(ctx, 0, dq, dk, dv, dout, NULL) == ASRKF_OK);
        CHECK(asrkf_restore(ctx, NULL, t == 6 ? ASRKF_FR : ASRKF_AUTO, NULL) == ASRKF_OK);
        CHECK(hipMemcpy(out, dout, sizeof out, hipMemcpyDeviceToHost) == hipSuccess);
        for (int b = 0; b < B; ++b) {
            const int n = plen[b] + t;                  /* every position attends */
            attended += n;
            for (int h = 0; h < HQ; ++h) {
                const int g = h / (HQ / HKV);
                double m = -INFINITY, s = 0.0, acc[D];
                double x[CAP];
                for (int j = 0; j < n; ++j) {
                    double dot = 0.0;
                    for (int e = 0; e < D; ++e) dot += (double)q[b][h][e] * kall[b][j][g][e];
                    x[j] = dot / sqrt((double)D);
                    if (x[j] > m) m = x[j];
                }
                for (int e = 0; e < D; ++e) acc[e] = 0.0;
                for (int j = 0; j < n; ++j) {
                    const double w = exp(x[j] - m);
                    s += w;
                    for (int e = 0; e < D; ++e) acc[e] += w * vall[b][j][g][e];
                }
                for (int e = 0; e < D; ++e) {
                    const double ref = acc[e] / s;
                    if (fabs(ref - out[b][h][e]) > 2e-4) {
                        fprintf(stderr, "step %d seq %d head %d dim %d: %g vs %g\n", t, b, h, e,
                                (double)out[b][h][e], ref);
                        return 1;
                    }
                }
            }
        }
    }
    asrkf_stats_t st;
    CHECK(asrkf_stats(ctx, &st) == ASRKF_OK);
    CHECK(st.step == STEPS);
    CHECK(st.attended_total == attended);
    CHECK(st.total_positions == (long long)(P0 + P1 + 2 * STEPS));
    CHECK(st.active_positions == st.total_positions);   /* nothing frozen */
    CHECK(st.recoveries[3] == B);                         /* the forced Full Reset */
    asrkf_destroy(ctx);
    CHECK(hipFree(dk) == hipSuccess && hipFree(dv) == hipSuccess);
    CHECK(hipFree(dq) == hipSuccess && hipFree(dout) == hipSuccess);
    printf("C ABI GPU run passed: %d steps, %lld attended token-layers\n", STEPS, attended);
    return 0;
}
