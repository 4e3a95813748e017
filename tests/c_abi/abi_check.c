/* A plain C caller of the library's C ABI (host-only calls: no GPU needed).
 * Exit status 0 when every check holds; the failing check is printed otherwise.
 *  - asrkf_schedule_table for k = 2 against Eq. 3's closed form
 *    d(c) = floor(sqrt(c) / 2) = floor(isqrt(c) / 2), computed here in integers;
 *  - the table's argument checks;
 *  - asrkf_init rejecting an invalid configuration with ASRKF_EINVAL and a
 *    message from asrkf_last_error. */
#include <stdio.h>
#include <string.h>

#include "asrkf.h"

static int isqrt(int c) {
    int r = 0;
    while ((r + 1) * (r + 1) <= c) ++r;
    return r;
}

#define CHECK(cond)                                                  \
    do {                                                             \
        if (!(cond)) {                                               \
            fprintf(stderr, "check failed: %s (line %d)\n", #cond, __LINE__); \
            return 1;                                                \
        }                                                            \
    } while (0)

int main(void) {
    enum { N = 5000 };
    static int32_t d[N];
    CHECK(asrkf_schedule_table(2.0f, N, d) == ASRKF_OK);
    for (int c = 0; c < N; ++c) CHECK(d[c] == isqrt(c) / 2);
    CHECK(d[1] == 0 && d[4] == 1 && d[9] == 1 && d[16] == 2);
    CHECK(asrkf_schedule_table(0.0f, 10, d) == ASRKF_EINVAL);
    CHECK(asrkf_schedule_table(2.0f, 0, d) == ASRKF_EINVAL);

    asrkf_config cfg;
    memset(&cfg, 0, sizeof cfg);
    cfg.n_layers = 1;
    cfg.batch = 1;
    cfg.n_q_heads = 8;
    cfg.n_kv_heads = 3;              /* not a supported number of KV heads */
    cfg.head_dim = 64;
    cfg.max_ctx = 100;
    cfg.window_K = 4;
    cfg.tau = 0.5f;
    cfg.k_soft = 2.0f;
    cfg.vocab = 16;
    cfg.dtype = ASRKF_F32;
    asrkf_ctx* ctx = NULL;
    CHECK(asrkf_init(&cfg, &ctx) == ASRKF_EINVAL);
    CHECK(ctx == NULL);
    CHECK(asrkf_last_error() != NULL && strlen(asrkf_last_error()) > 0);
    printf("C ABI checks passed (%s)\n", asrkf_last_error());
    return 0;
}
