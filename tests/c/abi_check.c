/* Plain-C client of the eviction library: the header compiles as C99 and the host-side entry points
 * (sizing, argument validation, status strings) behave as documented.  No GPU work is queued: every call
 * below is rejected or answered on the host. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "inertiakv.h"

static int failures = 0;
#define CHECK(cond)                                                        \
    do {                                                                   \
        if (!(cond)) {                                                     \
            fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
            ++failures;                                                    \
        }                                                                  \
    } while (0)

int main(void) {
    kv_shape s = {8, 32, 32, 8, 128, 32769, KV_BF16};
    size_t ws = 0, ws_small = 0, st = 0;
    CHECK(kv_workspace_bytes(&s, 3278, &ws_small) == KV_OK);
    CHECK(kv_workspace_bytes(&s, 32769, &ws) == KV_OK);
    CHECK(ws > ws_small && ws_small > 0);
    CHECK(kv_workspace_bytes(&s, 32770, &ws) == KV_ERR_INVALID_ARG);  /* beyond capacity */
    CHECK(kv_workspace_bytes(NULL, 10, &ws) == KV_ERR_INVALID_ARG);

    kv_shape bad = s;
    bad.head_dim = 96;
    CHECK(kv_workspace_bytes(&bad, 10, &ws) == KV_ERR_UNSUPPORTED);
    bad = s;
    bad.n_q_heads = 30; /* not a multiple of the KV heads */
    CHECK(kv_workspace_bytes(&bad, 10, &ws) == KV_ERR_INVALID_ARG);

    kv_params p;
    memset(&p, 0, sizeof p);
    p.alpha = 0.9f;
    p.budget = 3277;
    p.refresh_period = 4;
    p.nonrefresh_init = KV_INIT_MIN;
    p.rule = KV_RULE_EMA;
    p.score_variant = KV_SCORE_VNORM | KV_SCORE_ENTROPY;
    int32_t n_out = -7;
    void* fake = (void*)(uintptr_t)(1u << 20); /* never dereferenced: validation fails first */
    /* no workspace: rejected before anything is queued, n_out untouched */
    CHECK(kv_evict_step(&s, &p, 2, 3277, 40000, fake, fake, fake, fake, fake, (float*)fake, (int32_t*)fake, NULL, &n_out,
                        NULL, NULL, NULL, NULL, NULL, 0, NULL) == KV_ERR_WORKSPACE);
    CHECK(n_out == -7);
    p.alpha = 1.0f;
    CHECK(kv_evict_step(&s, &p, 2, 3277, 40000, fake, fake, fake, fake, fake, (float*)fake, (int32_t*)fake, NULL, &n_out,
                        NULL, NULL, NULL, NULL, NULL, 0, NULL) == KV_ERR_INVALID_ARG);
    p.alpha = 0.9f;
    p.score_merge = 3; /* not a divisor of the 8 KV heads */
    CHECK(kv_evict_step(&s, &p, 2, 3277, 40000, fake, fake, fake, fake, fake, (float*)fake, (int32_t*)fake, NULL, &n_out,
                        NULL, NULL, NULL, NULL, NULL, 0, NULL) == KV_ERR_INVALID_ARG);
    p.score_merge = 0;
    CHECK(kv_attend_score(&s, 30, 3, 3278, fake, fake, fake, (const int32_t*)fake, 40000, 0.5f, 64, 1, fake, NULL, 0,
                          NULL) == KV_ERR_INVALID_ARG); /* layers 30..32 past the last */
    CHECK(kv_rank_trace_state_bytes(8, 40000, &st) == KV_OK && st == 8 * (4 + 2 * 1250) * 4);

    /* scorer plan of a steady step (slabs of 3,278 rows fit one workgroup's LDS) */
    kv_score_info info = {-1, -1, -1};
    p.score_variant = 0;
    CHECK(kv_score_plan(&s, 3278, &p, &info) == KV_OK);
    CHECK(info.path == KV_PATH_LDS && info.chunks == 1 && info.merge >= 1 && 8 % info.merge == 0);
    CHECK(kv_score_plan(&s, 32770, &p, &info) == KV_ERR_INVALID_ARG);
    /* fault word: validated on the host (nothing queued) */
    CHECK(kv_fault_status(NULL, ws, (uint32_t*)fake, 0, NULL) == KV_ERR_WORKSPACE);
    CHECK(kv_fault_status(fake, ws, NULL, 0, NULL) == KV_ERR_INVALID_ARG);
    {
        const int32_t def = kv_set_exchange_wait_limit(3);
        CHECK(def > 0);
        CHECK(kv_set_exchange_wait_limit(-1) == 3);
        CHECK(kv_set_exchange_wait_limit(-1) == def);
    }
    (void)KV_FAULT_EXCHANGE_TIMEOUT;
    CHECK(kv_value_norms(&s, 0, fake, (float*)fake, NULL) == KV_ERR_INVALID_ARG);

    CHECK(strcmp(kv_status_string(KV_OK), "ok") == 0);
    CHECK(strlen(kv_status_string(KV_ERR_HIP)) > 0);
    CHECK(strlen(kv_status_string((kv_status)-99)) > 0);
    if (failures) return 1;
    printf("ok\n");
    return 0;
}
