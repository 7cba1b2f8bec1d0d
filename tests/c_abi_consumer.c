/*
 * A plain C99 program that uses the optimizer library through its header
 * alone: the header must compile as C, and every host-only entry point must
 * behave as documented when called from C (no GPU is needed; nothing here
 * launches a kernel). Prints one line per failed check and exits non-zero on
 * any failure.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "lamb_mi355x.h"

static int failures = 0;

#define CHECK(cond)                                                   \
    do {                                                              \
        if (!(cond)) {                                                \
            printf("FAILED line %d: %s\n", __LINE__, #cond);          \
            ++failures;                                               \
        }                                                             \
    } while (0)

static void status_strings(void) {
    int code;
    for (code = LAMB_ESYNC; code <= LAMB_OK; ++code) {
        const char *s = lamb_status_str(code);
        CHECK(s != NULL && s[0] != '\0' && strcmp(s, "unknown status") != 0);
    }
    CHECK(strcmp(lamb_status_str(-99), "unknown status") == 0);
}

/* Section 4 / Appendix H defaults as the header documents them. */
static void hparams(void) {
    lamb_hparams hp;
    CHECK(lamb_hparams_init(&hp, LAMB_VARIANT_LAMB) == LAMB_OK);
    CHECK(hp.variant == LAMB_VARIANT_LAMB && hp.norm == LAMB_NORM_L2 && hp.step == 1);
    CHECK(hp.beta1 == 0.9f && hp.beta2 == 0.999f && hp.eps == 1e-6f);
    CHECK(hp.weight_decay == 0.01f && hp.grad_scale == 1.0f && hp.bias_correction == 1);
    CHECK(lamb_hparams_init(&hp, LAMB_VARIANT_NLAMB) == LAMB_OK && hp.beta1 == 0.975f);
    CHECK(lamb_hparams_init(&hp, LAMB_VARIANT_LARS) == LAMB_OK && hp.trust_coef == 1.0f);
    CHECK(lamb_hparams_init(&hp, 9) == LAMB_EINVAL);
    CHECK(lamb_hparams_init(NULL, 0) == LAMB_ENULL);
}

/* Tensor i cut into ceil(n_i / C) chunks of C elements, the last ragged. */
static void chunk_table(void) {
    const int64_t numel[3] = {5, 1024, 1030};
    int32_t ct[8], cl[8], n = -1;
    int64_t cs[8];
    static const int32_t want_t[6] = {0, 1, 1, 2, 2, 2};
    static const int64_t want_s[6] = {0, 0, 512, 0, 512, 1024};
    static const int32_t want_l[6] = {5, 512, 512, 512, 512, 6};
    int k;
    CHECK(lamb_chunk_table(numel, 3, 512, 0, NULL, NULL, NULL, &n) == LAMB_OK && n == 6);
    CHECK(lamb_chunk_table(numel, 3, 512, 8, ct, cs, cl, &n) == LAMB_OK && n == 6);
    for (k = 0; k < 6; ++k)
        CHECK(ct[k] == want_t[k] && cs[k] == want_s[k] && cl[k] == want_l[k]);
    CHECK(lamb_chunk_table(numel, 3, 512, 5, ct, cs, cl, &n) == LAMB_EINVAL && n == 6);
    CHECK(lamb_chunk_table(numel, 3, 12, 8, ct, cs, cl, &n) == LAMB_EINVAL);
    CHECK(lamb_chunk_table(NULL, 3, 512, 8, ct, cs, cl, &n) == LAMB_ENULL);
    /* sizes beyond 2^40 are rejected before anything is counted */
    {
        const int64_t huge[2] = {5, INT64_MAX};
        CHECK(lamb_chunk_table(huge, 2, 8, 0, NULL, NULL, NULL, &n) == LAMB_EINVAL);
    }
}

/*
 * Three layers of 3, 1 and 2 tiles of 8192 elements with rounds of at most 4
 * entries (the wide tile puts no more of them on the single pass, so a plan
 * keeps the narrow one): two rounds are needed, and the narrowest width that
 * still packs into two is 3: [layer 0 x3][layer 2 x2, layer 1 x1]. Every
 * element of every layer is held by exactly one entry.
 */
static void tile_schedule(void) {
    const int64_t numel[3] = {3 * 8192 - 100, 8192, 2 * 8192};
    int32_t et[8], el[8], first[3], tiles[3], n = -1, round = -1, groups = -1, i, k;
    int64_t es[8], covered[3] = {0, 0, 0};
    CHECK(lamb_tile_schedule(numel, 3, 4, 0, 8, et, es, el, first, tiles, &n, &round,
                             &groups) == LAMB_OK);
    CHECK(groups == 8 && n == 6 && round == 3);
    CHECK(tiles[0] == 3 && tiles[1] == 1 && tiles[2] == 2);
    CHECK(first[0] == 0 && first[2] == 3 && first[1] == 5);
    for (k = 0; k < n; ++k) {
        CHECK(et[k] >= 0 && et[k] < 3);
        if (et[k] >= 0 && et[k] < 3) {
            covered[et[k]] += el[k];
            /* a layer's tiles are consecutive entries inside one round */
            CHECK(k - first[et[k]] >= 0 && k - first[et[k]] < tiles[et[k]]);
            CHECK(k / round == first[et[k]] / round);
            CHECK(es[k] == (int64_t)(k - first[et[k]]) * 1024);
        }
    }
    for (i = 0; i < 3; ++i)
        CHECK(covered[i] == numel[i]);
    /* five 8192-element tiles are too many for a round of 4, four of 10240
     * are not: a plan picks the wide tile for this layer */
    {
        const int64_t big[1] = {5 * 8192};
        CHECK(lamb_tile_schedule(big, 1, 4, 8, 8, et, es, el, first, tiles, &n, &round,
                                 NULL) == LAMB_OK);
        CHECK(tiles[0] == 0 && n == 0);
        CHECK(lamb_tile_schedule(big, 1, 4, 0, 8, et, es, el, first, tiles, &n, &round,
                                 &groups) == LAMB_OK);
        CHECK(groups == 10 && tiles[0] == 4 && n == 4 && el[3] == 10 * 1024);
        CHECK(lamb_tile_schedule(big, 1, 4, 9, 8, et, es, el, first, tiles, &n, &round,
                                 NULL) == LAMB_EINVAL);
    }
    {
        const int64_t huge[1] = {((int64_t)1 << 40) + 1};
        CHECK(lamb_tile_schedule(huge, 1, 4, 0, 8, et, es, el, first, tiles, &n, &round,
                                 NULL) == LAMB_EINVAL);
    }
}

/* Section 4: linear warmup, then polynomial decay; stages back to back. */
static void lr_schedule(void) {
    lamb_lr_stage st[2];
    double lr = -1.0;
    st[0].steps = 10; st[0].warmup_steps = 4; st[0].peak_lr = 1.0; st[0].power = 1.0;
    st[1].steps = 5;  st[1].warmup_steps = 0; st[1].peak_lr = 0.5; st[1].power = 2.0;
    CHECK(lamb_lr_at(st, 2, 1, &lr) == LAMB_OK && lr == 0.25);  /* (0 + 1) / 4 */
    CHECK(lamb_lr_at(st, 2, 4, &lr) == LAMB_OK && lr == 1.0);   /* last warmup step */
    CHECK(lamb_lr_at(st, 2, 5, &lr) == LAMB_OK && fabs(lr - 0.6) < 1e-15);  /* 1 - 4/10 */
    CHECK(lamb_lr_at(st, 2, 11, &lr) == LAMB_OK && lr == 0.5);  /* second stage, tau 0 */
    CHECK(lamb_lr_at(st, 2, 12, &lr) == LAMB_OK && fabs(lr - 0.5 * 0.8 * 0.8) < 1e-15);
    CHECK(lamb_lr_at(st, 2, 16, &lr) == LAMB_OK && lr == 0.0);  /* after the last stage */
    lr = 7.0;
    CHECK(lamb_lr_at(st, 2, 0, &lr) == LAMB_EINVAL && lr == 7.0);
    CHECK(lamb_sqrt_scaled_lr(1e-3, 512, 2048, &lr) == LAMB_OK && fabs(lr - 2e-3) < 1e-18);
    CHECK(lamb_sqrt_scaled_lr(1e-3, 0, 2048, &lr) == LAMB_EINVAL);
}

/* Validation runs on the host before any HIP call. */
static void rejected_calls(void) {
    lamb_plan *plan = NULL;
    lamb_tensor t;
    lamb_hparams hp;
    memset(&t, 0, sizeof t);
    CHECK(lamb_plan_create(&t, 0, LAMB_GRAD_F32, LAMB_ALGO_LAMB, 0, &plan) == LAMB_EINVAL);
    CHECK(plan == NULL && lamb_last_error()[0] != '\0');
    CHECK(lamb_plan_create(&t, 1, LAMB_GRAD_F32, LAMB_ALGO_LAMB, 0, &plan) == LAMB_ENULL);
    CHECK(lamb_plan_create(NULL, 1, LAMB_GRAD_F32, LAMB_ALGO_LAMB, 0, &plan) == LAMB_ENULL);
    /* out-of-range enum values are rejected, not assumed away */
    CHECK(lamb_plan_create(&t, 1, 2, LAMB_ALGO_LAMB, 0, &plan) == LAMB_EINVAL);
    CHECK(lamb_plan_create(&t, 1, -1, LAMB_ALGO_LAMB, 0, &plan) == LAMB_EINVAL);
    CHECK(lamb_plan_create(&t, 1, LAMB_GRAD_F32, 7, 0, &plan) == LAMB_EINVAL);
    CHECK(plan == NULL);
    CHECK(lamb_plan_destroy(NULL) == LAMB_OK);
    CHECK(lamb_step(NULL, 1e-3f, 0.9f, 0.999f, 1e-6f, 0.01f, 0.0f, 10.0f, 1, 1, NULL, NULL,
                    NULL) == LAMB_ENULL);
    CHECK(lars_step(NULL, 1e-3f, 0.9f, 0.01f, 0.0f, 10.0f, 1e-3f, NULL, NULL, NULL) ==
          LAMB_ENULL);
    CHECK(lamb_hparams_init(&hp, LAMB_VARIANT_LAMB) == LAMB_OK);
    CHECK(lamb_step_ex(NULL, &hp, NULL, NULL, NULL, NULL) == LAMB_ENULL);
    CHECK(lamb_plan_check(NULL, NULL) == LAMB_ENULL);
    {
        double totals[3] = {0.0, 0.0, 0.0};
        int32_t n = -1;
        CHECK(lamb_step_partials(NULL, &hp, NULL, totals) == LAMB_ENULL);
        CHECK(lamb_step_finish(NULL, &hp, NULL, totals, NULL, NULL, NULL) == LAMB_ENULL);
        CHECK(lamb_plan_set_u_check(NULL, 1) == LAMB_ENULL);
        CHECK(lamb_plan_u_partials(NULL, NULL, 0, NULL, NULL, &n) == LAMB_ENULL);
    }
}

int main(void) {
    status_strings();
    hparams();
    chunk_table();
    tile_schedule();
    lr_schedule();
    rejected_calls();
    if (failures == 0)
        printf("c abi consumer: all checks passed\n");
    return failures == 0 ? 0 : 1;
}
