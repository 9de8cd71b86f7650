/*
 * The host side of the C ABI under AddressSanitizer and
 * UndefinedBehaviorSanitizer: every entry point's argument checks (NULL
 * pointers, sizes, parameter ranges, alignment, short workspaces) and the
 * workspace-size and status-string functions. Every call here returns before
 * anything touches a GPU, so it runs on a machine without one.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "driftsched.h"

static int fails = 0;
#define EXPECT(call, want)                                                                  \
    do {                                                                                    \
        ds_status got_ = (call);                                                            \
        if (got_ != (want)) {                                                               \
            fprintf(stderr, "line %d: %s returned %d, want %d\n", __LINE__, #call, got_, want); \
            fails++;                                                                        \
        }                                                                                   \
    } while (0)

int main(void)
{
    /* fake device pointers: aligned, never dereferenced on these paths */
    void *p = (void *)(uintptr_t)0x10000;
    void *odd = (void *)(uintptr_t)0x10001;
    ds_score_params sp = {1024.0, 128.0, 512.0};
    ds_order_params op;
    memset(&op, 0, sizeof op);
    op.n_tiers = 3;
    for (int q = 0; q < 3; q++) {
        op.weight[q] = 1u + (uint32_t)q;
        op.tier_priority[q] = q;
    }
    op.aging_rate = 0.01;

    for (int op_ = 0; op_ < 8; op_++)
        for (uint64_t n = 0; n < (1ull << 31); n = n * 7 + 1)
            (void)ds_workspace_bytes((ds_op)op_, n, (uint32_t)(n % 5000));
    for (int st = -10; st <= 1; st++)
        if (!ds_status_string((ds_status)st)) fails++;
    if (ds_version() == 0) fails++;

    EXPECT(ds_characterize(p, 16, p, 0xFFFFFFFFu, p, p, 1 << 20, 0, NULL), DS_ERR_SIZE);
    EXPECT(ds_characterize(p, 16, NULL, 4, p, p, 1 << 20, 0, NULL), DS_ERR_NULL);
    EXPECT(ds_characterize(odd, 16, p, 4, p, p, 1 << 20, 0, NULL), DS_ERR_ALIGN);
    EXPECT(ds_characterize(p, 16, p, 4, p, p, 16, 0, NULL), DS_ERR_WORKSPACE);
    EXPECT(ds_characterize(p, 16, p, 0, p, NULL, 0, 0, NULL), DS_OK);

    EXPECT(ds_calibrate(p, p, p, 10, 1.5, 4, p, NULL, p, 1 << 20, 0, NULL), DS_ERR_ARG);
    EXPECT(ds_calibrate(p, p, p, 10, NAN, 4, p, NULL, p, 1 << 20, 0, NULL), DS_ERR_ARG);
    EXPECT(ds_calibrate(p, p, p, 10, 0.1, 0, p, NULL, p, 1 << 20, 0, NULL), DS_ERR_ARG);
    EXPECT(ds_calibrate(NULL, p, p, 10, 0.1, 4, p, NULL, p, 1 << 20, 0, NULL), DS_ERR_NULL);
    EXPECT(ds_calibrate(p, odd, p, 10, 0.1, 4, p, NULL, p, 1 << 20, 0, NULL), DS_ERR_ALIGN);
    EXPECT(ds_calibrate(p, p, p, (uint64_t)DS_MAX_ITEMS + 1, 0.1, 4, p, NULL, p, 1 << 20, 0, NULL),
           DS_ERR_SIZE);
    EXPECT(ds_calibrate(p, p, p, 10, 0.1, 4, p, NULL, p, 8, 0, NULL), DS_ERR_WORKSPACE);
    EXPECT(ds_calibrate_ex(p, p, p, 0, 0.1, 4, p, NULL, NULL, NULL, 0, 0, NULL), DS_OK);

    EXPECT(ds_score(4, p, p, p, p, p, 4, p, 3, p, 2, NULL, NULL, p, p, p, NULL, 0, 0, NULL), DS_ERR_NULL);
    EXPECT(ds_score(4, p, p, p, p, p, 0, p, 3, p, 2, &sp, NULL, p, p, p, NULL, 0, 0, NULL), DS_ERR_ARG);
    EXPECT(ds_score(4, p, p, p, NULL, p, 4, p, 3, p, 2, &sp, NULL, p, p, p, NULL, 0, 0, NULL), DS_ERR_ARG);
    EXPECT(ds_score(4, p, p, p, p, p, 4, p, 3, p, 2, &sp, NULL, NULL, p, p, NULL, 0, 0, NULL), DS_ERR_NULL);
    EXPECT(ds_score(4, p, p, p, p, odd, 4, p, 3, p, 2, &sp, NULL, p, p, p, NULL, 0, 0, NULL), DS_ERR_ALIGN);
    EXPECT(ds_score(4, p, p, p, p, p, 4, p, 3, p, 2, &sp, NULL, p, p, p, NULL, 0, DS_VALIDATE, NULL),
           DS_ERR_WORKSPACE);
    EXPECT(ds_score(0, p, p, p, NULL, p, 4, p, 3, p, 0, &sp, NULL, p, p, p, NULL, 0, 0, NULL), DS_OK);
    sp.f_ref = 0.0;
    EXPECT(ds_score(4, p, p, p, p, p, 4, p, 3, p, 2, &sp, NULL, p, p, p, NULL, 0, 0, NULL), DS_ERR_ARG);
    EXPECT(ds_characterize_score(p, 16, p, 4, p, p, p, p, p, 4, p, 3, p, 2, &sp, NULL, p, p, p, p, 1 << 20, 0,
                                 NULL),
           DS_ERR_ARG);
    sp.f_ref = 1024.0;
    EXPECT(ds_characterize_score(p, 16, p, 4, p, p, p, p, p, 4, p, 3, p, 2, &sp, NULL, p, p, p, p, 8, 0, NULL),
           DS_ERR_WORKSPACE);
    EXPECT(ds_characterize_score_noalloc(p, 16, p, DS_NOALLOC_MAX_PROMPTS + 1, p, p, p, p, p, 4, p, 3, p, 2,
                                         &sp, NULL, p, p, p, 0, NULL),
           DS_ERR_SIZE);
    EXPECT(ds_characterize_score_noalloc(p, 16, p, 4, p, p, p, p, p, 4, p, 3, p, 2, &sp, NULL, p, p, p,
                                         DS_VALIDATE, NULL),
           DS_ERR_ARG);

    uint32_t *perms[5] = {p, p, p, p, p};
    double *keys[5] = {NULL, NULL, NULL, NULL, NULL};
    EXPECT(ds_order(DS_FIFO, 10, p, p, NULL, NULL, NULL, p, NULL, p, 1 << 24, 0, NULL), DS_ERR_NULL);
    EXPECT(ds_order(DS_SJF, 10, p, p, NULL, NULL, &op, p, NULL, p, 1 << 24, 0, NULL), DS_ERR_NULL);
    EXPECT(ds_order(DS_FIFO, 10, p, odd, NULL, NULL, &op, p, NULL, p, 1 << 24, 0, NULL), DS_ERR_ALIGN);
    EXPECT(ds_order(DS_FIFO, 10, p, p, NULL, NULL, &op, p, NULL, p, 16, 0, NULL), DS_ERR_WORKSPACE);
    EXPECT(ds_order(DS_FIFO, DS_MAX_ITEMS + 1u, p, p, NULL, NULL, &op, p, NULL, p, 1 << 24, 0, NULL), DS_ERR_SIZE);
    EXPECT(ds_order((ds_policy)7, 10, p, p, NULL, NULL, &op, p, NULL, p, 1 << 24, 0, NULL), DS_ERR_ARG);
    op.weight[1] = 0;
    EXPECT(ds_order(DS_WEIGHTED, 10, p, p, NULL, NULL, &op, p, NULL, p, 1 << 24, 0, NULL), DS_ERR_ARG);
    op.weight[1] = 2;
    op.weighted_mode = DS_WRR_SMOOTH;
    op.weight[0] = 2000;
    EXPECT(ds_order(DS_WEIGHTED, 10, p, p, NULL, NULL, &op, p, NULL, p, 1 << 24, 0, NULL), DS_ERR_ARG);
    op.weight[0] = 1;
    op.weighted_mode = 9;
    EXPECT(ds_order(DS_WEIGHTED, 10, p, p, NULL, NULL, &op, p, NULL, p, 1 << 24, 0, NULL), DS_ERR_ARG);
    op.weighted_mode = 0;
    op.n_tiers = 17;
    EXPECT(ds_order(DS_FIFO, 10, p, p, NULL, NULL, &op, p, NULL, p, 1 << 24, 0, NULL), DS_ERR_ARG);
    op.n_tiers = 3;
    op.aging_rate = -1.0;
    EXPECT(ds_order(DS_AGING, 10, p, p, NULL, NULL, &op, p, NULL, p, 1 << 24, 0, NULL), DS_ERR_ARG);
    op.aging_rate = 0.01;
    EXPECT(ds_order_multi(0, 10, p, p, p, NULL, &op, perms, keys, p, 1 << 24, 0, NULL), DS_ERR_ARG);
    EXPECT(ds_order_multi(0x3F, 10, p, p, p, NULL, &op, perms, keys, p, 1 << 24, 0, NULL), DS_ERR_ARG);
    perms[3] = NULL;
    EXPECT(ds_order_multi(0x1F, 10, p, p, p, NULL, &op, perms, keys, p, 1 << 24, 0, NULL), DS_ERR_NULL);
    EXPECT(ds_order(DS_FIFO, 0, NULL, NULL, NULL, NULL, &op, NULL, NULL, NULL, 0, 0, NULL), DS_OK);

    EXPECT(ds_error_stats(10, p, NULL, p, p, 0, p, p, 1 << 20, 0, NULL), DS_ERR_ARG);
    EXPECT(ds_error_stats(10, NULL, NULL, p, NULL, 0, p, p, 1 << 20, 0, NULL), DS_ERR_NULL);
    EXPECT(ds_class_histogram(10, p, 0, p, p, NULL, 0, 0, NULL), DS_ERR_ARG);
    EXPECT(ds_class_histogram(10, p, 300, p, p, NULL, 0, 0, NULL), DS_ERR_ARG);

    ds_sim_params sim;
    memset(&sim, 0, sizeof sim);
    sim.policy = DS_FIFO;
    sim.batch = 0;
    sim.alpha = 0.1;
    sim.score = sp;
    sim.order = op;
    EXPECT(ds_simulate(10, p, p, p, p, p, p, p, p, 4, p, 3, 2, p, 5, &sim, p, p, p, p, p, 1 << 24, 0, NULL),
           DS_ERR_ARG);
    sim.batch = DS_MAX_BATCH + 1;
    EXPECT(ds_simulate(10, p, p, p, p, p, p, p, p, 4, p, 3, 2, p, 5, &sim, p, p, p, p, p, 1 << 24, 0, NULL),
           DS_ERR_ARG);
    sim.batch = 32;
    EXPECT(ds_simulate(10, p, p, p, p, p, p, p, p, 4, p, 3, 2, p, 5, NULL, p, p, p, p, p, 1 << 24, 0, NULL),
           DS_ERR_NULL);

    {
        ds_sim_params runs[2];
        runs[0] = sim;
        runs[1] = sim;
        double *st[2] = {p, p};
        uint32_t *sq[2] = {p, p};
        int32_t *tk[2] = {p, p};
        EXPECT(ds_simulate_multi(0, 10, p, p, p, p, p, p, p, p, 4, p, 3, 2, p, 5, runs, st, sq, tk, p, p, 1 << 26,
                                 0, NULL),
               DS_ERR_ARG);
        EXPECT(ds_simulate_multi(DS_SIM_MAX_RUNS + 1, 10, p, p, p, p, p, p, p, p, 4, p, 3, 2, p, 5, runs, st, sq,
                                 tk, p, p, 1 << 26, 0, NULL),
               DS_ERR_ARG);
        runs[1].batch = 0;
        EXPECT(ds_simulate_multi(2, 10, p, p, p, p, p, p, p, p, 4, p, 3, 2, p, 5, runs, st, sq, tk, p, p, 1 << 26,
                                 0, NULL),
               DS_ERR_ARG);
        runs[1].batch = 32;
        EXPECT(ds_simulate_multi(2, 10, p, p, p, p, p, p, p, p, 4, p, 3, 2, p, 5, runs, st, sq, tk, p, p, 64, 0,
                                 NULL),
               DS_ERR_WORKSPACE);
        EXPECT(ds_simulate_multi(2, 10, p, p, p, p, p, p, p, p, 4, p, 3, 2, p, 5, NULL, st, sq, tk, p, p, 1 << 26, 0,
                                 NULL),
               DS_ERR_NULL);
    }

    EXPECT(ds_read_bandwidth(odd, 16, p, NULL), DS_ERR_ALIGN);
    EXPECT(ds_read_bandwidth(p, 15, p, NULL), DS_ERR_ARG);

    if (fails) {
        fprintf(stderr, "%d checks failed\n", fails);
        return 1;
    }
    printf("ABI host-side sanitizer checks: ok\n");
    return 0;
}
