/*
 * Exercises every function of the CPU oracle on small inputs and their edge
 * cases (empty batches, ragged prompts, malformed UTF-8, out-of-range
 * indices, skipped events, all policies and readings, the tick loop), for a
 * build under AddressSanitizer and UndefinedBehaviorSanitizer. It checks
 * return codes and a few invariants; the values themselves are pinned by
 * the Python test suite.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int dsref_is_space(uint32_t cp);
uint32_t dsref_count_words(const uint8_t *s, uint64_t len);
int dsref_characterize(const uint8_t *text, uint64_t text_bytes, const uint64_t *offsets, uint64_t n,
                       uint32_t *counts);
int dsref_calibrate_ex(const uint32_t *group, const double *est, const uint32_t *obs, uint64_t n,
                       double alpha, uint32_t n_groups, double *state, double *trace, double *before);
int dsref_error_stats(uint64_t n, const double *est, const double *factor, const uint32_t *obs,
                      const uint32_t *group, uint32_t n_groups, double *stats);
int dsref_class_histogram(uint64_t n, const uint8_t *category, uint32_t n_cat, const uint8_t *job_class,
                          uint32_t *hist);
int dsref_score(uint64_t n, const uint32_t *counts, const uint8_t *category, const uint32_t *tenant,
                const uint32_t *group, const double *t_base, uint32_t n_cat, const double *s_tenant,
                uint32_t n_tenants, const double *state, uint32_t n_groups, double f_ref,
                double short_max, double medium_max, double *est_base, double *est, double *budget,
                uint8_t *job_class);
int dsref_order(int policy, uint32_t n, const uint8_t *tier, const double *arrival, const double *budget,
                uint32_t n_tiers, const uint32_t *weight, const double *tier_priority, double aging_rate,
                double t_now, double aging_floor, uint32_t *perm, double *key);
int dsref_simulate(int policy, uint32_t n, const double *arrival, const uint8_t *tier,
                   const uint32_t *counts, const uint8_t *category, const uint32_t *tenant,
                   const uint32_t *group, const uint32_t *observed, const double *t_base, uint32_t n_cat,
                   const double *s_tenant, uint32_t n_tenants, uint32_t n_groups, double f_ref,
                   double short_max, double medium_max, uint32_t n_tiers, const uint32_t *weight,
                   const double *tier_priority, double aging_rate, double aging_floor, double alpha,
                   uint32_t batch, const double *tick_t, uint32_t n_ticks, double *state, uint32_t *seq,
                   int32_t *tick_of, uint32_t *n_dispatched);

static uint64_t rs = 0x9E3779B97F4A7C15ull;
static uint32_t rnd(uint32_t k)   /* uniform in [0, k) */
{
    rs ^= rs << 13;
    rs ^= rs >> 7;
    rs ^= rs << 17;
    return k ? (uint32_t)(rs % k) : 0u;
}

static int fails = 0;
#define CHECK(c)                                                          \
    do {                                                                  \
        if (!(c)) {                                                       \
            fprintf(stderr, "check failed line %d: %s\n", __LINE__, #c); \
            fails++;                                                      \
        }                                                                 \
    } while (0)

/* exact-size heap copies so that an overrun is caught */
static void *dup(const void *p, size_t bytes)
{
    void *q = malloc(bytes ? bytes : 1);
    if (bytes) memcpy(q, p, bytes);
    return q;
}

static void characterize_cases(void)
{
    static const uint8_t pieces[][4] = {{'a'}, {' '}, {'\t'}, {0xC2, 0x85}, {0xC2, 0xA0}, {0xE3, 0x80, 0x80},
                                        {0xE2, 0x80, 0xAF}, {0xC3, 0x85}, {0xE4, 0xB8, 0x80}, {0xFF},
                                        {0xC2}, {0xE2, 0x80}, {0x80}, {0xF0, 0x9F, 0x98, 0x80}};
    static const int plen[] = {1, 1, 1, 2, 2, 3, 3, 2, 3, 1, 1, 2, 1, 4};
    for (int trial = 0; trial < 400; trial++) {
        uint32_t n = rnd(12);
        uint64_t *off = malloc(sizeof(uint64_t) * (n + 1));
        uint8_t buf[4096];
        uint64_t b = 0;
        off[0] = 0;
        for (uint32_t i = 0; i < n; i++) {
            uint32_t parts = rnd(20);
            for (uint32_t k = 0; k < parts && b + 4 < sizeof buf; k++) {
                int p = (int)rnd(14);
                memcpy(buf + b, pieces[p], (size_t)plen[p]);
                b += (uint64_t)plen[p];
            }
            off[i + 1] = b;
        }
        uint8_t *text = dup(buf, b);
        uint64_t *o = dup(off, sizeof(uint64_t) * (n + 1));
        uint32_t *counts = malloc(sizeof(uint32_t) * (n ? n : 1));
        CHECK(dsref_characterize(b ? text : NULL, b, o, n, counts) == 0);
        for (uint32_t i = 0; i < n; i++)
            CHECK(counts[i] == dsref_count_words(text + o[i], o[i + 1] - o[i]));
        if (n >= 2) {   /* offsets that go backwards or past the text are refused */
            o[1] = o[2] + 1;
            CHECK(dsref_characterize(text, b, o, n, counts) != 0 || o[2] + 1 > b);
        }
        free(text);
        free(o);
        free(off);
        free(counts);
    }
    CHECK(dsref_count_words(NULL, 0) == 0);
    for (uint32_t cp = 0; cp < 0x3100; cp++) (void)dsref_is_space(cp);
}

static void calibrate_score_cases(void)
{
    for (int trial = 0; trial < 300; trial++) {
        uint32_t n = rnd(200), G = 1 + rnd(9);
        uint32_t *grp = malloc(4 * (n ? n : 1)), *obs = malloc(4 * (n ? n : 1));
        double *est = malloc(8 * (n ? n : 1)), *trace = malloc(8 * (n ? n : 1)),
               *before = malloc(8 * (n ? n : 1)), *state = malloc(8 * G);
        for (uint32_t g = 0; g < G; g++) state[g] = 1.0;
        for (uint32_t e = 0; e < n; e++) {
            grp[e] = rnd(G);
            obs[e] = rnd(2000);
            uint32_t k = rnd(10);
            est[e] = k == 0 ? 0.0 : k == 1 ? -3.0 : k == 2 ? NAN : k == 3 ? INFINITY : 1.0 + rnd(900);
        }
        double alpha = (double)rnd(5) / 4.0;
        CHECK(dsref_calibrate_ex(grp, est, obs, n, alpha, G, state, trace, before) == 0);
        CHECK(dsref_calibrate_ex(grp, est, obs, n, alpha, G, state, NULL, NULL) == 0);
        double *stats = malloc(8 * 4 * (G + 1));
        CHECK(dsref_error_stats(n, est, trace, obs, grp, G, stats) == 0);
        CHECK(dsref_error_stats(n, est, NULL, obs, NULL, 0, stats) == 0);
        if (n) {
            grp[n - 1] = G;   /* out of range */
            CHECK(dsref_calibrate_ex(grp, est, obs, n, alpha, G, state, trace, before) != 0);
            CHECK(dsref_error_stats(n, est, NULL, obs, grp, G, stats) != 0);
        }
        /* score, grouped and per request */
        uint32_t *counts = malloc(4 * (n ? n : 1)), *ten = malloc(4 * (n ? n : 1)), *g2 = malloc(4 * (n ? n : 1));
        uint8_t *cat = malloc(n ? n : 1), *cls = malloc(n ? n : 1);
        double *eb = malloc(8 * (n ? n : 1)), *es = malloc(8 * (n ? n : 1)), *bu = malloc(8 * (n ? n : 1));
        double tb[4] = {32, 128, 256, 512}, s[3] = {1.25, 1.125, 1.0};
        for (uint32_t i = 0; i < n; i++) {
            counts[i] = rnd(5000);
            cat[i] = (uint8_t)rnd(4);
            ten[i] = rnd(3);
            g2[i] = rnd(G);
        }
        CHECK(dsref_score(n, counts, cat, ten, g2, tb, 4, s, 3, state, G, 1024.0, 128.0, 512.0, eb, es, bu,
                          cls) == 0);
        CHECK(dsref_score(n, counts, cat, ten, NULL, tb, 4, s, 3, est, n, 1024.0, 128.0, 512.0, NULL, es, bu,
                          cls) == 0);
        if (n) CHECK(dsref_score(n, counts, cat, ten, NULL, tb, 4, s, 3, est, n + 1, 1024.0, 128.0, 512.0,
                                 NULL, es, bu, cls) != 0);
        uint32_t *hist = malloc(4 * 3 * 4);
        CHECK(dsref_class_histogram(n, cat, 4, cls, hist) == 0);
        if (n) {
            cat[0] = 9;
            CHECK(dsref_class_histogram(n, cat, 4, cls, hist) != 0);
            CHECK(dsref_score(n, counts, cat, ten, g2, tb, 4, s, 3, state, G, 1024.0, 128.0, 512.0, eb, es,
                              bu, cls) != 0);
        }
        free(grp); free(obs); free(est); free(trace); free(before); free(state); free(stats);
        free(counts); free(ten); free(g2); free(cat); free(cls); free(eb); free(es); free(bu); free(hist);
    }
}

static void order_cases(void)
{
    for (int trial = 0; trial < 400; trial++) {
        uint32_t n = rnd(300), Q = 1 + rnd(5);
        uint8_t *tier = malloc(n ? n : 1);
        double *arr = malloc(8 * (n ? n : 1)), *bud = malloc(8 * (n ? n : 1)), *key = malloc(8 * (n ? n : 1));
        uint32_t *perm = malloc(4 * (n ? n : 1)), w[5];
        double prio[5];
        for (uint32_t q = 0; q < Q; q++) {
            w[q] = 1 + rnd(9);
            prio[q] = (double)rnd(3);
        }
        for (uint32_t i = 0; i < n; i++) {
            tier[i] = (uint8_t)rnd(Q);
            arr[i] = rnd(4) == 0 ? -0.0 : (double)rnd(50) * 0.25;
            bud[i] = (double)rnd(20);
        }
        for (int pol = 0; pol <= 6; pol++) {
            CHECK(dsref_order(pol, n, tier, arr, bud, Q, w, prio, 0.125, 10.0, pol == 4 ? -INFINITY : 0.0, perm,
                              key) == 0);
            uint8_t *seen = calloc(n ? n : 1, 1);
            for (uint32_t k = 0; k < n; k++) {
                CHECK(perm[k] < n);
                if (perm[k] < n) seen[perm[k]]++;
            }
            for (uint32_t i = 0; i < n; i++) CHECK(seen[i] == 1);
            free(seen);
        }
        CHECK(dsref_order(9, n, tier, arr, bud, Q, w, prio, 0.1, 0.0, 0.0, perm, NULL) != 0 || n == 0);
        if (n) {
            tier[0] = (uint8_t)Q;
            CHECK(dsref_order(0, n, tier, arr, bud, Q, w, prio, 0.1, 0.0, 0.0, perm, NULL) != 0);
        }
        free(tier); free(arr); free(bud); free(key); free(perm);
    }
}

static void simulate_cases(void)
{
    for (int trial = 0; trial < 150; trial++) {
        uint32_t n = rnd(150), G = 1 + rnd(4), ticks = rnd(30), batch = 1 + rnd(8);
        double *arr = malloc(8 * (n ? n : 1)), *tick_t = malloc(8 * (ticks ? ticks : 1)), state[4];
        uint8_t *tier = malloc(n ? n : 1), *cat = malloc(n ? n : 1);
        uint32_t *counts = malloc(4 * (n ? n : 1)), *ten = malloc(4 * (n ? n : 1)), *grp = malloc(4 * (n ? n : 1)),
                 *obs = malloc(4 * (n ? n : 1)), *seq = malloc(4 * (n ? n : 1)), nd = 0;
        int32_t *tick_of = malloc(4 * (n ? n : 1));
        uint32_t w[3] = {4, 2, 1};
        double prio[3] = {0, 1, 2}, tb[4] = {32, 128, 256, 512}, s[3] = {1.25, 1.125, 1.0};
        for (uint32_t i = 0; i < n; i++) {
            arr[i] = (double)rnd(100) * 0.01;
            tier[i] = (uint8_t)rnd(3);
            cat[i] = (uint8_t)rnd(4);
            counts[i] = rnd(600);
            ten[i] = rnd(3);
            grp[i] = rnd(G);
            obs[i] = rnd(900);
        }
        for (uint32_t k = 0; k < ticks; k++) tick_t[k] = 0.05 * (k + 1);
        for (int pol = 0; pol <= 6; pol++) {
            for (uint32_t g = 0; g < G; g++) state[g] = 1.0;
            CHECK(dsref_simulate(pol, n, arr, tier, counts, cat, ten, grp, obs, tb, 4, s, 3, G, 1024.0, 128.0,
                                 512.0, 3, w, prio, 0.01, 0.0, 0.25, batch, tick_t, ticks, state, seq, tick_of,
                                 &nd) == 0);
            CHECK(nd <= n);
        }
        CHECK(dsref_simulate(0, n, arr, tier, counts, cat, ten, grp, obs, tb, 4, s, 3, G, 1024.0, 128.0, 512.0, 3,
                             w, prio, 0.01, 0.0, 0.25, 0, tick_t, ticks, state, seq, tick_of, &nd) != 0);
        free(arr); free(tick_t); free(tier); free(cat); free(counts); free(ten); free(grp); free(obs);
        free(seq); free(tick_of);
    }
}

int main(void)
{
    characterize_cases();
    calibrate_score_cases();
    order_cases();
    simulate_cases();
    if (fails) {
        fprintf(stderr, "%d checks failed\n", fails);
        return 1;
    }
    printf("oracle sanitizer checks: ok\n");
    return 0;
}
