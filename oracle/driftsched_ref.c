/*
 * DriftSched admission hot path: plain single-threaded CPU oracle.
 *
 * TEST INFRASTRUCTURE. Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load or call this library. The product
 * path (the HIP library and its binding) never does; it shares no source,
 * header, table or helper with this file.
 *
 * Every routine here is written to be read against the paper
 * ("DriftSched: Adaptive QoS-Aware Scheduling under Runtime Token Drift for
 * Multi-Tenant GPU Inference"), not to be fast: plain loops, fp64 throughout,
 * built with -ffp-contract=off so that no multiply-add is fused.
 *
 * Functions and the passages they follow:
 *   dsref_count_words      whitespace proxy, Python str.split() semantics
 *                          (Sec. "Workload Characterization and Token Budget
 *                          Estimation"; Sec. "Admission-Time Workload
 *                          Characterization Overhead", tab:tokenizer_overhead)
 *   dsref_characterize     the same, over a packed batch of prompts
 *   dsref_calibrate        EMA update, Eq. (5) with the ratio of Eq. (6)
 *                          (Sec. "Runtime Calibration and Feedback Adaptation")
 *   dsref_score            Eq. (1), Eq. (2) in the order of Alg. 1, Eq. (4)
 *   dsref_order            FIFO, Priority, Weighted, SJF, Aging Priority
 *                          (Sec. "Scheduling Engine" and its subsections)
 *   dsref_calibrate_ex     dsref_calibrate, also recording the factor each
 *                          event's group had just before the event
 *   dsref_error_stats      MAE, RMSE and mean bias of estimates against
 *                          observed lengths (Sec. "Impact of Workload
 *                          Characterization and Runtime Calibration",
 *                          tab:four_mode_token_error, tab:error_reduction)
 *   dsref_class_histogram  runtime classes (Eq. (4)) per semantic category
 *                          (tab:workload_mapping)
 *   dsref_simulate         dispatch ticks of the online loop: order the
 *                          pending set, dispatch a batch, feed its
 *                          completions back (Sec. "Experimental
 *                          Configuration", Sec. "Calibration and Evaluation
 *                          Phases")
 */
#define _GNU_SOURCE
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Whitespace proxy                                                          */
/* ------------------------------------------------------------------------ */

/*
 * The paper counts input words with Python's str.split() (its platform table
 * names Python 3.10.12). With no argument, str.split() separates on the code
 * points for which str.isspace() is true. That set is written out here; the
 * test suite regenerates it from the running Python by enumerating every code
 * point and checks this function against it.
 */
int dsref_is_space(uint32_t cp)
{
    if (cp >= 0x09 && cp <= 0x0D) return 1;   /* TAB LF VT FF CR */
    if (cp >= 0x1C && cp <= 0x20) return 1;   /* FS GS RS US SPACE */
    if (cp == 0x85) return 1;                 /* NEXT LINE */
    if (cp == 0xA0) return 1;                 /* NO-BREAK SPACE */
    if (cp == 0x1680) return 1;               /* OGHAM SPACE MARK */
    if (cp >= 0x2000 && cp <= 0x200A) return 1; /* EN QUAD .. HAIR SPACE */
    if (cp == 0x2028) return 1;               /* LINE SEPARATOR */
    if (cp == 0x2029) return 1;               /* PARAGRAPH SEPARATOR */
    if (cp == 0x202F) return 1;               /* NARROW NO-BREAK SPACE */
    if (cp == 0x205F) return 1;               /* MEDIUM MATHEMATICAL SPACE */
    if (cp == 0x3000) return 1;               /* IDEOGRAPHIC SPACE */
    return 0;
}

static int is_cont(uint8_t b) { return b >= 0x80 && b <= 0xBF; }

/*
 * Decode one well-formed UTF-8 sequence starting at s (avail bytes left),
 * following the Unicode table of well-formed byte sequences. Returns its
 * length and stores the code point, or returns 0 when the bytes at s do not
 * begin a well-formed sequence.
 */
static int decode_one(const uint8_t *s, uint64_t avail, uint32_t *cp)
{
    uint8_t b0 = s[0];
    if (b0 <= 0x7F) { *cp = b0; return 1; }
    if (b0 >= 0xC2 && b0 <= 0xDF) {
        if (avail < 2 || !is_cont(s[1])) return 0;
        *cp = ((uint32_t)(b0 & 0x1F) << 6) | (s[1] & 0x3F);
        return 2;
    }
    if (b0 >= 0xE0 && b0 <= 0xEF) {
        uint8_t lo = 0x80, hi = 0xBF;
        if (b0 == 0xE0) lo = 0xA0;
        if (b0 == 0xED) hi = 0x9F;
        if (avail < 3 || s[1] < lo || s[1] > hi || !is_cont(s[2])) return 0;
        *cp = ((uint32_t)(b0 & 0x0F) << 12) | ((uint32_t)(s[1] & 0x3F) << 6) | (s[2] & 0x3F);
        return 3;
    }
    if (b0 >= 0xF0 && b0 <= 0xF4) {
        uint8_t lo = 0x80, hi = 0xBF;
        if (b0 == 0xF0) lo = 0x90;
        if (b0 == 0xF4) hi = 0x8F;
        if (avail < 4 || s[1] < lo || s[1] > hi || !is_cont(s[2]) || !is_cont(s[3])) return 0;
        *cp = ((uint32_t)(b0 & 0x07) << 18) | ((uint32_t)(s[1] & 0x3F) << 12) |
              ((uint32_t)(s[2] & 0x3F) << 6) | (s[3] & 0x3F);
        return 4;
    }
    return 0;
}

/*
 * Number of items len(prompt.split()) for one prompt of len bytes: the number
 * of maximal runs of non-whitespace characters. The prompt is decoded on its
 * own. A byte that does not start a well-formed sequence is taken as one
 * non-whitespace character, which is what decoding with the surrogateescape
 * error handler does; since every multi-byte whitespace code point begins
 * with a byte that is never a continuation byte, it does not matter for the
 * count how many bytes one decoding error spans.
 */
uint32_t dsref_count_words(const uint8_t *s, uint64_t len)
{
    uint32_t n = 0;
    int in_word = 0;
    uint64_t p = 0;
    while (p < len) {
        uint32_t cp = 0;
        int k = decode_one(s + p, len - p, &cp);
        int space;
        if (k == 0) { space = 0; k = 1; }
        else space = dsref_is_space(cp);
        if (space) {
            in_word = 0;
        } else {
            if (!in_word) n++;
            in_word = 1;
        }
        p += (uint64_t)k;
    }
    return n;
}

/*
 * Stage 1 over a batch: prompt i is text[offsets[i] .. offsets[i+1]).
 * Returns 0, or -1 if the offsets are not nondecreasing or exceed text_bytes.
 */
int dsref_characterize(const uint8_t *text, uint64_t text_bytes,
                       const uint64_t *offsets, uint64_t n, uint32_t *counts)
{
    for (uint64_t i = 0; i < n; i++) {
        uint64_t a = offsets[i], b = offsets[i + 1];
        if (b < a || b > text_bytes) return -1;
        counts[i] = dsref_count_words(text + a, b - a);
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Calibration: Eq. (5) and Eq. (6)                                         */
/* ------------------------------------------------------------------------ */

/*
 * Completion events are taken in array order, which is completion order.
 * For an event of group g with admission estimate est (the B-free estimate
 * T_base*S*F of the request) and observed output length obs:
 *     B_measured = obs / est                       (Eq. 6)
 *     B[g] = (1 - alpha) * B[g] + alpha * B_measured  (Eq. 5)
 * evaluated as t1 = (1-alpha)*B; t2 = alpha*r; B = t1 + t2.
 * An event whose est is not finite or not positive carries no usable ratio
 * and leaves B[g] unchanged. trace[e] (if trace is not NULL) is B[g] after
 * event e. Events whose group is >= n_groups are rejected (return -1).
 */
int dsref_calibrate_ex(const uint32_t *group, const double *est, const uint32_t *obs,
                       uint64_t n_events, double alpha, uint32_t n_groups,
                       double *state, double *trace, double *trace_before)
{
    for (uint64_t e = 0; e < n_events; e++)
        if (group[e] >= n_groups) return -1;
    for (uint64_t e = 0; e < n_events; e++) {
        uint32_t g = group[e];
        double x = est[e];
        if (trace_before) trace_before[e] = state[g];
        if (isfinite(x) && x > 0.0) {
            double r = (double)obs[e] / x;
            double t1 = (1.0 - alpha) * state[g];
            double t2 = alpha * r;
            state[g] = t1 + t2;
        }
        if (trace) trace[e] = state[g];
    }
    return 0;
}

int dsref_calibrate(const uint32_t *group, const double *est, const uint32_t *obs,
                    uint64_t n_events, double alpha, uint32_t n_groups,
                    double *state, double *trace)
{
    return dsref_calibrate_ex(group, est, obs, n_events, alpha, n_groups, state, trace, NULL);
}

/*
 * Estimation error (tab:four_mode_token_error). The estimate of event e is
 * x = est[e] * factor[e] (factor NULL: est[e]); events whose x is not finite
 * and positive are left out, as in the calibration update. With
 * d = x - observed: MAE = mean |d|, RMSE = sqrt(mean d^2), mean bias =
 * mean(observed / x), the ratio that the calibration factor tracks (Eq. (6)).
 * stats[4 g .. 4 g + 3] = count, MAE, RMSE, mean bias of group g, and at
 * g = n_groups the same over all events. Plain sums in event order.
 */
int dsref_error_stats(uint64_t n, const double *est, const double *factor, const uint32_t *obs,
                      const uint32_t *group, uint32_t n_groups, double *stats)
{
    uint64_t slots = (uint64_t)n_groups + 1;
    double *sum = calloc(4 * slots, sizeof(double));
    if (!sum) return -2;
    for (uint64_t e = 0; e < n; e++) {
        if (group && group[e] >= n_groups) { free(sum); return -1; }
    }
    for (uint64_t e = 0; e < n; e++) {
        double x = est[e];
        if (factor) x = x * factor[e];
        if (!(isfinite(x) && x > 0.0)) continue;
        double o = (double)obs[e];
        double d = x - o;
        uint64_t idx[2];
        int m = 0;
        if (group) idx[m++] = group[e];
        idx[m++] = n_groups;
        for (int k = 0; k < m; k++) {
            double *s = sum + 4 * idx[k];
            s[0] += 1.0;
            s[1] += fabs(d);
            s[2] += d * d;
            s[3] += o / x;
        }
    }
    for (uint64_t g = 0; g < slots; g++) {
        double *s = sum + 4 * g;
        stats[4 * g] = s[0];
        if (s[0] > 0.0) {
            stats[4 * g + 1] = s[1] / s[0];
            stats[4 * g + 2] = sqrt(s[2] / s[0]);
            stats[4 * g + 3] = s[3] / s[0];
        } else {
            stats[4 * g + 1] = stats[4 * g + 2] = stats[4 * g + 3] = NAN;
        }
    }
    free(sum);
    return 0;
}

/* hist[c * 3 + k] = number of requests of category c in runtime class k. */
int dsref_class_histogram(uint64_t n, const uint8_t *category, uint32_t n_cat,
                          const uint8_t *job_class, uint32_t *hist)
{
    memset(hist, 0, (size_t)n_cat * 3 * sizeof(uint32_t));
    for (uint64_t i = 0; i < n; i++) {
        if (category[i] >= n_cat || job_class[i] > 2) return -1;
        hist[category[i] * 3u + job_class[i]] += 1;
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Budget and class: Eq. (1), Eq. (2), Alg. 1, Eq. (4)                      */
/* ------------------------------------------------------------------------ */

/*
 * For request i with word count n_i = counts[i], semantic category cat_i,
 * tenant ten_i and calibration group g_i:
 *   F       = 1 + n_i / f_ref                       (prompt complexity factor)
 *   est     = T_base[cat] * B[g] * S[ten] * F       (Eq. 2, left to right as
 *                                                    Alg. 1 gathers them)
 *   est_base= T_base[cat] * S[ten] * F              (the same without B)
 *   budget  = n_i + est                             (Eq. 1)
 *   class   = 0 short if budget <= short_max, 1 medium if <= medium_max,
 *             2 long otherwise                      (Eq. 4)
 * est_base may be NULL. group may be NULL: then state holds one factor per
 * request (state[i] scores request i, n_groups = n), the factor its group
 * had when the request was admitted (as-of scoring; the paper's updated
 * factors serve the estimates that follow them, Sec. "Runtime Calibration
 * and Feedback Adaptation"). Returns -1 if an index is out of range.
 */
int dsref_score(uint64_t n, const uint32_t *counts, const uint8_t *category,
                const uint32_t *tenant, const uint32_t *group,
                const double *t_base, uint32_t n_cat,
                const double *s_tenant, uint32_t n_tenants,
                const double *state, uint32_t n_groups,
                double f_ref, double short_max, double medium_max,
                double *est_base, double *est, double *budget, uint8_t *job_class)
{
    if (!group && n_groups != n) return -1;
    for (uint64_t i = 0; i < n; i++) {
        uint64_t g = group ? group[i] : i;   /* no groups: request i's own factor */
        if (category[i] >= n_cat || tenant[i] >= n_tenants || g >= n_groups)
            return -1;
        double words = (double)counts[i];
        double F = 1.0 + words / f_ref;
        double tb = t_base[category[i]];
        double s = s_tenant[tenant[i]];
        double b = state[g];
        double e = tb * b;
        e = e * s;
        e = e * F;
        if (est_base) {
            double e0 = tb * s;
            e0 = e0 * F;
            est_base[i] = e0;
        }
        est[i] = e;
        double total = words + e;
        budget[i] = total;
        uint8_t c;
        if (total <= short_max) c = 0;
        else if (total <= medium_max) c = 1;
        else c = 2;
        job_class[i] = c;
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Dispatch orders                                                           */
/* ------------------------------------------------------------------------ */

enum { REF_FIFO = 0, REF_PRIORITY = 1, REF_WEIGHTED = 2, REF_SJF = 3, REF_AGING = 4,
       REF_WEIGHTED_SMOOTH = 5, REF_WEIGHTED_STRIDE = 6 };

/* Sort context: primary key (may be NULL), then arrival, then index. */
struct sort_ctx {
    const double *primary;
    const double *arrival;
};

static int cmp_req(const void *pa, const void *pb, void *vctx)
{
    const struct sort_ctx *c = (const struct sort_ctx *)vctx;
    uint32_t a = *(const uint32_t *)pa, b = *(const uint32_t *)pb;
    if (c->primary) {
        if (c->primary[a] < c->primary[b]) return -1;
        if (c->primary[a] > c->primary[b]) return 1;
    }
    if (c->arrival[a] < c->arrival[b]) return -1;
    if (c->arrival[a] > c->arrival[b]) return 1;
    if (a < b) return -1;
    if (a > b) return 1;
    return 0;
}

static void sort_requests(uint32_t *perm, uint32_t n, const double *primary,
                          const double *arrival)
{
    struct sort_ctx c = { primary, arrival };
    for (uint32_t i = 0; i < n; i++) perm[i] = i;
    qsort_r(perm, n, sizeof(uint32_t), cmp_req, &c);
}

/*
 * Dispatch order of n pending requests under one policy. perm[k] is the
 * request dispatched k-th. key (optional) receives each request's primary
 * key under the policy. Every policy ends ties in arrival order, and equal
 * arrivals by lower request index (FIFO within a tier, Sec. "Priority
 * Scheduling").
 *
 *  FIFO      arrival order (Sec. "FIFO Scheduling"). key = arrival.
 *  Priority  requests taken from the highest-priority non-empty tier queue,
 *            FIFO within a tier: the exact order of the score
 *            priority*10^12 + arrival of Sec. "Priority Scheduling", with a
 *            lower tier_priority value served first (Premium = 0).
 *            key = tier_priority[tier].
 *  Weighted  a cyclic dispatcher over the tier queues (Sec. "Weighted
 *            Scheduling"): each round serves up to weight[q] requests from
 *            queue q, q = 0, 1, ..., in FIFO order; an empty queue is passed
 *            over. key = the round in which the request is served.
 *  SJF       lower estimated budget first (Sec. "Shortest-Job-First
 *            Scheduling"). key = budget.
 *  Aging     effective score e = max(floor, p - rate * max(0, t_now - a)),
 *            lower first, where p = tier_priority[tier] and a = arrival:
 *            waiting lowers the score (Sec. "Aging Priority Scheduling").
 *            key = e.
 *  Weighted, smooth (policy 5; a reading of the same section: the paper
 *            fixes the ratio and the cyclic dispatch, not how the tiers
 *            interleave inside a cycle): the smooth weighted round robin.
 *            Every queue holds a credit, 0 at the start. Before each
 *            dispatch every non-empty queue's credit grows by its weight;
 *            the queue with the largest credit (the lowest tier on ties)
 *            dispatches its head and gives up the sum of the weights of the
 *            non-empty queues. When a queue runs empty it leaves; the other
 *            queues keep their credits (the published smooth weighted round
 *            robin, which passes over an unavailable peer).
 *            key = floor(k / weight) for the k-th request of its tier, as
 *            for Weighted.
 *  Weighted, stride (policy 6; another reading of the same section):
 *            stride scheduling. Queue q advances its pass by the stride
 *            1 / weight[q], starting from one stride; the non-empty queue
 *            with the smallest pass (the lowest tier on ties) dispatches its
 *            head and advances. Passes are compared exactly, as the
 *            fractions they are (no fixed-point stride). key as for
 *            Weighted.
 * Returns -1 on a tier >= n_tiers, a zero weight or an unknown policy.
 */
int dsref_order(int policy, uint32_t n, const uint8_t *tier, const double *arrival,
                const double *budget, uint32_t n_tiers, const uint32_t *weight,
                const double *tier_priority, double aging_rate, double t_now,
                double aging_floor, uint32_t *perm, double *key)
{
    for (uint32_t i = 0; i < n; i++)
        if (tier[i] >= n_tiers) return -1;
    if (policy == REF_FIFO) {
        sort_requests(perm, n, NULL, arrival);
        if (key) for (uint32_t i = 0; i < n; i++) key[i] = arrival[i];
        return 0;
    }
    if (policy == REF_PRIORITY) {
        double *p = (double *)malloc(sizeof(double) * (n ? n : 1));
        for (uint32_t i = 0; i < n; i++) p[i] = tier_priority[tier[i]];
        sort_requests(perm, n, p, arrival);
        if (key) memcpy(key, p, sizeof(double) * n);
        free(p);
        return 0;
    }
    if (policy == REF_SJF) {
        sort_requests(perm, n, budget, arrival);
        if (key) for (uint32_t i = 0; i < n; i++) key[i] = budget[i];
        return 0;
    }
    if (policy == REF_AGING) {
        double *e = (double *)malloc(sizeof(double) * (n ? n : 1));
        for (uint32_t i = 0; i < n; i++) {
            double w = t_now - arrival[i];
            if (w < 0.0) w = 0.0;
            double d = aging_rate * w;
            double v = tier_priority[tier[i]] - d;
            if (v < aging_floor) v = aging_floor;
            e[i] = v;
        }
        sort_requests(perm, n, e, arrival);
        if (key) memcpy(key, e, sizeof(double) * n);
        free(e);
        return 0;
    }
    if (policy == REF_WEIGHTED || policy == REF_WEIGHTED_SMOOTH || policy == REF_WEIGHTED_STRIDE) {
        for (uint32_t q = 0; q < n_tiers; q++)
            if (weight[q] == 0) return -1;
        /* tier queues in FIFO order */
        uint32_t *fifo = (uint32_t *)malloc(sizeof(uint32_t) * (n ? n : 1));
        sort_requests(fifo, n, NULL, arrival);
        uint32_t *len = (uint32_t *)calloc(n_tiers, sizeof(uint32_t));
        uint32_t *start = (uint32_t *)calloc(n_tiers, sizeof(uint32_t));
        uint32_t *head = (uint32_t *)calloc(n_tiers, sizeof(uint32_t));
        uint32_t *queue = (uint32_t *)malloc(sizeof(uint32_t) * (n ? n : 1));
        for (uint32_t k = 0; k < n; k++) len[tier[fifo[k]]]++;
        for (uint32_t q = 1; q < n_tiers; q++) start[q] = start[q - 1] + len[q - 1];
        for (uint32_t k = 0; k < n; k++) {
            uint32_t i = fifo[k], q = tier[i];
            queue[start[q] + head[q]++] = i;
        }
        memset(head, 0, sizeof(uint32_t) * n_tiers);
        uint32_t pos = 0;
        if (policy == REF_WEIGHTED_SMOOTH) {
            long long *credit = (long long *)calloc(n_tiers, sizeof(long long));
            while (pos < n) {
                long long total = 0;
                for (uint32_t q = 0; q < n_tiers; q++)
                    if (head[q] < len[q]) total += weight[q];
                int best = -1;
                for (uint32_t q = 0; q < n_tiers; q++) {
                    if (head[q] >= len[q]) continue;
                    credit[q] += weight[q];
                    if (best < 0 || credit[q] > credit[best]) best = (int)q;
                }
                credit[best] -= total;
                uint32_t i = queue[start[best] + head[best]];
                perm[pos++] = i;
                if (key) key[i] = (double)(head[best] / weight[best]);
                head[best]++;
                /* a queue that runs empty leaves; the others keep their credits */
            }
            free(credit);
            free(fifo); free(len); free(start); free(head); free(queue);
            return 0;
        }
        if (policy == REF_WEIGHTED_STRIDE) {
            while (pos < n) {
                /* the pass of queue q is (head[q] + 1) / weight[q]: compare
                   a / w_a < b / w_b as a w_b < b w_a (below 2^62) */
                int best = -1;
                for (uint32_t q = 0; q < n_tiers; q++) {
                    if (head[q] >= len[q]) continue;
                    if (best < 0 || (uint64_t)(head[q] + 1) * weight[best] <
                                        (uint64_t)(head[best] + 1) * weight[q])
                        best = (int)q;
                }
                uint32_t i = queue[start[best] + head[best]];
                perm[pos++] = i;
                if (key) key[i] = (double)(head[best] / weight[best]);
                head[best]++;
            }
            free(fifo); free(len); free(start); free(head); free(queue);
            return 0;
        }
        double round = 0.0;
        while (pos < n) {
            for (uint32_t q = 0; q < n_tiers; q++) {
                uint32_t take = 0;
                while (take < weight[q] && head[q] < len[q]) {
                    uint32_t i = queue[start[q] + head[q]];
                    perm[pos++] = i;
                    if (key) key[i] = round;
                    head[q]++;
                    take++;
                }
            }
            round += 1.0;
        }
        free(fifo); free(len); free(start); free(head); free(queue);
        return 0;
    }
    return -1;
}

/* ------------------------------------------------------------------------ */
/* Dispatch ticks: the online loop                                           */
/* ------------------------------------------------------------------------ */

/*
 * The scheduler dispatches pending requests in batches (Sec. "Experimental
 * Configuration": batch size 32) and keeps adapting its estimates as
 * requests complete (Sec. "Calibration and Evaluation Phases"; Sec.
 * "Runtime Calibration and Feedback Adaptation"). At tick k, with time
 * tick_t[k]:
 *   1. the pending set is every request with arrival <= tick_t[k] that has
 *      not been dispatched, taken in index order;
 *   2. it is ordered by dsref_order under the policy, on the pending
 *      requests alone: SJF with budgets scored (dsref_score) from the
 *      factors as they stand, Aging with t_now = tick_t[k], Weighted with a
 *      fresh round-robin cycle over the pending tier queues;
 *   3. the first min(batch, pending) requests of that order are dispatched;
 *   4. their completions, in dispatch order, update the factors with
 *      dsref_calibrate: group[i], the B-free estimate est_base[i] of
 *      dsref_score, observed[i].
 * seq[d] = the request dispatched d-th (0xFFFFFFFF past the last one),
 * tick_of[i] = the tick that dispatched request i (-1 if none), and
 * *n_dispatched the number dispatched. state (n_groups) is updated in place.
 * Returns -1 on an out-of-range index, a zero weight or batch == 0.
 */
int dsref_simulate(int policy, uint32_t n, const double *arrival, const uint8_t *tier,
                   const uint32_t *counts, const uint8_t *category, const uint32_t *tenant,
                   const uint32_t *group, const uint32_t *observed,
                   const double *t_base, uint32_t n_cat, const double *s_tenant,
                   uint32_t n_tenants, uint32_t n_groups,
                   double f_ref, double short_max, double medium_max,
                   uint32_t n_tiers, const uint32_t *weight, const double *tier_priority,
                   double aging_rate, double aging_floor, double alpha, uint32_t batch,
                   const double *tick_t, uint32_t n_ticks, double *state,
                   uint32_t *seq, int32_t *tick_of, uint32_t *n_dispatched)
{
    if (batch == 0) return -1;
    uint32_t m = n ? n : 1;
    double *est_base = (double *)malloc(sizeof(double) * m);
    double *est = (double *)malloc(sizeof(double) * m);
    double *budget = (double *)malloc(sizeof(double) * m);
    uint8_t *cls = (uint8_t *)malloc(m);
    uint8_t *done = (uint8_t *)calloc(m, 1);
    uint32_t *pend = (uint32_t *)malloc(sizeof(uint32_t) * m);
    uint8_t *p_tier = (uint8_t *)malloc(m);
    double *p_arrival = (double *)malloc(sizeof(double) * m);
    double *p_budget = (double *)malloc(sizeof(double) * m);
    uint32_t *perm = (uint32_t *)malloc(sizeof(uint32_t) * m);
    uint32_t *ev_group = (uint32_t *)malloc(sizeof(uint32_t) * m);
    uint32_t *ev_obs = (uint32_t *)malloc(sizeof(uint32_t) * m);
    double *ev_est = (double *)malloc(sizeof(double) * m);
    int rc = dsref_score(n, counts, category, tenant, group, t_base, n_cat, s_tenant, n_tenants,
                         state, n_groups, f_ref, short_max, medium_max, est_base, est, budget, cls);
    for (uint32_t i = 0; i < n; i++) {
        seq[i] = 0xFFFFFFFFu;
        tick_of[i] = -1;
    }
    uint32_t total = 0;
    for (uint32_t k = 0; rc == 0 && k < n_ticks; k++) {
        double t = tick_t[k];
        uint32_t np = 0;
        for (uint32_t i = 0; i < n; i++)
            if (arrival[i] <= t && !done[i]) pend[np++] = i;
        if (policy == REF_SJF)
            rc = dsref_score(n, counts, category, tenant, group, t_base, n_cat, s_tenant,
                             n_tenants, state, n_groups, f_ref, short_max, medium_max, NULL, est,
                             budget, cls);
        for (uint32_t j = 0; j < np; j++) {
            p_tier[j] = tier[pend[j]];
            p_arrival[j] = arrival[pend[j]];
            p_budget[j] = budget[pend[j]];
        }
        if (rc == 0)
            rc = dsref_order(policy, np, p_tier, p_arrival, p_budget, n_tiers, weight,
                             tier_priority, aging_rate, t, aging_floor, perm, NULL);
        if (rc != 0) break;
        uint32_t take = np < batch ? np : batch;
        for (uint32_t j = 0; j < take; j++) {
            uint32_t i = pend[perm[j]];
            done[i] = 1;
            seq[total++] = i;
            tick_of[i] = (int32_t)k;
            ev_group[j] = group[i];
            ev_est[j] = est_base[i];
            ev_obs[j] = observed[i];
        }
        /* their completions, in dispatch order */
        rc = dsref_calibrate(ev_group, ev_est, ev_obs, take, alpha, n_groups, state, NULL);
    }
    *n_dispatched = total;
    free(est_base); free(est); free(budget); free(cls); free(done); free(pend);
    free(p_tier); free(p_arrival); free(p_budget); free(perm);
    free(ev_group); free(ev_obs); free(ev_est);
    return rc;
}
