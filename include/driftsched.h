/*
 * driftsched.h - C ABI of the DriftSched admission hot path on AMD Instinct
 * MI355X (gfx950).
 *
 * The paper ("DriftSched: Adaptive QoS-Aware Scheduling under Runtime Token
 * Drift for Multi-Tenant GPU Inference") admits each request by estimating
 * its token budget from its prompt, folds completed requests' observed
 * output lengths into calibration factors, classifies the request, and
 * dispatches it under one of five policies. This library runs those steps
 * over a whole batch of pending requests on one GPU:
 *
 *   ds_characterize   word counts of the prompts (whitespace proxy)
 *   ds_calibrate      EMA calibration factors from completion events
 *   ds_score          calibrated output estimate, budget and runtime class
 *   ds_order          dispatch permutation for one policy
 *
 * and, beside it, the diagnostics of the paper's evaluation:
 *
 *   ds_calibrate_ex     calibration with the factor before each event
 *   ds_error_stats      MAE, RMSE and mean bias of estimates vs observed
 *   ds_class_histogram  runtime classes per semantic category
 *
 * and the online loop that ties the stages together:
 *
 *   ds_simulate         dispatch ticks: order the pending set, dispatch a
 *                       batch, feed its completions back into the factors
 *   ds_simulate_multi   several such loops (e.g. the five policies) in one launch
 *
 * and one measurement aid:
 *
 *   ds_read_bandwidth   the read side of ds_characterize alone
 *
 * Conventions shared by every entry point:
 *  - Array arguments are DEVICE pointers (memory from hipMalloc or any
 *    allocator of the same device, e.g. torch tensors); parameter structs
 *    are HOST pointers, read during the call only.
 *  - The caller owns every buffer. The library never allocates or frees
 *    device memory and keeps no state between calls. Scratch memory is a
 *    caller-provided workspace of at least ds_workspace_bytes() bytes,
 *    256-byte aligned; its contents need no initialisation and are
 *    undefined after the call. Calls that may run at the same time (on
 *    different streams) need workspaces of their own.
 *  - Work is enqueued on `stream` (a hipStream_t; NULL is the null stream)
 *    and the call returns without waiting, except with DS_VALIDATE, where
 *    it waits for the stream to report data errors.
 *  - Host-checkable errors (NULL pointers, sizes, parameter ranges, a short
 *    workspace) are returned before anything is enqueued. A launch failure
 *    returns DS_ERR_HIP. Without DS_VALIDATE, device data that break a
 *    stated contract give unspecified results but never out-of-bounds
 *    memory accesses.
 *  - n == 0 is valid and enqueues nothing.
 *  - No C++ exception crosses this interface.
 */
#ifndef DRIFTSCHED_H
#define DRIFTSCHED_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DS_OK = 0,
    DS_ERR_NULL = -1,       /* a required pointer is NULL */
    DS_ERR_ARG = -2,        /* a scalar argument or parameter is out of range */
    DS_ERR_SIZE = -3,       /* a count exceeds the supported maximum */
    DS_ERR_WORKSPACE = -4,  /* workspace NULL, misaligned or smaller than required */
    DS_ERR_DATA = -5,       /* DS_VALIDATE found device data breaking the contract */
    DS_ERR_HIP = -6,        /* the HIP runtime reported an error */
    DS_ERR_ALIGN = -7,      /* an array pointer is not aligned as required */
    DS_ERR_WAIT = -8        /* a bounded device-side wait ran out (DS_VALIDATE): the
                               call's results are invalid */
} ds_status;

typedef enum {
    DS_FIFO = 0,            /* arrival order */
    DS_PRIORITY = 1,        /* tier priority first, FIFO within equal priority */
    DS_WEIGHTED = 2,        /* cyclic weighted round robin over tier queues */
    DS_SJF = 3,             /* smaller budget first */
    DS_AGING = 4            /* aged priority, smaller first */
} ds_policy;

typedef enum {
    DS_OP_CHARACTERIZE = 0,
    DS_OP_CALIBRATE = 1,
    DS_OP_SCORE = 2,
    DS_OP_ORDER = 3,
    DS_OP_ORDER_MULTI = 4,
    DS_OP_ERROR_STATS = 5,
    DS_OP_CLASS_HIST = 6,
    DS_OP_SIMULATE = 7,
    DS_OP_SIMULATE_MULTI = 8   /* third argument of ds_workspace_bytes: the number of runs */
} ds_op;

/* flags */
#define DS_VALIDATE 1u      /* check device data, wait, and report DS_ERR_DATA */
#define DS_SERIAL_SORT 2u   /* ds_order, ds_order_multi: up to 2^18 requests, run the
                               single-workgroup sort that is otherwise the fallback of
                               an overflowing sample-sort bucket (diagnostic; slow) */
#define DS_NO_WAIT 4u       /* diagnostic of the error path below: every bounded
                               device-side wait gives up at once, as if it had run out */

/*
 * Bounded waits. The sorts behind ds_order, ds_order_multi, ds_calibrate
 * (above 4096 groups) and ds_simulate split their work into tiles that wait,
 * each for at most about 0.2 s, on counts published by tiles of smaller
 * index (decoupled look-back); the orders of more than 2^18 and at most
 * 2^20 requests have no such waits. ds_calibrate of at most 64 chunks of
 * 512, 1024 or 2048 events (and at most 16384 chunk-group pairs) runs in one
 * launch whose chunks wait the same way for the maps of the chunks before
 * them. In normal operation no wait runs out (a tile waits only on tiles
 * that have already started and publish before they wait). If one does:
 *  - in a sample-sort scatter (up to 2^18 requests), the call finishes on
 *    the single-workgroup path instead, with exact results;
 *  - anywhere else the results are invalid, and the call's status word is
 *    set: the uint32 at byte DS_WS_STATUS_OFFSET of the workspace, zeroed by
 *    the call's first kernel. With DS_VALIDATE the call waits for its work
 *    and returns DS_ERR_WAIT; without it, the word is left for the caller
 *    (read it after the stream has completed the call).
 */
#define DS_WS_STATUS_OFFSET 4

#define DS_MAX_TIERS 16
#define DS_MAX_ITEMS (1u << 30)   /* max events for ds_calibrate, requests for ds_order */
#define DS_MAX_GROUPS (1u << 20)  /* max groups for ds_error_stats */
#define DS_MAX_BATCH 1024         /* max requests per dispatch tick for ds_simulate */

typedef void *ds_stream;    /* hipStream_t */

/* Parameters of the budget estimate (Eq. 2) and the classes (Eq. 4). */
typedef struct {
    double f_ref;           /* prompt-complexity factor F = 1 + n / f_ref; > 0 */
    double short_max;       /* budget <= short_max is short (128 in the paper) */
    double medium_max;      /* budget <= medium_max is medium (512 in the paper) */
} ds_score_params;

/* Parameters of the dispatch policies. */
typedef struct {
    uint32_t n_tiers;                    /* 1..DS_MAX_TIERS; tier values < n_tiers */
    uint32_t weight[DS_MAX_TIERS];       /* DS_WEIGHTED: requests per round, >= 1 */
    double tier_priority[DS_MAX_TIERS];  /* DS_PRIORITY/DS_AGING: smaller first; finite */
    double aging_rate;                   /* DS_AGING: priority units per second, >= 0 */
    double t_now;                        /* DS_AGING: current time (same clock as arrival) */
    double aging_floor;                  /* DS_AGING: lower clamp of the aged score (may be -inf) */
    uint32_t weighted_mode;              /* DS_WEIGHTED: DS_WRR_BLOCKED, _SMOOTH or _STRIDE */
} ds_order_params;

/* ds_order_params.weighted_mode: how the tiers interleave inside a cycle */
#define DS_WRR_BLOCKED 0u                /* each tier's share of a round in one block */
#define DS_WRR_SMOOTH 1u                 /* smooth interleaving; weights sum to at most
                                            DS_WRR_MAX_WEIGHT_SUM */
#define DS_WRR_STRIDE 2u                 /* stride scheduling */
#define DS_WRR_MAX_WEIGHT_SUM 1024u

/*
 * Stage 1: whitespace-proxy word counts (Sec. "Workload Characterization and
 * Token Budget Estimation"; the split() column of tab:tokenizer_overhead).
 *
 * counts[i] = len(p.decode('utf-8', 'surrogateescape').split()) for prompt
 * p = text[offsets[i] .. offsets[i+1]), i < n: the number of maximal runs of
 * characters that are not among the 29 code points Python's str.split()
 * separates on (ASCII 09-0D, 1C-20; U+0085, U+00A0, U+1680, U+2000-200A,
 * U+2028, U+2029, U+202F, U+205F, U+3000). Each prompt is decoded on its own;
 * an undecodable byte counts as a non-space character.
 *
 *  text       device, text_bytes bytes, 16-byte aligned; read-only
 *  text_bytes size of the text buffer; the kernels read exactly [0, text_bytes)
 *  offsets    device, n+1 uint64; contract: nondecreasing, offsets[n] <= text_bytes
 *  n          number of prompts (< 2^32 - 1)
 *  counts     device, n uint32; written
 *  ws         workspace of ds_workspace_bytes(DS_OP_CHARACTERIZE, n, 0) bytes
 */
ds_status ds_characterize(const uint8_t *text, uint64_t text_bytes,
                          const uint64_t *offsets, uint32_t n, uint32_t *counts,
                          void *ws, size_t ws_bytes, uint32_t flags, ds_stream stream);

/*
 * Stages 1 and 3 in one pass: the results of ds_characterize followed by
 * ds_score on its counts, bit for bit, with each request scored as soon as
 * its count is known (no second launch, no second read of the counts).
 * Arguments as in those two calls (the counts are written as by
 * ds_characterize; state, if calibrated in the same step, must be final
 * before this call). Workspace: ds_workspace_bytes(DS_OP_CHARACTERIZE, n, 0).
 * Errors: those of either call; with DS_VALIDATE both calls' checks run.
 */
ds_status ds_characterize_score(const uint8_t *text, uint64_t text_bytes,
                                const uint64_t *offsets, uint32_t n, uint32_t *counts,
                                const uint8_t *category, const uint32_t *tenant,
                                const uint32_t *group, const double *t_base, uint32_t n_cat,
                                const double *s_tenant, uint32_t n_tenants,
                                const double *state, uint32_t n_groups,
                                const ds_score_params *params, double *est_base, double *est,
                                double *budget, uint8_t *job_class, void *ws, size_t ws_bytes,
                                uint32_t flags, ds_stream stream);

/*
 * ds_characterize_score for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation. It takes no workspace: its scratch memory is a static device
 * array of the library, DS_NOALLOC_SCRATCH_BYTES on each GPU it runs on, held
 * from the library's load until the process ends. The call itself allocates
 * and frees nothing (its first call on a GPU looks up that GPU's copy of the
 * array, once).
 *
 *  n          <= DS_NOALLOC_MAX_PROMPTS (else DS_ERR_SIZE)
 *  flags      0 (else DS_ERR_ARG: DS_VALIDATE waits and copies to the host)
 * Other arguments, results and errors as ds_characterize_score.
 * Every call on one GPU uses that GPU's one array and leaves its contents
 * behind (nothing in it needs clearing between calls): calls that overlap on
 * one GPU (on two streams, or from host threads without ordering) race and
 * give undefined results.
 */
#define DS_NOALLOC_MAX_PROMPTS (1u << 20)
#define DS_NOALLOC_SCRATCH_BYTES 4456960u
ds_status ds_characterize_score_noalloc(const uint8_t *text, uint64_t text_bytes,
                                        const uint64_t *offsets, uint32_t n, uint32_t *counts,
                                        const uint8_t *category, const uint32_t *tenant,
                                        const uint32_t *group, const double *t_base, uint32_t n_cat,
                                        const double *s_tenant, uint32_t n_tenants,
                                        const double *state, uint32_t n_groups,
                                        const ds_score_params *params, double *est_base, double *est,
                                        double *budget, uint8_t *job_class, uint32_t flags,
                                        ds_stream stream);

/*
 * Stage 2: calibration factors, Eq. (5) with the ratio of Eq. (6)
 * (Sec. "Runtime Calibration and Feedback Adaptation").
 *
 * Events are in completion order. For each event e with est[e] finite and
 * > 0, in that order, the factor of its group g = group[e] is updated
 *     state[g] <- (1 - alpha) * state[g] + alpha * (observed[e] / est[e]);
 * other events leave it unchanged. trace[e] receives state[g] after event e.
 * The GPU evaluates the recurrence as a parallel scan over the affine maps
 * x -> a x + b, so results match the sequential evaluation up to rounding
 * (relative differences of order 1e-15; the contract is 1e-12).
 *
 *  group      device, n_events uint32; contract: < n_groups
 *  est        device, n_events double: the B-free admission estimate
 *             T_base * S_tenant * F_input of the completed request
 *  observed   device, n_events uint32: observed output tokens
 *  n_events   <= DS_MAX_ITEMS
 *  alpha      EMA rate, 0 <= alpha <= 1
 *  n_groups   number of calibration groups (>= 1)
 *  state      device, n_groups double; in: factors before the events (1.0
 *             initially), out: after. Groups without events are unchanged.
 *  trace      device, n_events double, or NULL
 *  ws         workspace of ds_workspace_bytes(DS_OP_CALIBRATE, n_events, n_groups)
 */
ds_status ds_calibrate(const uint32_t *group, const double *est, const uint32_t *observed,
                       uint64_t n_events, double alpha, uint32_t n_groups,
                       double *state, double *trace,
                       void *ws, size_t ws_bytes, uint32_t flags, ds_stream stream);

/*
 * Stage 3: budget and class, Eq. (1), Eq. (2) in the order of Alg. 1, Eq. (4)
 * (Sec. "Workload Characterization and Token Budget Estimation" and
 * "Workload Classification"). For request i, with n_i = counts[i]:
 *     F         = 1 + n_i / f_ref
 *     est[i]    = ((t_base[category[i]] * state[group[i]]) * s_tenant[tenant[i]]) * F
 *     est_base  = (t_base[category[i]] * s_tenant[tenant[i]]) * F
 *     budget[i] = n_i + est[i]
 *     class[i]  = 0 if budget <= short_max, 1 if <= medium_max, else 2
 * in IEEE double with no fused multiply-add, so results are bit-identical to
 * any plain evaluation in that order.
 *
 *  counts, category, tenant, group   device, n entries; contract: indices in range
 *  t_base     device, n_cat double (baseline estimate per semantic category)
 *  s_tenant   device, n_tenants double (tenant safety scaling)
 *  state      device, n_groups double (calibration factors, e.g. from ds_calibrate)
 *  group      may be NULL: state then holds one factor per request (state[i]
 *             scores request i; n_groups must be n, else DS_ERR_ARG). This is
 *             as-of scoring: each request with the factor its group had when
 *             it was admitted (Sec. "Runtime Calibration and Feedback
 *             Adaptation": the updated factors serve later estimates), e.g.
 *             trace_before of ds_calibrate_ex gathered to the requests'
 *             positions. Calibration keyed by semantic category (the paper's
 *             workload-specific factor) is group = category.
 *  est_base   device, n double, or NULL
 *  est, budget device, n double; job_class device, n uint8
 *  params     host; f_ref > 0
 *  ws         workspace of ds_workspace_bytes(DS_OP_SCORE, n, 0) bytes (used
 *             by DS_VALIDATE only; may be NULL without that flag)
 * Out-of-range indices (without DS_VALIDATE) give NaN estimates and class 2.
 */
ds_status ds_score(uint32_t n, const uint32_t *counts, const uint8_t *category,
                   const uint32_t *tenant, const uint32_t *group,
                   const double *t_base, uint32_t n_cat,
                   const double *s_tenant, uint32_t n_tenants,
                   const double *state, uint32_t n_groups,
                   const ds_score_params *params,
                   double *est_base, double *est, double *budget, uint8_t *job_class,
                   void *ws, size_t ws_bytes, uint32_t flags, ds_stream stream);

/*
 * Stage 4: dispatch order of one policy (Sec. "Scheduling Engine").
 * perm[k] is the index of the request dispatched k-th. Every policy breaks
 * ties by FIFO rank: arrival, then lower request index (-0.0 equals +0.0).
 *
 *  DS_FIFO      key (arrival, index)                   (Sec. "FIFO Scheduling")
 *  DS_PRIORITY  key (tier_priority[tier], FIFO rank): the exact order of the
 *               score priority * 10^12 + arrival       (Sec. "Priority Scheduling")
 *  DS_WEIGHTED  cyclic weighted round robin over the tier queues (Sec.
 *               "Weighted Scheduling"). The paper fixes the ratio w_q and the
 *               cyclic service; params->weighted_mode picks how the tiers
 *               interleave inside a cycle:
 *               DS_WRR_BLOCKED  round r serves, for q = 0, 1, ..., the
 *                 requests of tier q with FIFO rank within the tier in
 *                 [r w_q, (r+1) w_q); empty queues are passed over
 *               DS_WRR_SMOOTH  smooth weighted round robin: before each
 *                 dispatch every non-empty queue's credit grows by w_q; the
 *                 largest credit (lowest tier on ties) is served and gives
 *                 up W, the sum of the non-empty queues' weights; credits
 *                 start at 0, and a queue that runs empty leaves while the
 *                 others keep their credits. Sum of the weights <=
 *                 DS_WRR_MAX_WEIGHT_SUM (else DS_ERR_ARG)
 *               DS_WRR_STRIDE  stride scheduling: the k-th request of tier q
 *                 (FIFO rank within the tier) has pass (k+1) / w_q, compared
 *                 exactly; smaller pass first, equal passes by lower tier
 *               key: floor(k / w_q) for the k-th request of tier q in every mode
 *  DS_SJF       key (budget, FIFO rank)                (Sec. "Shortest-Job-First Scheduling")
 *  DS_AGING     key (e, FIFO rank), e = max(aging_floor,
 *               tier_priority[tier] - aging_rate * max(0, t_now - arrival))
 *                                                      (Sec. "Aging Priority Scheduling")
 *
 *  tier       device, n uint8; contract: < params->n_tiers
 *  arrival    device, n double; contract: not NaN
 *  budget     device, n double (DS_SJF only; else may be NULL); contract: not NaN
 *  fifo_in    device, n uint32, or NULL. When given it must be the DS_FIFO
 *             permutation of the same arrival array (e.g. a previous DS_FIFO
 *             call's perm); the FIFO sort is then skipped.
 *  perm       device, n uint32; written
 *  key        device, n double, or NULL: each request's primary key (arrival,
 *             tier_priority, round number, budget, or e)
 *  n          <= DS_MAX_ITEMS
 *  ws         workspace of ds_workspace_bytes(DS_OP_ORDER, n, 0) bytes
 */
ds_status ds_order(ds_policy policy, uint32_t n, const uint8_t *tier, const double *arrival,
                   const double *budget, const uint32_t *fifo_in,
                   const ds_order_params *params, uint32_t *perm, double *key,
                   void *ws, size_t ws_bytes, uint32_t flags, ds_stream stream);

/*
 * Stage 4 for several policies in one call: the FIFO permutation is computed
 * once (or taken from fifo_in) and the requested policy sorts run together,
 * sharing kernel launches. Results are identical to separate ds_order calls.
 *
 *  policy_mask  bit p set: produce the order of policy p (ds_policy values);
 *               non-zero, at most 0x1F
 *  perms        HOST array of 5 device pointers; perms[p] (n uint32) must be
 *               non-NULL for every requested p, others are ignored
 *  keys         HOST array of 5 device pointers (n double each, or NULL
 *               entries), or NULL for no keys
 *  budget       required when DS_SJF is requested
 *  ws           workspace of ds_workspace_bytes(DS_OP_ORDER_MULTI, n, 0) bytes
 * Other arguments and errors as ds_order.
 */
ds_status ds_order_multi(uint32_t policy_mask, uint32_t n, const uint8_t *tier,
                         const double *arrival, const double *budget, const uint32_t *fifo_in,
                         const ds_order_params *params, uint32_t *const *perms,
                         double *const *keys, void *ws, size_t ws_bytes, uint32_t flags,
                         ds_stream stream);

/*
 * ds_calibrate, and in addition trace_before[e]: the factor of e's group just
 * before event e, i.e. the factor a request admitted at that point of the
 * completion stream is scored with (the admission-time factor of Sec.
 * "Runtime Calibration and Feedback Adaptation"). Either trace may be NULL.
 * Same workspace (DS_OP_CALIBRATE), arguments and errors as ds_calibrate.
 */
ds_status ds_calibrate_ex(const uint32_t *group, const double *est, const uint32_t *observed,
                          uint64_t n_events, double alpha, uint32_t n_groups,
                          double *state, double *trace, double *trace_before,
                          void *ws, size_t ws_bytes, uint32_t flags, ds_stream stream);

/*
 * Estimation error of token estimates against observed output lengths: the
 * MAE, RMSE and mean bias of Sec. "Impact of Workload Characterization and
 * Runtime Calibration" (tab:four_mode_token_error; their BIAS=OFF / BIAS=ON
 * ratio per policy is tab:error_reduction).
 *
 * For every event e whose estimate x = est[e] * factor[e] (factor NULL: 1)
 * is finite and > 0 (other events are skipped), d = x - observed[e]. For
 * each group g < n_groups (the events with group[e] == g) and then for all
 * events together, stats receives four doubles:
 *     count, MAE = mean |d|, RMSE = sqrt(mean d^2), mean bias = mean(observed / x).
 * A set without events gives count 0 and NaN for the three means.
 *
 *  est        device, n double: e.g. the B-free estimate (BIAS=OFF)
 *  factor     device, n double, or NULL: multiplies est, e.g. trace_before
 *             of ds_calibrate_ex for the admission-time calibrated estimate
 *             (BIAS=ON)
 *  observed   device, n uint32 (tokens)
 *  group      device, n uint32, or NULL; contract: < n_groups
 *  n_groups   number of groups; 0 exactly when group is NULL; <= DS_MAX_GROUPS
 *  stats      device, 4 * (n_groups + 1) double; written
 *  n          <= DS_MAX_ITEMS
 *  ws         workspace of ds_workspace_bytes(DS_OP_ERROR_STATS, n, n_groups)
 * Every sum is taken in an order fixed by the data and n (no floating-point
 * atomics): the same inputs give the same bits on every run. Against exact
 * arithmetic each sum is within the rounding of an n-term sum (relative
 * error at most about n * 2^-53).
 * Unlike the stages, n == 0 still writes stats (counts 0).
 */
ds_status ds_error_stats(uint64_t n, const double *est, const double *factor,
                         const uint32_t *observed, const uint32_t *group, uint32_t n_groups,
                         double *stats, void *ws, size_t ws_bytes, uint32_t flags,
                         ds_stream stream);

/*
 * Runtime classes per semantic category (Eq. (4) classes against the
 * categories of tab:workload_mapping): hist[c * 3 + k] = number of requests
 * i with category[i] == c and job_class[i] == k.
 *
 *  category   device, n uint8; contract: < n_cat
 *  n_cat      1..256
 *  job_class  device, n uint8 (0 short, 1 medium, 2 long; e.g. from ds_score)
 *  hist       device, 3 * n_cat uint32; written
 *  ws         workspace of ds_workspace_bytes(DS_OP_CLASS_HIST, n, 0) bytes
 *             (used by DS_VALIDATE only; may be NULL without that flag)
 * Requests outside the contract are not counted (DS_VALIDATE reports them).
 * n == 0 writes a zero histogram.
 */
ds_status ds_class_histogram(uint32_t n, const uint8_t *category, uint32_t n_cat,
                             const uint8_t *job_class, uint32_t *hist,
                             void *ws, size_t ws_bytes, uint32_t flags, ds_stream stream);

/* Parameters of the dispatch-tick loop. */
typedef struct {
    ds_policy policy;       /* dispatch policy of every tick */
    uint32_t batch;         /* requests dispatched per tick: 1..DS_MAX_BATCH (32 in the paper) */
    double alpha;           /* EMA weight of Eq. (5), in [0, 1] */
    ds_score_params score;  /* budget and factor F of Eq. (1)/(2); the class bounds are unused */
    ds_order_params order;  /* tiers, weights, priorities, aging; t_now is unused (tick k
                               ages to tick_t[k]) */
} ds_sim_params;

/*
 * Dispatch ticks of the online loop (Sec. "Experimental Configuration":
 * dispatch in batches of 32; Sec. "Calibration and Evaluation Phases" and
 * Sec. "Runtime Calibration and Feedback Adaptation": completed requests keep
 * refining later estimates).
 *
 * At tick k the pending set is every request i with arrival[i] <= tick_t[k]
 * that no earlier tick dispatched. It is ordered as ds_order orders it on
 * those requests alone: SJF with the budgets ds_score gives with the factors
 * as they stand, Aging with t_now = tick_t[k], Weighted with a fresh
 * round-robin cycle over the pending tier queues; ties in FIFO order. The
 * first min(batch, pending) requests are dispatched, then their completions
 * update the factors as ds_calibrate does, in dispatch order: event
 * (group[i], B-free estimate of request i as ds_score's est_base, observed[i]).
 *
 *  n          requests, <= DS_MAX_ITEMS
 *  arrival    device, n double; contract: not NaN
 *  tier       device, n uint8; contract: < params->order.n_tiers
 *  counts     device, n uint32: input words (e.g. from ds_characterize)
 *  category   device, n uint8; contract: < n_cat
 *  tenant     device, n uint32; contract: < n_tenants
 *  group      device, n uint32: calibration group; contract: < n_groups
 *  observed   device, n uint32: output tokens the request turns out to have
 *  t_base     device, n_cat double;  s_tenant: device, n_tenants double
 *  n_groups   >= 1
 *  tick_t     device, n_ticks double; contract: non-decreasing, not NaN
 *  n_ticks    <= 2^31 - 1
 *  state      device, n_groups double: factors before the first tick; updated in place
 *  seq        device, n uint32: seq[d] = the request dispatched d-th;
 *             0xFFFFFFFF past the last dispatch
 *  tick_of    device, n int32: the tick that dispatched request i, -1 if none
 *  n_dispatched  device, 1 uint32: number of requests dispatched
 *  ws         workspace of ds_workspace_bytes(DS_OP_SIMULATE, n, 0) bytes
 * One workgroup runs all ticks in one launch. A tick's cost does not grow
 * with the pending set for FIFO, Priority, Weighted and Aging (per-tier
 * queues), nor for SJF with batch <= 32: requests sharing category, tenant
 * and group keep one order whatever the factors, and a tick works on the
 * classes it touches (about 16 us a tick with 1.5 M requests pending). SJF
 * with a larger batch, or from the tick at which (T_base B) S_tenant turns
 * negative or non-finite or a budget exceeds 2^50, passes over the whole
 * pending set every tick (meant for pending sets up to about 10^5); results
 * are the same either way. n == 0 writes *n_dispatched = 0.
 */
ds_status ds_simulate(uint32_t n, const double *arrival, const uint8_t *tier,
                      const uint32_t *counts, const uint8_t *category, const uint32_t *tenant,
                      const uint32_t *group, const uint32_t *observed,
                      const double *t_base, uint32_t n_cat, const double *s_tenant,
                      uint32_t n_tenants, uint32_t n_groups,
                      const double *tick_t, uint32_t n_ticks, const ds_sim_params *params,
                      double *state, uint32_t *seq, int32_t *tick_of, uint32_t *n_dispatched,
                      void *ws, size_t ws_bytes, uint32_t flags, ds_stream stream);

/*
 * Several dispatch-tick loops over the same requests and ticks in one launch
 * (one workgroup per run, after one shared FIFO sort), e.g. the five
 * policies, or a sweep of EMA weights: up to DS_SIM_MAX_RUNS runs, one per
 * compute unit of the device. Run r is ds_simulate with params[r],
 * state[r], seq[r], tick_of[r] and n_dispatched[r]; its results are
 * identical to that call's. The workspace grows with n_runs (about 75 bytes
 * per request per run, plus the shared part).
 *
 *  n_runs        1..DS_SIM_MAX_RUNS
 *  params        HOST array of n_runs parameter sets (each checked as ds_simulate's)
 *  state, seq, tick_of  HOST arrays of n_runs device pointers; the runs'
 *                buffers must not overlap
 *  n_dispatched  device, n_runs uint32
 *  ws            workspace of ds_workspace_bytes(DS_OP_SIMULATE_MULTI, n, n_runs) bytes
 * Other arguments and errors as ds_simulate.
 */
#define DS_SIM_MAX_RUNS 256
ds_status ds_simulate_multi(uint32_t n_runs, uint32_t n, const double *arrival, const uint8_t *tier,
                            const uint32_t *counts, const uint8_t *category, const uint32_t *tenant,
                            const uint32_t *group, const uint32_t *observed, const double *t_base,
                            uint32_t n_cat, const double *s_tenant, uint32_t n_tenants, uint32_t n_groups,
                            const double *tick_t, uint32_t n_ticks, const ds_sim_params *params,
                            double *const *state, uint32_t *const *seq, int32_t *const *tick_of,
                            uint32_t *n_dispatched, void *ws, size_t ws_bytes, uint32_t flags,
                            ds_stream stream);

/*
 * Measurement aid: the practical HBM read rate of ds_characterize's access
 * pattern. Streams `bytes` of buf with the same wave ranges and 16-byte
 * nontemporal loads as the characterize kernel, with no classification. Each
 * wave writes the XOR of its words to a word of its own in xor_out, so the
 * XOR of the DS_READ_BW_WORDS words written there is the XOR of all the
 * buffer's 32-bit (little-endian) words, and no load can be dropped.
 *
 *  buf      device, 16-byte aligned (else DS_ERR_ALIGN); may be NULL if bytes == 0
 *  bytes    a multiple of 16 (else DS_ERR_ARG)
 *  xor_out  device, DS_READ_BW_WORDS uint32, 4-byte aligned; written
 * No workspace; asynchronous on stream.
 */
#define DS_READ_BW_WORDS 32768
ds_status ds_read_bandwidth(const void *buf, uint64_t bytes, uint32_t *xor_out, ds_stream stream);

/* Workspace size for op at size n (prompts, events or requests); n_groups
 * is used by DS_OP_CALIBRATE only. */
size_t ds_workspace_bytes(ds_op op, uint64_t n, uint32_t n_groups);

/* Static description of a status code. */
const char *ds_status_string(ds_status status);

/* Library version as major*10000 + minor*100 + patch. */
uint32_t ds_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DRIFTSCHED_H */
