// Host-side launchers of the DriftSched kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ds {

// ---- stage 3 arguments (also taken by the fused stage 1 + 3) ------------------
struct ScoreArgs {
    uint32_t n;
    const uint32_t *counts;
    const uint8_t *category;
    const uint32_t *tenant;
    const uint32_t *group;
    const double *t_base;
    uint32_t n_cat;
    const double *s_tenant;
    uint32_t n_tenants;
    const double *state;
    uint32_t n_groups;
    double f_ref, short_max, medium_max;
    double *est_base, *est, *budget;
    uint8_t *job_class;
};

// ---- stage 1: characterize -------------------------------------------------
size_t char_ws_bytes(uint64_t n);
// flag: device word set non-zero by the validation kernel (NULL: no checks).
// score (or NULL): also score each request as its count is written, with
// these arguments (their counts pointer is not used).
hipError_t char_launch(const uint8_t *text, uint64_t text_bytes, const uint64_t *offsets,
                       uint32_t n, uint32_t *counts, void *ws, uint32_t *flag,
                       hipStream_t s, const ScoreArgs *score = nullptr);

// ---- radix sort machinery ----------------------------------------------------
// Producers of (key, value) pairs for the sorts used by calibrate and order.
enum class SortKind : int {
    Fifo = 0,      // key = ordered(arrival[j]), val = j
    Budget = 1,    // key = ordered(budget[fifo[j]]), val = fifo[j]
    Aging = 2,     // key = ordered(aged score of fifo[j]), val = fifo[j]
    Class = 3,     // key = cls[tier[fifo[j]]], val = fifo[j]  (1 pass)
    Tier = 4,      // key = tier[fifo[j]], val = fifo[j]       (1 pass, weighted scatter)
    Group = 5      // key = group[j], val = j                  (calibration partition)
};

constexpr uint32_t kMaxSorts = 4;   // sorts of one batch (same length, same launches)
constexpr uint32_t kWrrMaxWeightSum = 1024;   // smooth round robin: largest sum of the weights
// How Weighted interleaves the tiers inside a cycle (the ABI's weighted_mode).
enum : uint32_t { kWrrBlocked = 0, kWrrSmooth = 1, kWrrStride = 2 };

// Bounded device-side waits (the look-backs of the sorts). A wait that runs
// out sets *status (a word of the caller's workspace) non-zero, or, in a
// sample-sort scatter, sends the sort to its single-workgroup path. `clear`:
// this launch is the call's first to touch *status and zeroes it first.
// no_wait: every wait gives up at once (a diagnostic of the error path).
// A zero-initialised WaitCfg means: bounded waits, errors kept internal.
struct WaitCfg {
    uint32_t *status;
    bool no_wait;
    bool clear;
};

// Inputs and parameters shared by the sorts of a batch.
struct SortInput {
    uint32_t n;
    const double *arrival;
    const double *budget;
    const uint8_t *tier;
    const uint32_t *group;
    const uint32_t *fifo;      // LSD sorts: sequence to reorder (Budget/Aging/Class/Tier)
    uint32_t n_tiers;
    uint32_t cls[16];          // Class: priority class of each tier
    double prio[16];           // Aging/Class keys
    uint32_t weight[16];       // Tier: weighted round robin
    uint32_t wrr_mode;         // Tier: kWrrBlocked, kWrrSmooth (weights sum <= kWrrMaxWeightSum), kWrrStride
    double aging_rate, t_now, aging_floor;
    WaitCfg wait;
};

struct SortJob {
    SortKind kind;
    uint32_t key_bits;         // significant key bits (<= 64)
    double *key_out;           // optional per-request key (indexed by request)
    uint32_t *out;             // n values in key order (Tier: at weighted positions)
};

size_t sort_ws_bytes(uint64_t n, uint32_t nsorts);
// Stable sorts of the produced pairs by key, all jobs in the same launches.
hipError_t sort_launch(const SortInput &in, const SortJob *jobs, uint32_t nsorts, void *ws,
                       hipStream_t s);

// The dispatch orders of at most kSsMaxN requests: a batch of up to
// kSsMaxSorts sample sorts (Fifo, Budget, Aging; at most one of each) by
// composite keys, in three launches; none needs the FIFO order as an input.
// The Fifo job also places the Priority (perm[0]) and Weighted (perm[1])
// orders given in parts (NULL entries: not wanted; the Fifo job's own out
// may then be NULL). `serial` sorts in one workgroup instead (the path taken
// when a bucket overflows).
constexpr uint32_t kSsMaxN = 1u << 18;
constexpr uint32_t kSsMaxSorts = 3;
struct SsPartitions {
    uint32_t *perm[2];
    double *key[2];
};
size_t ssort_ws_bytes(uint64_t n, uint32_t nsorts);   // 0 above kSsMaxN
hipError_t ssort_launch(const SortInput &in, const SortJob *jobs, uint32_t nsorts, bool serial,
                        void *ws, hipStream_t s, const SsPartitions *parts = nullptr);

// The orders of kSsMaxN < n <= kLsMaxN requests, several in the same
// launches: sorts (Fifo; Budget, Aging over in.fifo) by (key, position)
// with sampled splitters, and partitions (Class, Tier over in.fifo) placed
// at the Priority / Weighted positions. job.out receives the values in order
// and job.key_out (if given) each request's key. No waits between blocks.
// The FIFO sort can write the inputs in FIFO order (LsCopies; bud may be
// NULL), which a batch over that sequence then reads instead of gathering
// through in.fifo.
constexpr uint32_t kLsMaxN = 1u << 20;
struct LsCopies {
    double *arr;
    double *bud;
    uint8_t *tier;
};
// A batch's Class partition can also lay out the priority classes' runs for
// the Aging merge (am_merge_launch): each request's aged-score bits and FIFO
// position at its Priority place, and the classes' starts (17 words).
struct LsRuns {
    uint64_t *rk;
    uint32_t *rp;
    uint32_t *cstart;
};
// SJF's splitter sample drawn beside the FIFO sort (draw: that call draws
// it): its keys are the budgets of the sampled requests, with the request
// index standing in for the FIFO position on ties, so it needs no FIFO
// order; a later batch's Budget row (draw false) takes its splitters from
// here. Any sorted splitters give exact results: the bucket sizes come from
// the counts.
struct LsSample {
    uint64_t *raw_k;
    uint32_t *rpart;
    uint64_t *smp_k;
    uint32_t *smp_j;
    bool draw;
};
size_t lsort_sample_bytes(uint64_t n);               // 0 outside (kSsMaxN, kLsMaxN]
LsSample lsort_sample_at(uint64_t n, void *p);       // the buffers at p (lsort_sample_bytes(n) bytes)
size_t lsort_ws_bytes(uint64_t n, uint32_t nsort, uint32_t npart);   // 0 outside (kSsMaxN, kLsMaxN]
hipError_t lsort_launch(const SortInput &in, const SortJob *jobs, uint32_t njobs, void *ws, hipStream_t s,
                        const LsCopies *fifo_in_copies = nullptr, const LsCopies *fifo_out_copies = nullptr,
                        const LsRuns *aging_runs = nullptr, const LsSample *sjf = nullptr);

// Aging above the sample-sort limit as a merge of the priority classes' runs
// of the FIFO sequence (in.fifo, in.cls and the aging parameters set;
// n_classes = the number of distinct priorities). wait_status (may be NULL):
// zeroed by the first kernel (no waits here).
constexpr uint32_t kAmMaxN = 1u << 24;
size_t am_ws_bytes(uint64_t n);
hipError_t am_launch(const SortInput &in, uint32_t n_classes, uint32_t *perm, double *key_out, void *ws,
                     hipStream_t s, uint32_t *wait_status);
// The stable partition of the FIFO sequence by in.cls[tier] alone (16
// classes): run_pos (n) receives the FIFO positions class by class, each
// class in FIFO order, run_start (17) each class's first entry and n.
// The merge rounds alone, over runs formed elsewhere: rk[0] / rp[0] hold
// the K runs (aged-score bits, FIFO position) one after another from
// cstart[0], cstart[K..16] = n; rk[1] / rp[1] are scratch of the same size.
hipError_t am_merge_launch(const SortInput &in, uint32_t n_classes, uint32_t *cstart, uint64_t *const rk[2],
                           uint32_t *const rp[2], uint32_t *perm, double *key_out, hipStream_t s);
size_t am_partition_ws_bytes(uint64_t n);
hipError_t am_partition(const SortInput &in, uint32_t *run_pos, uint32_t *run_start, void *ws, hipStream_t s);

// ---- stage 2: calibrate -------------------------------------------------------
// Up to kCalGroupsLds groups: chunked scan without a global partition.
constexpr uint32_t kCalGroupsLds = 4096;
size_t calc_ws_bytes(uint64_t n, uint32_t n_groups);
// wait.status (may be NULL): zeroed by the first kernel when wait.clear, set
// when a chunk's wait for the maps of the chunks before it runs out.
hipError_t calc_launch(const uint32_t *group, const double *est, const uint32_t *obs, uint32_t n,
                       double alpha, uint32_t n_groups, double *state, double *trace,
                       double *trace_before, void *ws, hipStream_t s, WaitCfg wait = {});
size_t cal_ws_bytes(uint64_t n, uint32_t n_groups);
hipError_t cal_launch(const uint32_t *group, const double *est, const uint32_t *obs,
                      uint32_t n, double alpha, uint32_t n_groups, double *state,
                      double *trace, double *trace_before, void *ws, uint32_t *flag,
                      hipStream_t s, WaitCfg wait = {});

// ---- stage 3: score --------------------------------------------------------------
hipError_t score_launch(uint32_t n, const uint32_t *counts, const uint8_t *category,
                        const uint32_t *tenant, const uint32_t *group, const double *t_base,
                        uint32_t n_cat, const double *s_tenant, uint32_t n_tenants,
                        const double *state, uint32_t n_groups, double f_ref,
                        double short_max, double medium_max, double *est_base, double *est,
                        double *budget, uint8_t *job_class, uint32_t *flag, hipStream_t s);

// ---- stage 4: order ---------------------------------------------------------------
size_t order_ws_bytes(uint64_t n, uint32_t npolicies);
struct OrderArgs {
    uint32_t mask;             // bit p: produce the order of policy p
    uint32_t n;
    const uint8_t *tier;
    const double *arrival;
    const double *budget;
    const uint32_t *fifo_in;
    uint32_t n_tiers;
    uint32_t weight[16];
    uint32_t wrr_mode;         // Weighted: kWrrBlocked, kWrrSmooth or kWrrStride
    double prio[16];
    double aging_rate, t_now, aging_floor;
    uint32_t *perm[5];
    double *key[5];
    bool serial_sort;          // sample-sort path: sort in one workgroup
};
hipError_t order_launch(const OrderArgs &a, void *ws, uint32_t *flag, hipStream_t s,
                        WaitCfg wait = {});

// ---- estimation error and class histogram ------------------------------------------
size_t err_ws_bytes(uint64_t n, uint32_t n_groups);
hipError_t err_launch(uint64_t n, const double *est, const double *factor, const uint32_t *obs,
                      const uint32_t *group, uint32_t n_groups, double *stats, void *ws,
                      uint32_t *flag, hipStream_t s);
hipError_t hist_launch(uint32_t n, const uint8_t *category, uint32_t n_cat,
                       const uint8_t *job_class, uint32_t *hist, uint32_t *flag, hipStream_t s);

// ---- dispatch-tick simulator --------------------------------------------------------
struct SimArgs {
    uint32_t n, n_groups, policy, batch, n_ticks;
    const double *tick_t;      // device, n_ticks, non-decreasing
    double alpha;
    const double *arrival;
    const uint8_t *tier;
    const uint32_t *counts, *tenant, *group, *observed;
    const uint8_t *category;
    const double *t_base, *s_tenant;
    uint32_t n_cat, n_tenants;
    double f_ref;
    uint32_t n_tiers;
    uint32_t weight[16];
    uint32_t wrr_mode;         // Weighted: kWrrBlocked, kWrrSmooth or kWrrStride
    double prio[16];
    double aging_rate, aging_floor;
    double *state;
    uint32_t *seq;
    int32_t *tick_of;
    uint32_t *n_dispatched;
};
constexpr uint32_t kSimMaxBatch = 1024;
constexpr uint32_t kSimMaxRuns = 256;
size_t sim_ws_bytes(uint64_t n, uint32_t n_runs);
// n_runs runs sharing every input array, the ticks and n (their parameters
// and outputs may differ; run r's n_dispatched is runs[0].n_dispatched + r).
hipError_t sim_launch(const SimArgs *runs, uint32_t n_runs, void *ws, uint32_t *flag, hipStream_t s,
                      WaitCfg wait = {});

// ---- misc --------------------------------------------------------------------------
hipError_t fill_u32(uint32_t *p, uint32_t v, uint64_t n, hipStream_t s);
// The read side of characterize alone (bytes a multiple of 16): the XOR of
// the kReadBwWords words of xor_out = the XOR of the buffer's 32-bit words.
constexpr uint32_t kReadBwWords = 32768;   // one per wave (at most this many waves)
hipError_t readbw_launch(const void *buf, uint64_t bytes, uint32_t *xor_out, hipStream_t s);

}  // namespace ds
