// C ABI of the DriftSched admission hot path: argument checks, workspace
// carving, validation, and kernel launches on the caller's stream.
#include <math.h>
#include <string.h>

#include <memory>
#include <new>

#include <mutex>

#include "../../include/driftsched.h"
#include "common.h"
#include "kernels.h"

static_assert(DS_WRR_MAX_WEIGHT_SUM == ds::kWrrMaxWeightSum, "smooth round robin weight bound");
static_assert(DS_READ_BW_WORDS == ds::kReadBwWords, "read-rate output words");
static_assert(DS_SIM_MAX_RUNS == ds::kSimMaxRuns, "runs of one simulation launch");
static_assert(DS_WRR_BLOCKED == ds::kWrrBlocked && DS_WRR_SMOOTH == ds::kWrrSmooth &&
                  DS_WRR_STRIDE == ds::kWrrStride,
              "weighted modes");

using namespace ds;

namespace {

constexpr size_t kFlagBytes = 256;   // validation word at the start of every workspace

ds_status hip_status(hipError_t e) { return e == hipSuccess ? DS_OK : DS_ERR_HIP; }

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Runs the enqueue function twice under DS_VALIDATE: first the data checks
// (with a cleared flag), then, if the stream reports no violation, the work.
template <typename F>
ds_status run(void *ws, uint32_t flags, hipStream_t s, F &&enqueue)
{
    uint32_t *flag = static_cast<uint32_t *>(ws);
    if (flags & DS_VALIDATE) {
        hipError_t e = fill_u32(flag, 0u, 1, s);
        if (e == hipSuccess) e = enqueue(flag);
        uint32_t host = 0;
        if (e == hipSuccess) e = hipMemcpyAsync(&host, flag, 4, hipMemcpyDeviceToHost, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) return DS_ERR_HIP;
        if (host) return DS_ERR_DATA;
    }
    return hip_status(enqueue(nullptr));
}

void *after_flag(void *ws) { return static_cast<uint8_t *>(ws) + kFlagBytes; }

// The integer a C caller passed for an enum-typed argument. C allows any int
// there; in C++ a value outside the enumeration's range may not be read as
// the enum type, so it is copied out as bytes first.
template <typename E>
int enum_int(const E &e)
{
    static_assert(sizeof(E) == sizeof(int), "the ABI's enums are int-sized");
    int v;
    memcpy(&v, &e, sizeof v);
    return v;
}

// The calls whose kernels wait on each other (the look-backs of the sorts)
// keep a status word in the workspace, at byte DS_WS_STATUS_OFFSET: the
// call's first kernel zeroes it and a wait that runs out sets it. With
// DS_VALIDATE the call waits for the work and returns DS_ERR_WAIT if it is
// set; without, the word is left for the caller to read.
WaitCfg wait_cfg(void *ws, uint32_t flags)
{
    WaitCfg w;
    w.status = reinterpret_cast<uint32_t *>(static_cast<uint8_t *>(ws) + DS_WS_STATUS_OFFSET);
    w.no_wait = (flags & DS_NO_WAIT) != 0;
    w.clear = true;
    return w;
}

template <typename F>
ds_status run_waits(void *ws, uint32_t flags, hipStream_t s, F &&enqueue)
{
    ds_status st = run(ws, flags, s, enqueue);
    if (st != DS_OK || !(flags & DS_VALIDATE)) return st;
    uint32_t host = 0;
    hipError_t e = hipMemcpyAsync(&host, wait_cfg(ws, flags).status, 4, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return DS_ERR_HIP;
    return host ? DS_ERR_WAIT : DS_OK;
}

}  // namespace

extern "C" {

uint32_t ds_version(void) { return 10000u; }

const char *ds_status_string(ds_status status)
{
    switch (enum_int(status)) {
    case DS_OK: return "ok";
    case DS_ERR_NULL: return "a required pointer is NULL";
    case DS_ERR_ARG: return "argument out of range";
    case DS_ERR_SIZE: return "size exceeds the supported maximum";
    case DS_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case DS_ERR_DATA: return "device data violate the call's contract";
    case DS_ERR_HIP: return "HIP runtime error";
    case DS_ERR_ALIGN: return "array pointer misaligned";
    case DS_ERR_WAIT: return "a bounded device-side wait ran out: the results are invalid";
    }
    return "unknown status";
}

size_t ds_workspace_bytes(ds_op op_arg, uint64_t n, uint32_t n_groups)
{
    switch (enum_int(op_arg)) {
    case DS_OP_CHARACTERIZE: return kFlagBytes + char_ws_bytes(n);
    case DS_OP_CALIBRATE: return kFlagBytes + cal_ws_bytes(n, n_groups ? n_groups : 1);
    case DS_OP_SCORE: return kFlagBytes;
    case DS_OP_ORDER: return kFlagBytes + order_ws_bytes(n, 1);
    case DS_OP_ORDER_MULTI: return kFlagBytes + order_ws_bytes(n, 4);
    case DS_OP_ERROR_STATS: return kFlagBytes + err_ws_bytes(n, n_groups);
    case DS_OP_CLASS_HIST: return kFlagBytes;
    case DS_OP_SIMULATE: return kFlagBytes + sim_ws_bytes(n, 1);
    case DS_OP_SIMULATE_MULTI:
        return n_groups >= 1 && n_groups <= DS_SIM_MAX_RUNS ? kFlagBytes + sim_ws_bytes(n, n_groups) : 0;
    }
    return 0;
}

static ds_status check_ws(void *ws, size_t ws_bytes, size_t need)
{
    if (!ws || ws_bytes < need || !aligned(ws, 256)) return DS_ERR_WORKSPACE;
    return DS_OK;
}

ds_status ds_characterize(const uint8_t *text, uint64_t text_bytes, const uint64_t *offsets,
                          uint32_t n, uint32_t *counts, void *ws, size_t ws_bytes, uint32_t flags,
                          ds_stream stream)
{
    if (n == 0xFFFFFFFFu) return DS_ERR_SIZE;
    if (n == 0) return DS_OK;
    if (!offsets || !counts || (text_bytes > 0 && !text)) return DS_ERR_NULL;
    if (text && !aligned(text, 16)) return DS_ERR_ALIGN;
    if (!aligned(offsets, 8) || !aligned(counts, 4)) return DS_ERR_ALIGN;
    if (text_bytes >= (1ull << 46)) return DS_ERR_SIZE;
    ds_status st = check_ws(ws, ws_bytes, ds_workspace_bytes(DS_OP_CHARACTERIZE, n, 0));
    if (st != DS_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    return run(ws, flags, s, [&](uint32_t *flag) {
        return char_launch(text, text_bytes, offsets, n, counts, after_flag(ws), flag, s);
    });
}

ds_status ds_calibrate_ex(const uint32_t *group, const double *est, const uint32_t *observed,
                          uint64_t n_events, double alpha, uint32_t n_groups, double *state,
                          double *trace, double *trace_before, void *ws, size_t ws_bytes,
                          uint32_t flags, ds_stream stream)
{
    if (n_events > DS_MAX_ITEMS) return DS_ERR_SIZE;
    if (!(alpha >= 0.0 && alpha <= 1.0)) return DS_ERR_ARG;
    if (n_groups == 0) return DS_ERR_ARG;
    if (n_events == 0) return DS_OK;
    if (!group || !est || !observed || !state) return DS_ERR_NULL;
    if (!aligned(group, 4) || !aligned(est, 8) || !aligned(observed, 4) || !aligned(state, 8) ||
        (trace && !aligned(trace, 8)) || (trace_before && !aligned(trace_before, 8)))
        return DS_ERR_ALIGN;
    ds_status st = check_ws(ws, ws_bytes, ds_workspace_bytes(DS_OP_CALIBRATE, n_events, n_groups));
    if (st != DS_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    return run_waits(ws, flags, s, [&](uint32_t *flag) {
        return cal_launch(group, est, observed, (uint32_t)n_events, alpha, n_groups, state, trace,
                          trace_before, after_flag(ws), flag, s, wait_cfg(ws, flags));
    });
}

ds_status ds_calibrate(const uint32_t *group, const double *est, const uint32_t *observed,
                       uint64_t n_events, double alpha, uint32_t n_groups, double *state,
                       double *trace, void *ws, size_t ws_bytes, uint32_t flags, ds_stream stream)
{
    return ds_calibrate_ex(group, est, observed, n_events, alpha, n_groups, state, trace, nullptr,
                           ws, ws_bytes, flags, stream);
}

ds_status ds_score(uint32_t n, const uint32_t *counts, const uint8_t *category,
                   const uint32_t *tenant, const uint32_t *group, const double *t_base,
                   uint32_t n_cat, const double *s_tenant, uint32_t n_tenants, const double *state,
                   uint32_t n_groups, const ds_score_params *params, double *est_base, double *est,
                   double *budget, uint8_t *job_class, void *ws, size_t ws_bytes, uint32_t flags,
                   ds_stream stream)
{
    if (!params) return DS_ERR_NULL;
    if (!(params->f_ref > 0.0) || isnan(params->short_max) || isnan(params->medium_max))
        return DS_ERR_ARG;
    if (n_cat == 0 || n_tenants == 0 || (group && n_groups == 0)) return DS_ERR_ARG;
    if (n == 0) return DS_OK;
    if (!group && n_groups != n) return DS_ERR_ARG;   // one factor per request
    if (!counts || !category || !tenant || !t_base || !s_tenant || !state || !est ||
        !budget || !job_class)
        return DS_ERR_NULL;
    if (!aligned(counts, 4) || !aligned(tenant, 4) || !aligned(group, 4) || !aligned(t_base, 8) ||
        !aligned(s_tenant, 8) || !aligned(state, 8) || !aligned(est, 8) || !aligned(budget, 8) ||
        (est_base && !aligned(est_base, 8)))
        return DS_ERR_ALIGN;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (flags & DS_VALIDATE) {
        ds_status st = check_ws(ws, ws_bytes, ds_workspace_bytes(DS_OP_SCORE, n, 0));
        if (st != DS_OK) return st;
    }
    return run(ws, flags, s, [&](uint32_t *flag) {
        return score_launch(n, counts, category, tenant, group, t_base, n_cat, s_tenant, n_tenants,
                            state, n_groups, params->f_ref, params->short_max, params->medium_max,
                            est_base, est, budget, job_class, flag, s);
    });
}

// The checks and launches of ds_characterize_score on a workspace of at
// least ds_workspace_bytes(DS_OP_CHARACTERIZE, n, 0) bytes (checked by the
// caller).
static ds_status char_score_checks(const uint8_t *text, uint64_t text_bytes, const uint64_t *offsets,
                                   uint32_t n, uint32_t *counts, const uint8_t *category,
                                   const uint32_t *tenant, const uint32_t *group, const double *t_base,
                                   uint32_t n_cat, const double *s_tenant, uint32_t n_tenants,
                                   const double *state, uint32_t n_groups,
                                   const ds_score_params *params, double *est_base, double *est,
                                   double *budget, uint8_t *job_class)
{
    // the checks of ds_characterize and of ds_score
    if (n == 0xFFFFFFFFu) return DS_ERR_SIZE;
    if (!params) return DS_ERR_NULL;
    if (!(params->f_ref > 0.0) || isnan(params->short_max) || isnan(params->medium_max))
        return DS_ERR_ARG;
    if (n_cat == 0 || n_tenants == 0 || (group && n_groups == 0)) return DS_ERR_ARG;
    if (n == 0) return DS_OK;
    if (!group && n_groups != n) return DS_ERR_ARG;   // one factor per request
    if (!offsets || !counts || (text_bytes > 0 && !text)) return DS_ERR_NULL;
    if (!category || !tenant || !t_base || !s_tenant || !state || !est || !budget || !job_class)
        return DS_ERR_NULL;
    if (text && !aligned(text, 16)) return DS_ERR_ALIGN;
    if (!aligned(offsets, 8) || !aligned(counts, 4)) return DS_ERR_ALIGN;
    if (!aligned(tenant, 4) || !aligned(group, 4) || !aligned(t_base, 8) || !aligned(s_tenant, 8) ||
        !aligned(state, 8) || !aligned(est, 8) || !aligned(budget, 8) || (est_base && !aligned(est_base, 8)))
        return DS_ERR_ALIGN;
    if (text_bytes >= (1ull << 46)) return DS_ERR_SIZE;
    return DS_OK;
}

static ds_status char_score_enqueue(const uint8_t *text, uint64_t text_bytes, const uint64_t *offsets,
                                    uint32_t n, uint32_t *counts, const uint8_t *category,
                                    const uint32_t *tenant, const uint32_t *group, const double *t_base,
                                    uint32_t n_cat, const double *s_tenant, uint32_t n_tenants,
                                    const double *state, uint32_t n_groups,
                                    const ds_score_params *params, double *est_base, double *est,
                                    double *budget, uint8_t *job_class, void *ws, uint32_t flags,
                                    hipStream_t s)
{
    ScoreArgs sc = {n, counts, category, tenant, group, t_base, n_cat, s_tenant, n_tenants, state, n_groups,
                    params->f_ref, params->short_max, params->medium_max, est_base, est, budget, job_class};
    return run(ws, flags, s, [&](uint32_t *flag) {
        if (flag) {
            hipError_t e = char_launch(text, text_bytes, offsets, n, counts, after_flag(ws), flag, s);
            if (e != hipSuccess) return e;
            return score_launch(n, counts, category, tenant, group, t_base, n_cat, s_tenant, n_tenants, state,
                                n_groups, params->f_ref, params->short_max, params->medium_max, est_base, est,
                                budget, job_class, flag, s);
        }
        return char_launch(text, text_bytes, offsets, n, counts, after_flag(ws), nullptr, s, &sc);
    });
}

ds_status ds_characterize_score(const uint8_t *text, uint64_t text_bytes, const uint64_t *offsets,
                                uint32_t n, uint32_t *counts, const uint8_t *category,
                                const uint32_t *tenant, const uint32_t *group, const double *t_base,
                                uint32_t n_cat, const double *s_tenant, uint32_t n_tenants,
                                const double *state, uint32_t n_groups, const ds_score_params *params,
                                double *est_base, double *est, double *budget, uint8_t *job_class,
                                void *ws, size_t ws_bytes, uint32_t flags, ds_stream stream)
{
    ds_status st = char_score_checks(text, text_bytes, offsets, n, counts, category, tenant, group, t_base,
                                     n_cat, s_tenant, n_tenants, state, n_groups, params, est_base, est,
                                     budget, job_class);
    if (st != DS_OK || n == 0) return st;
    st = check_ws(ws, ws_bytes, ds_workspace_bytes(DS_OP_CHARACTERIZE, n, 0));
    if (st != DS_OK) return st;
    return char_score_enqueue(text, text_bytes, offsets, n, counts, category, tenant, group, t_base, n_cat,
                              s_tenant, n_tenants, state, n_groups, params, est_base, est, budget,
                              job_class, ws, flags, static_cast<hipStream_t>(stream));
}

}  // extern "C"

// ---- ds_characterize_score without a caller workspace ------------------------------
// Its scratch memory is this static device array: one copy per GPU, held until
// the process ends. On the host, `scratch` names a host-side stand-in, so the
// device address of each GPU's copy is looked up once per device and kept.
namespace {
constexpr size_t kNoAllocScratch = DS_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_dev[kMaxDevices];
}  // namespace

static __device__ __align__(256) uint8_t scratch[kNoAllocScratch];

// The device address of `scratch` on the device that stream s runs on (the
// current device for the null stream).
static ds_status scratch_for(hipStream_t s, void **out)
{
    int dev = 0;
    hipError_t e = s ? hipStreamGetDevice(s, &dev) : hipGetDevice(&dev);
    if (e != hipSuccess || dev < 0 || dev >= kMaxDevices) return DS_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        int cur = 0;
        if (hipGetDevice(&cur) != hipSuccess) return DS_ERR_HIP;
        if (cur != dev && hipSetDevice(dev) != hipSuccess) return DS_ERR_HIP;
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur != dev) (void)hipSetDevice(cur);
        if (e != hipSuccess || !p) return DS_ERR_HIP;
        g_scratch_dev[dev] = p;
    }
    *out = g_scratch_dev[dev];
    return DS_OK;
}

extern "C" {

ds_status ds_characterize_score_noalloc(const uint8_t *text, uint64_t text_bytes,
                                        const uint64_t *offsets, uint32_t n, uint32_t *counts,
                                        const uint8_t *category, const uint32_t *tenant,
                                        const uint32_t *group, const double *t_base, uint32_t n_cat,
                                        const double *s_tenant, uint32_t n_tenants,
                                        const double *state, uint32_t n_groups,
                                        const ds_score_params *params, double *est_base, double *est,
                                        double *budget, uint8_t *job_class, uint32_t flags,
                                        ds_stream stream)
{
    if (n > DS_NOALLOC_MAX_PROMPTS) return DS_ERR_SIZE;
    if (flags != 0) return DS_ERR_ARG;
    ds_status st = char_score_checks(text, text_bytes, offsets, n, counts, category, tenant, group, t_base,
                                     n_cat, s_tenant, n_tenants, state, n_groups, params, est_base, est,
                                     budget, job_class);
    if (st != DS_OK || n == 0) return st;
    if (ds_workspace_bytes(DS_OP_CHARACTERIZE, n, 0) > kNoAllocScratch) return DS_ERR_SIZE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    void *ws = nullptr;
    st = scratch_for(s, &ws);
    if (st != DS_OK) return st;
    return char_score_enqueue(text, text_bytes, offsets, n, counts, category, tenant, group, t_base, n_cat,
                              s_tenant, n_tenants, state, n_groups, params, est_base, est, budget,
                              job_class, ws, 0u, s);
}

static ds_status check_order_params(const ds_order_params *params, uint32_t mask)
{
    if (!params) return DS_ERR_NULL;
    if (params->n_tiers < 1 || params->n_tiers > DS_MAX_TIERS) return DS_ERR_ARG;
    uint64_t wsum = 0;
    for (uint32_t q = 0; q < params->n_tiers; q++) {
        if ((mask & (1u << DS_WEIGHTED)) && params->weight[q] == 0) return DS_ERR_ARG;
        if (!isfinite(params->tier_priority[q])) return DS_ERR_ARG;
        wsum += params->weight[q];
    }
    if (mask & (1u << DS_WEIGHTED)) {
        if (params->weighted_mode > DS_WRR_STRIDE) return DS_ERR_ARG;
        if (params->weighted_mode == DS_WRR_SMOOTH && wsum > DS_WRR_MAX_WEIGHT_SUM) return DS_ERR_ARG;
    }
    if ((mask & (1u << DS_AGING)) &&
        (!(params->aging_rate >= 0.0) || !isfinite(params->aging_rate) ||
         !isfinite(params->t_now) || isnan(params->aging_floor)))
        return DS_ERR_ARG;
    return DS_OK;
}

static ds_status order_common(uint32_t mask, uint32_t n, const uint8_t *tier,
                              const double *arrival, const double *budget,
                              const uint32_t *fifo_in, const ds_order_params *params,
                              uint32_t *const *perms, double *const *keys, void *ws,
                              size_t ws_bytes, ds_op op, uint32_t flags, ds_stream stream)
{
    ds_status st = check_order_params(params, mask);
    if (st != DS_OK) return st;
    if (n > DS_MAX_ITEMS) return DS_ERR_SIZE;
    if (n == 0) return DS_OK;
    if (!tier || !arrival || ((mask & (1u << DS_SJF)) && !budget)) return DS_ERR_NULL;
    for (int p = 0; p < 5; p++)
        if ((mask >> p) & 1u) {
            if (!perms[p]) return DS_ERR_NULL;
            if (!aligned(perms[p], 4) || (keys && keys[p] && !aligned(keys[p], 8))) return DS_ERR_ALIGN;
        }
    if (!aligned(arrival, 8) || (budget && !aligned(budget, 8)) || (fifo_in && !aligned(fifo_in, 4)))
        return DS_ERR_ALIGN;
    st = check_ws(ws, ws_bytes, ds_workspace_bytes(op, n, 0));
    if (st != DS_OK) return st;
    OrderArgs a;
    memset(&a, 0, sizeof(a));
    a.mask = mask;
    a.n = n;
    a.tier = tier;
    a.arrival = arrival;
    a.budget = budget;
    a.fifo_in = fifo_in;
    a.n_tiers = params->n_tiers;
    for (uint32_t q = 0; q < DS_MAX_TIERS; q++) {
        a.weight[q] = q < params->n_tiers ? params->weight[q] : 1u;
        a.prio[q] = q < params->n_tiers ? params->tier_priority[q] : 0.0;
    }
    a.aging_rate = params->aging_rate;
    a.t_now = params->t_now;
    a.aging_floor = params->aging_floor;
    a.wrr_mode = (mask & (1u << DS_WEIGHTED)) ? params->weighted_mode : kWrrBlocked;
    a.serial_sort = (flags & DS_SERIAL_SORT) != 0;
    for (int p = 0; p < 5; p++) {
        a.perm[p] = ((mask >> p) & 1u) ? perms[p] : nullptr;
        a.key[p] = ((mask >> p) & 1u) && keys ? keys[p] : nullptr;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    return run_waits(ws, flags, s, [&](uint32_t *flag) {
        return order_launch(a, after_flag(ws), flag, s, wait_cfg(ws, flags));
    });
}

ds_status ds_order(ds_policy policy, uint32_t n, const uint8_t *tier, const double *arrival,
                   const double *budget, const uint32_t *fifo_in, const ds_order_params *params,
                   uint32_t *perm, double *key, void *ws, size_t ws_bytes, uint32_t flags,
                   ds_stream stream)
{
    const int pol = enum_int(policy);
    if (pol < 0 || pol > 4) return DS_ERR_ARG;
    uint32_t *perms[5] = {nullptr, nullptr, nullptr, nullptr, nullptr};
    double *keys[5] = {nullptr, nullptr, nullptr, nullptr, nullptr};
    perms[pol] = perm;
    keys[pol] = key;
    return order_common(1u << pol, n, tier, arrival, budget, fifo_in, params, perms, keys, ws,
                        ws_bytes, DS_OP_ORDER, flags, stream);
}

ds_status ds_order_multi(uint32_t policy_mask, uint32_t n, const uint8_t *tier,
                         const double *arrival, const double *budget, const uint32_t *fifo_in,
                         const ds_order_params *params, uint32_t *const *perms,
                         double *const *keys, void *ws, size_t ws_bytes, uint32_t flags,
                         ds_stream stream)
{
    if (policy_mask == 0 || policy_mask > 0x1Fu) return DS_ERR_ARG;
    if (!perms) return DS_ERR_NULL;
    return order_common(policy_mask, n, tier, arrival, budget, fifo_in, params, perms, keys, ws,
                        ws_bytes, DS_OP_ORDER_MULTI, flags, stream);
}

ds_status ds_error_stats(uint64_t n, const double *est, const double *factor,
                         const uint32_t *observed, const uint32_t *group, uint32_t n_groups,
                         double *stats, void *ws, size_t ws_bytes, uint32_t flags,
                         ds_stream stream)
{
    if (n > DS_MAX_ITEMS) return DS_ERR_SIZE;
    if ((group != nullptr) != (n_groups > 0)) return DS_ERR_ARG;
    if (n_groups > DS_MAX_GROUPS) return DS_ERR_SIZE;
    if (!stats || (n > 0 && (!est || !observed))) return DS_ERR_NULL;
    if (!aligned(stats, 8) || (est && !aligned(est, 8)) || (factor && !aligned(factor, 8)) ||
        (observed && !aligned(observed, 4)) || (group && !aligned(group, 4)))
        return DS_ERR_ALIGN;
    ds_status st = check_ws(ws, ws_bytes, ds_workspace_bytes(DS_OP_ERROR_STATS, n, n_groups));
    if (st != DS_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    return run(ws, flags, s, [&](uint32_t *flag) {
        return err_launch(n, est, factor, observed, group, n_groups, stats, after_flag(ws), flag, s);
    });
}

ds_status ds_class_histogram(uint32_t n, const uint8_t *category, uint32_t n_cat,
                             const uint8_t *job_class, uint32_t *hist, void *ws, size_t ws_bytes,
                             uint32_t flags, ds_stream stream)
{
    if (n_cat == 0 || n_cat > 256) return DS_ERR_ARG;
    if (!hist || (n > 0 && (!category || !job_class))) return DS_ERR_NULL;
    if (!aligned(hist, 4)) return DS_ERR_ALIGN;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (flags & DS_VALIDATE) {
        ds_status st = check_ws(ws, ws_bytes, ds_workspace_bytes(DS_OP_CLASS_HIST, n, 0));
        if (st != DS_OK) return st;
    }
    return run(ws, flags, s, [&](uint32_t *flag) {
        return hist_launch(n, category, n_cat, job_class, hist, flag, s);
    });
}

// Host checks of one run's parameters and outputs; fills a (shared inputs
// set by the caller).
static ds_status sim_run_args(const ds_sim_params *params, uint32_t n, double *state, uint32_t *seq,
                              int32_t *tick_of, SimArgs &a)
{
    if (!params) return DS_ERR_NULL;
    const int policy = enum_int(params->policy);
    if (policy < 0 || policy > 4) return DS_ERR_ARG;
    if (params->batch < 1 || params->batch > DS_MAX_BATCH) return DS_ERR_ARG;
    if (!(params->alpha >= 0.0 && params->alpha <= 1.0)) return DS_ERR_ARG;
    if (!(params->score.f_ref > 0.0)) return DS_ERR_ARG;
    ds_order_params op = params->order;
    op.t_now = 0.0;   // each tick ages to its own time
    ds_status st = check_order_params(&op, 1u << policy);
    if (st != DS_OK) return st;
    if (n > 0 && (!state || !seq || !tick_of)) return DS_ERR_NULL;
    if ((state && !aligned(state, 8)) || (seq && !aligned(seq, 4)) || (tick_of && !aligned(tick_of, 4)))
        return DS_ERR_ALIGN;
    a.policy = (uint32_t)policy;
    a.batch = params->batch;
    a.alpha = params->alpha;
    a.f_ref = params->score.f_ref;
    a.n_tiers = params->order.n_tiers;
    for (uint32_t q = 0; q < DS_MAX_TIERS; q++) {
        a.weight[q] = q < a.n_tiers ? params->order.weight[q] : 1u;
        a.prio[q] = q < a.n_tiers ? params->order.tier_priority[q] : 0.0;
    }
    a.wrr_mode = policy == DS_WEIGHTED ? params->order.weighted_mode : kWrrBlocked;
    a.aging_rate = params->order.aging_rate;
    a.aging_floor = params->order.aging_floor;
    a.state = state;
    a.seq = seq;
    a.tick_of = tick_of;
    return DS_OK;
}

static ds_status sim_common(uint32_t n_runs, uint32_t n, const double *arrival, const uint8_t *tier,
                            const uint32_t *counts, const uint8_t *category, const uint32_t *tenant,
                            const uint32_t *group, const uint32_t *observed, const double *t_base,
                            uint32_t n_cat, const double *s_tenant, uint32_t n_tenants, uint32_t n_groups,
                            const double *tick_t, uint32_t n_ticks, const ds_sim_params *params,
                            double *const *state, uint32_t *const *seq, int32_t *const *tick_of,
                            uint32_t *n_dispatched, void *ws, size_t ws_bytes, ds_op op, uint32_t flags,
                            ds_stream stream)
{
    if (n_runs < 1 || n_runs > DS_SIM_MAX_RUNS) return DS_ERR_ARG;
    if (!params || !state || !seq || !tick_of) return DS_ERR_NULL;
    std::unique_ptr<SimArgs[]> runs(new (std::nothrow) SimArgs[n_runs]);
    if (!runs) return DS_ERR_HIP;
    memset(runs.get(), 0, n_runs * sizeof(SimArgs));
    for (uint32_t r = 0; r < n_runs; r++) {
        ds_status st = sim_run_args(params + r, n, state[r], seq[r], tick_of[r], runs[r]);
        if (st != DS_OK) return st;
    }
    if (n_cat == 0 || n_cat > 256 || n_tenants == 0 || n_groups == 0) return DS_ERR_ARG;
    if (n > DS_MAX_ITEMS) return DS_ERR_SIZE;
    if (n_ticks > 0x7FFFFFFFu) return DS_ERR_SIZE;
    if (!n_dispatched) return DS_ERR_NULL;
    if (n > 0 && (!arrival || !tier || !counts || !category || !tenant || !group || !observed ||
                  !t_base || !s_tenant || (n_ticks && !tick_t)))
        return DS_ERR_NULL;
    if (!aligned(n_dispatched, 4) || (arrival && !aligned(arrival, 8)) ||
        (counts && !aligned(counts, 4)) || (tenant && !aligned(tenant, 4)) ||
        (group && !aligned(group, 4)) || (observed && !aligned(observed, 4)) ||
        (t_base && !aligned(t_base, 8)) || (s_tenant && !aligned(s_tenant, 8)) ||
        (tick_t && !aligned(tick_t, 8)))
        return DS_ERR_ALIGN;
    ds_status st = check_ws(ws, ws_bytes, ds_workspace_bytes(op, n, op == DS_OP_SIMULATE ? 0 : n_runs));
    if (st != DS_OK) return st;
    for (uint32_t r = 0; r < n_runs; r++) {
        SimArgs &a = runs[r];
        a.n = n;
        a.n_groups = n_groups;
        a.n_ticks = n_ticks;
        a.tick_t = tick_t;
        a.arrival = arrival;
        a.tier = tier;
        a.counts = counts;
        a.tenant = tenant;
        a.group = group;
        a.observed = observed;
        a.category = category;
        a.t_base = t_base;
        a.s_tenant = s_tenant;
        a.n_cat = n_cat;
        a.n_tenants = n_tenants;
        a.n_dispatched = n_dispatched + r;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    return run_waits(ws, flags, s, [&](uint32_t *flag) {
        return sim_launch(runs.get(), n_runs, after_flag(ws), flag, s, wait_cfg(ws, flags));
    });
}

ds_status ds_simulate(uint32_t n, const double *arrival, const uint8_t *tier,
                      const uint32_t *counts, const uint8_t *category, const uint32_t *tenant,
                      const uint32_t *group, const uint32_t *observed, const double *t_base,
                      uint32_t n_cat, const double *s_tenant, uint32_t n_tenants,
                      uint32_t n_groups, const double *tick_t, uint32_t n_ticks,
                      const ds_sim_params *params, double *state, uint32_t *seq,
                      int32_t *tick_of, uint32_t *n_dispatched, void *ws, size_t ws_bytes,
                      uint32_t flags, ds_stream stream)
{
    return sim_common(1, n, arrival, tier, counts, category, tenant, group, observed, t_base, n_cat, s_tenant,
                      n_tenants, n_groups, tick_t, n_ticks, params, &state, &seq, &tick_of, n_dispatched, ws,
                      ws_bytes, DS_OP_SIMULATE, flags, stream);
}

ds_status ds_simulate_multi(uint32_t n_runs, uint32_t n, const double *arrival, const uint8_t *tier,
                            const uint32_t *counts, const uint8_t *category, const uint32_t *tenant,
                            const uint32_t *group, const uint32_t *observed, const double *t_base,
                            uint32_t n_cat, const double *s_tenant, uint32_t n_tenants, uint32_t n_groups,
                            const double *tick_t, uint32_t n_ticks, const ds_sim_params *params,
                            double *const *state, uint32_t *const *seq, int32_t *const *tick_of,
                            uint32_t *n_dispatched, void *ws, size_t ws_bytes, uint32_t flags,
                            ds_stream stream)
{
    return sim_common(n_runs, n, arrival, tier, counts, category, tenant, group, observed, t_base, n_cat,
                      s_tenant, n_tenants, n_groups, tick_t, n_ticks, params, state, seq, tick_of, n_dispatched,
                      ws, ws_bytes, DS_OP_SIMULATE_MULTI, flags, stream);
}

ds_status ds_read_bandwidth(const void *buf, uint64_t bytes, uint32_t *xor_out, ds_stream stream)
{
    if (bytes % 16 != 0) return DS_ERR_ARG;
    if (!xor_out || (bytes && !buf)) return DS_ERR_NULL;
    if (!aligned(xor_out, 4) || (buf && !aligned(buf, 16))) return DS_ERR_ALIGN;
    hipStream_t s = static_cast<hipStream_t>(stream);
    return hip_status(readbw_launch(buf, bytes, xor_out, s));
}

}  // extern "C"
