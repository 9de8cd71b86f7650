// Stage 2: EMA calibration factors, Eq. (5) with the ratio of Eq. (6), over
// completion events in completion order, per calibration group. This file
// serves more than kCalGroupsLds groups; up to that, calchunk.hip.
//
// The recurrence c <- (1 - alpha) c + alpha r is, per group, a composition
// of affine maps x -> a x + b (a = 1 - alpha, b = alpha * obs / est; the
// identity for an event without a usable estimate). Composition is
// associative, so the whole event stream is evaluated as a segmented scan:
//   1. stable partition of the events by group (radix sort on the group id;
//      completion order is kept inside each group),
//   2. per 1024-event tile, per-thread sequential composition of 4 events
//      and a block scan of those: tile aggregates (segment flag, a, b),
//   3. one block scans the tile aggregates (fixed order: deterministic),
//   4. each thread composes its carry-in map, applies it to the group's
//      initial factor, and then runs its 4 events sequentially with the
//      exact update t1 = (1-alpha) c, t2 = alpha r, c = t1 + t2; it writes
//      the factor before and after each event (the traces) and, at a
//      group's last event, the group's final factor.
// Every combine runs in a fixed order, so results are run-to-run identical.
#include "common.h"
#include "kernels.h"

namespace ds {
namespace {

constexpr int kT = 256;
constexpr int kPer = 4;
constexpr uint32_t kTile = kT * kPer;
constexpr uint32_t kNoGroup = 0xFFFFFFFFu;

struct Map {
    uint32_t f;   // a segment (group) starts inside
    double a, b;
};

// x then y
__device__ __forceinline__ Map combine(const Map &x, const Map &y)
{
    if (y.f) return y;
    Map r;
    r.f = x.f;
    r.a = y.a * x.a;
    double t = y.a * x.b;
    r.b = t + y.b;
    return r;
}

struct Events {
    const uint32_t *sidx;    // events in group-major, completion-minor order
    const uint32_t *group;
    const double *est;
    const uint32_t *obs;
    uint32_t E, G;
    double alpha, oma;       // alpha and 1 - alpha
};

__device__ __forceinline__ bool usable(double x) { return isfinite(x) && x > 0.0; }

__device__ __forceinline__ uint32_t group_at(const Events &ev, uint32_t j)
{
    uint32_t e = ev.sidx[j];
    return e < ev.E ? ev.group[e] : kNoGroup;
}

// The (up to) kPer events of this thread: groups, and the affine map of each.
struct Chunk {
    uint32_t e[kPer], g[kPer];
    double a[kPer], b[kPer];
    uint32_t gprev, gnext;   // groups of the events just before and just after
};

__device__ __forceinline__ void load_chunk(const Events &ev, uint32_t j0, Chunk &c)
{
#pragma unroll
    for (int k = 0; k < kPer; k++) {
        uint32_t j = j0 + k;
        uint32_t e = j < ev.E ? ev.sidx[j] : 0u;
        c.e[k] = e < ev.E ? e : 0u;
    }
    c.gprev = j0 == 0 ? kNoGroup : (j0 - 1 < ev.E ? group_at(ev, j0 - 1) : kNoGroup);
    c.gnext = j0 + kPer < ev.E ? group_at(ev, j0 + kPer) : kNoGroup;
#pragma unroll
    for (int k = 0; k < kPer; k++) {
        uint32_t j = j0 + k;
        uint32_t g = j < ev.E ? ev.group[c.e[k]] : kNoGroup;
        double x = j < ev.E ? ev.est[c.e[k]] : 0.0;
        uint32_t o = j < ev.E ? ev.obs[c.e[k]] : 0u;
        c.g[k] = g;
        if (g < ev.G && usable(x)) {
            double r = (double)o / x;
            c.a[k] = ev.oma;
            c.b[k] = ev.alpha * r;
        } else {
            c.a[k] = 1.0;
            c.b[k] = 0.0;
        }
    }
}

// Aggregate of this thread's events.
__device__ __forceinline__ Map chunk_aggregate(const Events &ev, uint32_t j0, const Chunk &c)
{
    Map acc = {0u, 1.0, 0.0};
    uint32_t gprev = c.gprev;
#pragma unroll
    for (int k = 0; k < kPer; k++) {
        uint32_t j = j0 + k;
        if (j >= ev.E) break;
        Map m;
        m.f = (j == 0 || c.g[k] != gprev) ? 1u : 0u;
        gprev = c.g[k];
        m.a = c.a[k];
        m.b = c.b[k];
        acc = combine(acc, m);
    }
    return acc;
}

// Inclusive scan of one Map per thread over the block (Kogge-Stone, fixed order).
__device__ Map block_scan(Map v, uint32_t *sf, double *sa, double *sb)
{
    const int t = threadIdx.x;
    sf[t] = v.f;
    sa[t] = v.a;
    sb[t] = v.b;
    __syncthreads();
    for (int d = 1; d < kT; d <<= 1) {
        Map x = {0u, 1.0, 0.0};
        if (t >= d) { x.f = sf[t - d]; x.a = sa[t - d]; x.b = sb[t - d]; }
        __syncthreads();
        if (t >= d) {
            v = combine(x, v);
            sf[t] = v.f;
            sa[t] = v.a;
            sb[t] = v.b;
        }
        __syncthreads();
    }
    return v;
}

__global__ __launch_bounds__(kT) void k_cal_reduce(Events ev, Map *__restrict__ tile_agg,
                                                   const double *__restrict__ state,
                                                   double *__restrict__ c0)
{
    __shared__ uint32_t sf[kT];
    __shared__ double sa[kT], sb[kT];
    for (uint32_t g = blockIdx.x * kT + threadIdx.x; g < ev.G; g += gridDim.x * kT) c0[g] = state[g];
    const uint32_t j0 = blockIdx.x * kTile + threadIdx.x * kPer;
    Chunk ck;
    load_chunk(ev, j0, ck);
    Map v = chunk_aggregate(ev, j0, ck);
    v = block_scan(v, sf, sa, sb);
    if (threadIdx.x == kT - 1) tile_agg[blockIdx.x] = v;
}

// Exclusive scan over tiles (one block of 1024 threads).
__global__ __launch_bounds__(1024) void k_cal_scan(const Map *__restrict__ tile_agg, uint32_t T,
                                                   Map *__restrict__ tile_carry)
{
    __shared__ uint32_t sf[1024];
    __shared__ double sa[1024], sb[1024];
    const int t = threadIdx.x;
    const uint32_t per = (T + 1023) / 1024;
    const uint32_t b0 = t * per;
    Map acc = {0u, 1.0, 0.0};
    for (uint32_t k = 0; k < per; k++)
        if (b0 + k < T) acc = combine(acc, tile_agg[b0 + k]);
    sf[t] = acc.f;
    sa[t] = acc.a;
    sb[t] = acc.b;
    __syncthreads();
    Map v = acc;
    for (int d = 1; d < 1024; d <<= 1) {
        Map x = {0u, 1.0, 0.0};
        if (t >= d) { x.f = sf[t - d]; x.a = sa[t - d]; x.b = sb[t - d]; }
        __syncthreads();
        if (t >= d) {
            v = combine(x, v);
            sf[t] = v.f;
            sa[t] = v.a;
            sb[t] = v.b;
        }
        __syncthreads();
    }
    Map run = {0u, 1.0, 0.0};
    if (t > 0) { run.f = sf[t - 1]; run.a = sa[t - 1]; run.b = sb[t - 1]; }
    for (uint32_t k = 0; k < per; k++) {
        if (b0 + k < T) {
            tile_carry[b0 + k] = run;
            run = combine(run, tile_agg[b0 + k]);
        }
    }
}

__global__ __launch_bounds__(kT) void k_cal_apply(Events ev, const Map *__restrict__ tile_carry,
                                                  const double *__restrict__ c0,
                                                  double *__restrict__ state,
                                                  double *__restrict__ trace,
                                                  double *__restrict__ trace_before)
{
    __shared__ uint32_t sf[kT];
    __shared__ double sa[kT], sb[kT];
    const int t = threadIdx.x;
    const uint32_t j0 = blockIdx.x * kTile + t * kPer;
    Chunk ck;
    load_chunk(ev, j0, ck);
    Map mine = chunk_aggregate(ev, j0, ck);
    block_scan(mine, sf, sa, sb);
    Map excl = {0u, 1.0, 0.0};
    if (t > 0) { excl.f = sf[t - 1]; excl.a = sa[t - 1]; excl.b = sb[t - 1]; }
    Map cin = combine(tile_carry[blockIdx.x], excl);
    if (j0 >= ev.E) return;

    double c;
    {
        uint32_t g = ck.g[0];
        if (g < ev.G) {
            // carry-in: the composite from this group's first event up to j0
            double tt = cin.a * c0[g];
            c = tt + cin.b;
        } else {
            c = __builtin_nan("");
        }
    }
    uint32_t gprev = ck.gprev;
#pragma unroll
    for (int k = 0; k < kPer; k++) {
        uint32_t j = j0 + k;
        if (j >= ev.E) break;
        uint32_t g = ck.g[k];
        if (j == 0 || g != gprev) c = g < ev.G ? c0[g] : __builtin_nan("");
        if (trace_before) trace_before[ck.e[k]] = c;
        if (ck.a[k] != 1.0 || ck.b[k] != 0.0) {
            // the exact sequential update t1 = (1-alpha) c, t2 = alpha r
            double t1 = ck.a[k] * c;
            c = t1 + ck.b[k];
        }
        if (trace) trace[ck.e[k]] = c;
        uint32_t gn = (k + 1 < kPer) ? (j + 1 < ev.E ? ck.g[k + 1] : kNoGroup) : ck.gnext;
        if (g < ev.G && (j + 1 == ev.E || gn != g)) state[g] = c;
        gprev = g;
    }
}

__global__ void k_cal_validate(const uint32_t *__restrict__ group, uint32_t E, uint32_t G,
                               uint32_t *__restrict__ flag)
{
    uint32_t bad = 0;
    for (uint32_t j = blockIdx.x * blockDim.x + threadIdx.x; j < E; j += gridDim.x * blockDim.x)
        if (group[j] >= G) bad = 1;
    if (bad) atomicOr(flag, 1u);
}

uint32_t bits_for(uint32_t G)
{
    uint32_t b = 0;
    while (b < 32 && ((uint64_t)1 << b) < G) b++;
    return b;
}

}  // namespace

size_t cal_ws_bytes(uint64_t n, uint32_t n_groups)
{
    if (n_groups <= kCalGroupsLds) return calc_ws_bytes(n, n_groups);
    uint64_t T = cdiv(n, kTile);
    return sort_ws_bytes(n, 1) + align_up(n * 4, 256) +
           align_up((uint64_t)n_groups * 8, 256) + 2 * align_up(T * sizeof(Map), 256);
}

hipError_t cal_launch(const uint32_t *group, const double *est, const uint32_t *obs, uint32_t n,
                      double alpha, uint32_t G, double *state, double *trace, double *trace_before,
                      void *ws, uint32_t *flag, hipStream_t s, WaitCfg wait)
{
    if (flag) {
        uint32_t vb = (uint32_t)(cdiv(n, 256) < 1024 ? cdiv(n, 256) : 1024);
        hipLaunchKernelGGL(k_cal_validate, dim3(vb ? vb : 1), dim3(256), 0, s, group, n, G, flag);
        return hipGetLastError();
    }
    if (n == 0) return hipSuccess;
    if (G <= kCalGroupsLds)
        return calc_launch(group, est, obs, n, alpha, G, state, trace, trace_before, ws, s, wait);
    const uint32_t T = (uint32_t)cdiv(n, kTile);
    const uint32_t kb = bits_for(G);
    uint8_t *p = static_cast<uint8_t *>(ws);
    void *sort_ws = p;
    p += sort_ws_bytes(n, 1);
    uint32_t *sidx = reinterpret_cast<uint32_t *>(p);
    p += align_up((uint64_t)n * 4, 256);
    double *c0 = reinterpret_cast<double *>(p);
    p += align_up((uint64_t)G * 8, 256);
    Map *agg = reinterpret_cast<Map *>(p);
    p += align_up((uint64_t)T * sizeof(Map), 256);
    Map *carry = reinterpret_cast<Map *>(p);

    SortInput in = {};
    in.n = n;
    in.group = group;
    in.wait = wait;
    SortJob job = {SortKind::Group, kb, nullptr, sidx};
    hipError_t err = sort_launch(in, &job, 1, sort_ws, s);
    if (err != hipSuccess) return err;

    Events ev;
    ev.sidx = sidx;
    ev.group = group;
    ev.est = est;
    ev.obs = obs;
    ev.E = n;
    ev.G = G;
    ev.alpha = alpha;
    ev.oma = 1.0 - alpha;
    hipLaunchKernelGGL(k_cal_reduce, dim3(T), dim3(kT), 0, s, ev, agg, (const double *)state, c0);
    hipLaunchKernelGGL(k_cal_scan, dim3(1), dim3(1024), 0, s, (const Map *)agg, T, carry);
    hipLaunchKernelGGL(k_cal_apply, dim3(T), dim3(kT), 0, s, ev, (const Map *)carry,
                       (const double *)c0, state, trace, trace_before);
    return hipGetLastError();
}

}  // namespace ds
