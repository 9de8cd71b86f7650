// Stage 2 for up to kCalGroupsLds groups: Eq. (5) with the ratio of Eq. (6)
// (Sec. "Runtime Calibration and Feedback Adaptation") without a global
// partition of the events by group, so that every access is coalesced.
//
// The events, in completion order, are cut into C chunks of L events (L a
// multiple of the sub-tile). With M(c, g) the composition of the affine maps
// x -> (1 - alpha) x + alpha r of group g's events in chunk c (in order):
//   k_calc_agg    per chunk (one block): each sub-tile (512 or 4096 events) is
//                 sorted by group in LDS (stable LSD passes, wave ballots),
//                 scanned as a segmented scan of maps, and each group's part
//                 is composed into that group's map in LDS; the chunk writes
//                 M(c, g) for every group (or "no usable event"). For the
//                 large tables it also writes each event's map from the
//                 chunk's start (through the event when only the trace is
//                 wanted, else to just before it), as a count k of usable
//                 events (its slope is (1 - alpha)^k) and an offset.
//   k_calc_scan   per 64 groups (one block, lane = group): the group's
//                 factor before chunk c is M(c-1, g) o ... o M(0, g) applied
//                 to its initial factor (sixteen stretches of chunks composed
//                 by sixteen waves, then chained in order); writes those
//                 carries and the final factor, and the powers of 1 - alpha.
//   k_calc_ev     large tables, per event: its chunk's carry through its
//                 map; without the event, followed by the exact update t1 =
//                 (1 - alpha) c, t2 = alpha r, c = t1 + t2.
//   k_calc_apply  small tables, per chunk: the same sub-tile sort and scan;
//                 every event then runs the exact update from its carried
//                 factor, in order, and the traces are staged in LDS and
//                 written in event order.
// When the table of chunk maps is small (C x G <= kSmallTable), k_calc_scan
// is left out: each k_calc_apply block applies the maps of the chunks before
// it to the initial factors itself (k_calc_agg keeps a copy of them), and
// the last chunk's block writes the final factors.
// When besides there are at most kOneChunks chunks of one sub-tile each,
// k_calc_one does all of it in one pass over the events: each block sorts
// and scans its sub-tile once, publishes its chunk's maps, reads those of
// the chunks before it (a bounded wait for words not yet written), and
// applies the updates; a small launch before it marks the words unwritten.
// Results match the sequential recurrence up to the rounding of the
// composed maps (a few ulps; the contract is 1e-12 relative).
#include "common.h"
#include "kernels.h"
#include "lookback.h"

namespace ds {
namespace {

constexpr int kT = 512;                  // threads per block
// events per thread per sub-tile (kE) is a template parameter: 1 for the
// small tables (more, shorter blocks; 1, 2 or 4 in one launch), kBigE for
// the large ones; kSub = kT * kE events per sub-tile
constexpr int kW = kT / 64;
constexpr uint32_t kG = kCalGroupsLds;   // groups held in LDS
constexpr uint32_t kMaxTable = 1u << 20; // C x G entries at most (C >= 1)
constexpr uint32_t kMaxChunks = 512;
constexpr uint32_t kSmallTable = 16384;  // C x G up to which the carries are formed in k_calc_apply
constexpr uint32_t kCarryR = 4;          // chunk maps per thread held in registers for the carry
constexpr uint32_t kBigE = 8;            // events per thread per sub-tile of the large tables

struct CalArgs {
    const uint32_t *group;
    const double *est;
    const uint32_t *obs;
    uint32_t E, G;
    double alpha, oma;       // alpha and 1 - alpha
    uint32_t C;              // chunks
    uint32_t L;              // events per chunk
    uint32_t passes;         // 8-bit LSD passes over the group key (key < 2^(8 passes))
    uint32_t keybits;        // bits of the largest key (G, for an event outside the groups)
    double *aggA, *aggB;     // [C][G]: M(c, g) = x -> A x + B; A < 0: no usable event
    double *carry;           // [C][G]: factor of g before chunk c
    double *s0;              // [G] the initial factors (small tables: no k_calc_scan)
    uint32_t small;          // C x G <= kSmallTable
    double *state;           // [G] in: before all events, out: after
    double *trace, *trace_before;
    uint32_t *status;        // the call's wait status word, or NULL: set by a wait that runs out
    uint32_t clear;          // the call's first kernel zeroes *status
    uint32_t no_wait;        // every wait gives up at once (a diagnostic of the error path)
    // large tables with traces: each event's map from its chunk's start to
    // just before it, x -> (1 - alpha)^xk x + xb, in event order; pw[j][d] =
    // (1 - alpha)^(d 256^j)
    // incl: the maps include the event itself (only the trace is wanted)
    double *xb;
    uint32_t *xk;
    double *pw;
    uint32_t incl;
};

// A composed affine map: x -> a x + b, f = a segment starts inside,
// u = some usable event inside, k = how many (a = (1 - alpha)^k).
struct Map {
    uint32_t f, u;
    double a, b;
    uint32_t k;
};

// x then y
__device__ __forceinline__ Map combine(const Map &x, const Map &y)
{
    if (y.f) return y;
    Map r;
    r.f = x.f;
    r.u = x.u | y.u;
    r.a = y.a * x.a;
    const double t = y.a * x.b;
    r.b = t + y.b;
    r.k = x.k + y.k;
    return r;
}

__device__ __forceinline__ double shfl_up_d(double x, int d)
{
    const long long v = __double_as_longlong(x);
    const int lo = __shfl_up((int)(uint32_t)v, d, 64), hi = __shfl_up((int)(uint32_t)(v >> 32), d, 64);
    return __longlong_as_double((long long)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo));
}

__device__ __forceinline__ double shfl_down_d(double x, int d)
{
    const long long v = __double_as_longlong(x);
    const int lo = __shfl_down((int)(uint32_t)v, d, 64), hi = __shfl_down((int)(uint32_t)(v >> 32), d, 64);
    return __longlong_as_double((long long)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo));
}

__device__ __forceinline__ Map shfl_up_map(const Map &m, int d)
{
    Map r;
    r.f = (uint32_t)__shfl_up((int)m.f, d, 64);
    r.u = (uint32_t)__shfl_up((int)m.u, d, 64);
    r.a = shfl_up_d(m.a, d);
    r.b = shfl_up_d(m.b, d);
    r.k = (uint32_t)__shfl_up((int)m.k, d, 64);
    return r;
}

// Inclusive scan of one map per lane over the wave (fixed order).
__device__ __forceinline__ Map wave_scan(Map v)
{
    const int lane = lane_id();
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const Map o = shfl_up_map(v, d);
        if (lane >= d) v = combine(o, v);
    }
    return v;
}

template <int kE>
struct SubShared {
    static constexpr uint32_t kSub = kT * kE;
    uint32_t wcnt[kW][256];
    uint32_t texcl[256];
    Map wagg[kW];
    uint16_t key[kSub];      // group (G for an event outside the groups)
    uint16_t slot[kSub];     // position in the sub-tile
    double b[kSub];          // alpha * r, or 0; reused for trace staging once read
    uint8_t ok[kSub];        // usable
};

// The raw events of a sub-tile (wave-major slots as in load_sort_scan),
// loaded one sub-tile ahead of their use.
template <int kE>
struct Raw {
    uint32_t g[kE], o[kE];
    double x[kE];
};

template <int kE>
__device__ __forceinline__ void load_raw(const CalArgs &a, uint32_t s0, uint32_t m, Raw<kE> &raw)
{
    const int w = (int)(threadIdx.x >> 6), lane = lane_id();
#pragma unroll
    for (int r = 0; r < kE; r++) {
        const uint32_t sl = (uint32_t)w * (64u * kE) + (uint32_t)r * 64u + (uint32_t)lane;
        raw.g[r] = 0;
        raw.o[r] = 0;
        raw.x[r] = 0.0;
        if (sl < m) {
            const uint32_t e = s0 + sl;
            raw.g[r] = a.group[e];
            raw.x[r] = a.est[e];
            raw.o[r] = a.obs[e];
        }
    }
}

// The big sub-tiles (several per chunk) are loaded one ahead: the current
// one's events come from `next`, and the following one's loads are issued
// before the current one is sorted (the barriers there wait on LDS only).
// The small ones are loaded where they are used.
template <int kE>
constexpr bool kPrefetch = kE > 1;

template <int kE>
__device__ __forceinline__ void fetch(const CalArgs &a, uint64_t s0, uint64_t c1, uint32_t m, Raw<kE> &raw,
                                      Raw<kE> &next)
{
    constexpr uint32_t kSub = kT * kE;
    if constexpr (kPrefetch<kE>) {
        raw = next;
        if (s0 + kSub < c1)
            load_raw<kE>(a, (uint32_t)(s0 + kSub), (uint32_t)(c1 - s0 - kSub < kSub ? c1 - s0 - kSub : kSub), next);
    } else {
        load_raw<kE>(a, (uint32_t)s0, m, raw);
    }
}

// The sub-tile of m <= kSub events (m > 0) held in raw, sorted by group and
// scanned. On return (after a barrier that follows every thread's
// reads of sh.b, sh.slot and sh.ok), thread t holds sorted positions 4t ..
// 4t+3: key, slot, b, usable and the segment-start flags; and, when its first
// position continues a segment that starts at p < 4t, `excl`, the
// composition of the maps of positions p .. 4t-1. sh.key keeps the sorted
// keys.
template <int kE>
struct Sub {
    uint32_t key[kE], slot[kE], ok[kE], flag[kE];
    double b[kE];
    Map excl;
};

template <int kE>
__device__ void load_sort_scan(const CalArgs &a, const Raw<kE> &raw, uint32_t m, SubShared<kE> &sh, Sub<kE> &out)
{
    const uint32_t t = threadIdx.x;
    const int w = (int)(t >> 6), lane = lane_id();
    // wave-major slots: wave w holds slots [64 kE w, 64 kE (w + 1)), round r
    // the 64 slots from 64 kE w + 64 r; every load is coalesced
    uint32_t key[kE], slot[kE], ok[kE];
    double b[kE];
#pragma unroll
    for (int r = 0; r < kE; r++) {
        const uint32_t sl = (uint32_t)w * (64u * kE) + (uint32_t)r * 64u + (uint32_t)lane;
        slot[r] = sl;
        key[r] = 0;
        ok[r] = 0;
        b[r] = 0.0;
        if (sl < m) {
            const uint32_t g = raw.g[r];
            const double x = raw.x[r];
            const uint32_t o = raw.o[r];
            key[r] = g < a.G ? g : a.G;
            if (g < a.G && isfinite(x) && x > 0.0) {
                const double ratio = (double)o / x;
                b[r] = a.alpha * ratio;
                ok[r] = 1;
            }
        }
    }
    // stable LSD passes over the key (8 bits each); positions in LDS
    for (uint32_t p = 0; p < a.passes; p++) {
        for (uint32_t i = t; i < kW * 256u; i += kT) (&sh.wcnt[0][0])[i] = 0;
        lds_sync();
        uint32_t rk[kE];
#pragma unroll
        for (int r = 0; r < kE; r++) {
            const uint32_t sl = (uint32_t)w * (64u * kE) + (uint32_t)r * 64u + (uint32_t)lane;
            const bool v = sl < m;
            const uint32_t dg = (key[r] >> (8 * p)) & 255u;
            uint64_t peers = __ballot(v);
#pragma unroll
            for (int bb = 0; bb < 8; bb++) {
                if (8 * p + bb >= a.keybits) break;   // a bit no key has
                const bool bit = (dg >> bb) & 1u;
                const uint64_t mk = __ballot(bit);
                peers &= bit ? mk : ~mk;
            }
            const uint32_t below = (uint32_t)__popcll(peers & lanemask_lt());
            const uint32_t old = v ? sh.wcnt[w][dg] : 0u;
            rk[r] = old + below;
            if (v && below == 0) sh.wcnt[w][dg] = old + (uint32_t)__popcll(peers);
            __builtin_amdgcn_wave_barrier();
        }
        lds_sync();
        if (w == 0) {
            // digits 4 l .. 4 l + 3: per-wave exclusive offsets and digit starts
            uint32_t c[4][kW], tot[4];
#pragma unroll
            for (int e = 0; e < 4; e++)
#pragma unroll
                for (int q = 0; q < kW; q++) c[e][q] = sh.wcnt[q][4 * lane + e];
#pragma unroll
            for (int e = 0; e < 4; e++) {
                uint32_t acc = 0;
#pragma unroll
                for (int q = 0; q < kW; q++) {
                    sh.wcnt[q][4 * lane + e] = acc;
                    acc += c[e][q];
                }
                tot[e] = acc;
            }
            const uint32_t sum = tot[0] + tot[1] + tot[2] + tot[3];
            uint32_t ex = wave_incl_scan_dpp(sum) - sum;
#pragma unroll
            for (int e = 0; e < 4; e++) {
                sh.texcl[4 * lane + e] = ex;
                ex += tot[e];
            }
        }
        lds_sync();
#pragma unroll
        for (int r = 0; r < kE; r++) {
            const uint32_t sl = (uint32_t)w * (64u * kE) + (uint32_t)r * 64u + (uint32_t)lane;
            if (sl < m) {
                const uint32_t dg = (key[r] >> (8 * p)) & 255u;
                const uint32_t q = sh.texcl[dg] + sh.wcnt[w][dg] + rk[r];
                sh.key[q] = (uint16_t)key[r];
                sh.slot[q] = (uint16_t)slot[r];
                sh.b[q] = b[r];
                sh.ok[q] = (uint8_t)ok[r];
            }
        }
        lds_sync();
        if (p + 1 < a.passes) {
#pragma unroll
            for (int r = 0; r < kE; r++) {
                const uint32_t sl = (uint32_t)w * (64u * kE) + (uint32_t)r * 64u + (uint32_t)lane;
                if (sl < m) {
                    key[r] = sh.key[sl];
                    slot[r] = sh.slot[sl];
                    b[r] = sh.b[sl];
                    ok[r] = sh.ok[sl];
                }
            }
            lds_sync();
        }
    }
    // thread t takes sorted positions kE t .. kE t + kE - 1
    Map agg = {0u, 0u, 1.0, 0.0};
#pragma unroll
    for (int e = 0; e < kE; e++) {
        const uint32_t i = t * kE + (uint32_t)e;
        out.key[e] = kG;   // past the end: no group
        out.slot[e] = 0;
        out.ok[e] = 0;
        out.flag[e] = 0;
        out.b[e] = 0.0;
        if (i < m) {
            out.key[e] = sh.key[i];
            out.slot[e] = sh.slot[i];
            out.ok[e] = sh.ok[i];
            out.b[e] = sh.b[i];
            out.flag[e] = (i == 0 || sh.key[i - 1] != sh.key[i]) ? 1u : 0u;
            Map mp;
            mp.f = out.flag[e];
            mp.u = out.ok[e];
            mp.a = out.ok[e] ? a.oma : 1.0;
            mp.b = out.ok[e] ? out.b[e] : 0.0;
            mp.k = out.ok[e];
            agg = (e == 0) ? mp : combine(agg, mp);
        }
    }
    // exclusive scan of the threads' maps: wave scan, then the waves before
    const Map incl = wave_scan(agg);
    if (lane == 63) sh.wagg[w] = incl;
    lds_sync();
    Map before = {1u, 0u, 1.0, 0.0};   // nothing before
    for (int q = 0; q < w; q++) before = (q == 0) ? sh.wagg[0] : combine(before, sh.wagg[q]);
    Map ex = shfl_up_map(incl, 1);
    if (lane == 0) ex = before;
    else if (w > 0) ex = combine(before, ex);
    if (t == 0) ex = Map{1u, 0u, 1.0, 0.0};
    out.excl = ex;
}

// kEv: each event's map from the chunk's start to just before it is
// written as well (xb, xk), so that the updates need no second sort.
template <int kE, bool kEv>
__global__ __launch_bounds__(kT) void k_calc_agg(CalArgs a)
{
    constexpr uint32_t kSub = kT * kE;
    __shared__ SubShared<kE> sh;
    __shared__ double sA[kG], sB[kG];   // the chunk's map per group so far (A < 0: none)
    __shared__ uint32_t sK[kEv ? kG : 1];   // its count of usable events
    __shared__ uint32_t stK[kEv ? kSub : 1];   // per-event counts staged by slot
    const uint32_t t = threadIdx.x, c = blockIdx.x;
    if (a.clear && a.status && c == 0 && t == 0) *a.status = 0;
    for (uint32_t g = t; g < a.G; g += kT) {
        sA[g] = -1.0;
        sB[g] = 0.0;
        if constexpr (kEv) sK[g] = 0;
        if (a.small && c == 0) a.s0[g] = a.state[g];
    }
    const uint64_t c0 = (uint64_t)c * a.L;
    const uint64_t c1 = c0 + a.L < a.E ? c0 + a.L : a.E;
    Raw<kE> next;
    if (kPrefetch<kE> && c0 < c1) load_raw<kE>(a, (uint32_t)c0, (uint32_t)(c1 - c0 < kSub ? c1 - c0 : kSub), next);
    for (uint64_t s0 = c0; s0 < c1; s0 += kSub) {
        const uint32_t m = (uint32_t)(c1 - s0 < kSub ? c1 - s0 : kSub);
        Raw<kE> raw;
        fetch<kE>(a, s0, c1, m, raw, next);
        Sub<kE> sub;
        load_sort_scan<kE>(a, raw, m, sh, sub);   // (its first barrier orders the sA/sB writes)
        if constexpr (kEv) {
            // each event's map from the chunk's start: the chunk's map of
            // its group before this sub-tile, then the group's events of
            // this sub-tile before it; staged by slot, then written in
            // event order
            double *stB = sh.b;                  // read into sub by now
            Map pre = sub.excl;
#pragma unroll
            for (int e = 0; e < kE; e++) {
                const uint32_t i = t * kE + (uint32_t)e;
                if (i >= m) break;
                if (sub.flag[e]) pre = Map{0u, 0u, 1.0, 0.0, 0u};
                Map mp;
                mp.f = sub.flag[e];
                mp.u = sub.ok[e];
                mp.a = sub.ok[e] ? a.oma : 1.0;
                mp.b = sub.ok[e] ? sub.b[e] : 0.0;
                mp.k = sub.ok[e];
                const Map inc = combine(pre, mp);   // the group's events through this one
                if (a.incl) pre = inc;
                const uint32_t g = sub.key[e];
                double xb = pre.u ? pre.b : 0.0;
                uint32_t xk = pre.k;
                if (g < a.G && sA[g] >= 0.0) {
                    const double pb = sB[g];
                    if (pre.u) {
                        const double tt = pre.a * pb;
                        xb = tt + pre.b;
                    } else {
                        xb = pb;
                    }
                    xk += sK[g];
                }
                stB[sub.slot[e]] = xb;
                stK[sub.slot[e]] = xk;
                pre = inc;
            }
            lds_sync();   // every read of sA, sB, sK above precedes the updates below
            for (uint32_t i = t; i < m; i += kT) {
                a.xb[s0 + i] = stB[i];
                a.xk[s0 + i] = stK[i];
            }
        }
        // the segment of each group in this sub-tile, composed into the
        // group's map at the segment's last position (one thread per group)
        Map run = sub.excl;
#pragma unroll
        for (int e = 0; e < kE; e++) {
            const uint32_t i = t * kE + (uint32_t)e;
            if (i >= m) break;
            Map mp;
            mp.f = sub.flag[e];
            mp.u = sub.ok[e];
            mp.a = sub.ok[e] ? a.oma : 1.0;
            mp.b = sub.ok[e] ? sub.b[e] : 0.0;
            mp.k = sub.ok[e];
            run = mp.f ? mp : combine(run, mp);
            const bool last = (i + 1 == m) || (e + 1 < kE ? sub.flag[e + 1] != 0u : sh.key[i + 1] != sh.key[i]);
            const uint32_t g = sub.key[e];
            if (last && g < a.G && run.u) {
                const double pa = sA[g];
                if (pa < 0.0) {
                    sA[g] = run.a;
                    sB[g] = run.b;
                    if constexpr (kEv) sK[g] = run.k;
                } else {
                    // the chunk so far, then this segment
                    sA[g] = run.a * pa;
                    const double tt = run.a * sB[g];
                    sB[g] = tt + run.b;
                    if constexpr (kEv) sK[g] += run.k;
                }
            }
        }
        lds_sync();
    }
    for (uint32_t g = t; g < a.G; g += kT) {
        a.aggA[(uint64_t)c * a.G + g] = sA[g];
        a.aggB[(uint64_t)c * a.G + g] = sB[g];
    }
}

// Carries before every chunk, and the final factors: one block per 64
// groups (lane = group, so every read of a chunk's row is 512 contiguous
// bytes), its sixteen waves over sixteen stretches of the chunks. Each wave
// composes its stretch's maps per group; each then takes the initial factor
// through the earlier stretches' maps in order and walks its own stretch,
// writing the factor before each chunk.
constexpr uint32_t kScanW = 16;
constexpr uint32_t kScanRegs = 16;   // a wave's stretch of chunk maps held in registers, at most
__global__ __launch_bounds__(64 * kScanW) void k_calc_scan(CalArgs a)
{
    __shared__ double sA[kScanW][64], sB[kScanW][64];
    __shared__ uint32_t sU[kScanW][64];
    // the powers of 1 - alpha for the per-event maps: digit d of place j
    if (a.pw && blockIdx.x == 0) {
        const uint32_t j = threadIdx.x >> 8, d = threadIdx.x & 255u;
        a.pw[threadIdx.x] = pow(a.oma, (double)d * (double)(1u << (8 * j)));
    }
    const uint32_t w = threadIdx.x >> 6;
    const int lane = lane_id();
    const uint32_t g = blockIdx.x * 64u + (uint32_t)lane;
    const bool in = g < a.G;
    const uint32_t per = (a.C + kScanW - 1) / kScanW;
    const uint32_t cb = w * per < a.C ? w * per : a.C, ce = cb + per < a.C ? cb + per : a.C;
    if (per <= kScanRegs) {
        // the stretch's maps in registers: one round of loads, walked twice
        double A[kScanRegs], B[kScanRegs];
        Map agg = {0u, 0u, 1.0, 0.0};
#pragma unroll
        for (uint32_t r = 0; r < kScanRegs; r++) {
            A[r] = -1.0;
            B[r] = 0.0;
            if (in && cb + r < ce) {
                A[r] = a.aggA[(uint64_t)(cb + r) * a.G + g];
                B[r] = a.aggB[(uint64_t)(cb + r) * a.G + g];
            }
        }
#pragma unroll
        for (uint32_t r = 0; r < kScanRegs; r++)
            if (A[r] >= 0.0) agg = combine(agg, Map{0u, 1u, A[r], B[r]});
        sA[w][lane] = agg.a;
        sB[w][lane] = agg.b;
        sU[w][lane] = agg.u;
        __syncthreads();
        if (!in) return;
        double v = a.state[g];
        bool touched = false;
        for (uint32_t q = 0; q < kScanW; q++) {
            if (!sU[q][lane]) continue;
            touched = true;
            if (q < w) {
                const double tt = sA[q][lane] * v;
                v = tt + sB[q][lane];
            }
        }
#pragma unroll
        for (uint32_t r = 0; r < kScanRegs; r++) {
            if (cb + r >= ce) break;
            a.carry[(uint64_t)(cb + r) * a.G + g] = v;
            if (A[r] >= 0.0) {
                const double tt = A[r] * v;
                v = tt + B[r];
            }
        }
        // the wave holding the last chunk writes the factor after all events
        // (a group without usable events keeps its factor untouched)
        if (ce == a.C && cb < ce && touched) a.state[g] = v;
        return;
    }
    // four chunks' maps in flight at a time
    constexpr uint32_t kR = 4;
    Map agg = {0u, 0u, 1.0, 0.0};
    if (in)
        for (uint32_t c0 = cb; c0 < ce; c0 += kR) {
            double A[kR], B[kR];
#pragma unroll
            for (uint32_t r = 0; r < kR; r++) {
                A[r] = -1.0;
                B[r] = 0.0;
                if (c0 + r < ce) {
                    A[r] = a.aggA[(uint64_t)(c0 + r) * a.G + g];
                    B[r] = a.aggB[(uint64_t)(c0 + r) * a.G + g];
                }
            }
#pragma unroll
            for (uint32_t r = 0; r < kR; r++)
                if (A[r] >= 0.0) agg = combine(agg, Map{0u, 1u, A[r], B[r]});
        }
    sA[w][lane] = agg.a;
    sB[w][lane] = agg.b;
    sU[w][lane] = agg.u;
    __syncthreads();
    if (!in) return;
    double v = a.state[g];
    bool touched = false;
    for (uint32_t q = 0; q < kScanW; q++) {
        if (!sU[q][lane]) continue;
        touched = true;
        if (q < w) {
            const double tt = sA[q][lane] * v;
            v = tt + sB[q][lane];
        }
    }
    for (uint32_t c0 = cb; c0 < ce; c0 += kR) {
        double A[kR], B[kR];
#pragma unroll
        for (uint32_t r = 0; r < kR; r++) {
            A[r] = -1.0;
            B[r] = 0.0;
            if (c0 + r < ce) {
                A[r] = a.aggA[(uint64_t)(c0 + r) * a.G + g];
                B[r] = a.aggB[(uint64_t)(c0 + r) * a.G + g];
            }
        }
#pragma unroll
        for (uint32_t r = 0; r < kR; r++) {
            if (c0 + r >= ce) break;
            a.carry[(uint64_t)(c0 + r) * a.G + g] = v;
            if (A[r] >= 0.0) {
                const double tt = A[r] * v;
                v = tt + B[r];
            }
        }
    }
    // the wave holding the last chunk writes the factor after all events
    // (a group without usable events keeps its factor untouched)
    if (ce == a.C && cb < ce && touched) a.state[g] = v;
}

// Large tables: every event's factor from its chunk's carry and its map
// from the chunk's start. With incl (the trace alone) the map includes the
// event and gives its trace; otherwise it gives the factor before the
// event, followed by the exact update (Eq. 5 with the ratio of Eq. 6) for a
// usable event. Blocks of 1024 events, which lie in one chunk (chunks are a
// multiple of 2048 events). The dispatcher deals blocks to the 8 XCDs round
// robin; consecutive event ranges go to blocks on the same XCD, so that each
// chunk's row of carries is fetched into one XCD's L2 (not all eight).
constexpr uint32_t kEvR = 4;
constexpr uint32_t kXcds = 8;
static_assert(256 * kEvR == 1024, "");
__global__ __launch_bounds__(256) void k_calc_ev(CalArgs a)
{
    __shared__ double pw[1024];
    const uint32_t t = threadIdx.x;
    const uint32_t per = gridDim.x / kXcds, b = blockIdx.x;
    const uint32_t lb = b < per * kXcds ? (b % kXcds) * per + b / kXcds : b;
    const uint32_t e0 = lb * 1024u;
    const uint64_t row = (uint64_t)(e0 / a.L) * a.G;
    uint32_t g[kEvR], k[kEvR], o[kEvR];
    double xb[kEvR], x[kEvR];
#pragma unroll
    for (uint32_t r = 0; r < kEvR; r++) {
        const uint32_t i = e0 + r * 256u + t;
        g[r] = a.G;
        k[r] = 0;
        o[r] = 0;
        xb[r] = 0.0;
        x[r] = 0.0;
        if (i < a.E) {
            g[r] = a.group[i];
            k[r] = a.xk[i];
            xb[r] = a.xb[i];
            if (!a.incl) {
                x[r] = a.est[i];
                o[r] = a.obs[i];
            }
        }
    }
    double pv[4];
#pragma unroll
    for (uint32_t r = 0; r < 4; r++) pv[r] = a.pw[r * 256u + t];
    double cv[kEvR];
#pragma unroll
    for (uint32_t r = 0; r < kEvR; r++) cv[r] = g[r] < a.G ? a.carry[row + g[r]] : 0.0;
#pragma unroll
    for (uint32_t r = 0; r < 4; r++) pw[r * 256u + t] = pv[r];
    __syncthreads();
    const double nan = __builtin_nan("");
#pragma unroll
    for (uint32_t r = 0; r < kEvR; r++) {
        const uint32_t i = e0 + r * 256u + t;
        if (i >= a.E) break;
        double before = nan, after = nan;
        if (g[r] < a.G) {
            double v = cv[r];
            if (k[r]) {
                // (1 - alpha)^k from its base-256 digits
                const uint32_t kk = k[r];
                double p = pw[kk & 255u];
                p *= pw[256u + ((kk >> 8) & 255u)];
                p *= pw[512u + ((kk >> 16) & 255u)];
                p *= pw[768u + (kk >> 24)];
                const double tt = p * v;
                v = tt + xb[r];
            }
            before = v;
            if (!a.incl && isfinite(x[r]) && x[r] > 0.0) {
                const double ratio = (double)o[r] / x[r];
                const double t1 = a.oma * v;
                v = t1 + a.alpha * ratio;
            }
            after = v;
        }
        if (a.trace) a.trace[i] = after;
        if (a.trace_before) a.trace_before[i] = before;
    }
}

template <int kE>
__global__ __launch_bounds__(kT) void k_calc_apply(CalArgs a)
{
    constexpr uint32_t kSub = kT * kE;
    __shared__ SubShared<kE> sh;
    __shared__ double trb[kSub];   // trace_before staging (the trace goes to sh.b)
    __shared__ double sv[kG];      // each group's factor at the current point of the chunk
    __shared__ uint8_t su[kG];     // small tables: the group has a usable event so far
    const uint32_t t = threadIdx.x, c = blockIdx.x;
    // small tables: the carry is the maps of the chunks before this one,
    // composed in order (tpg threads per group, each over a contiguous range
    // of chunks, kCarryR maps loaded at a time, then an ordered tree of
    // shuffles), applied to the initial factor; a chunk without usable
    // events of the group leaves it untouched. The first kCarryR maps are
    // loaded before the first sub-tile's events and composed after them, so
    // that both loads are in flight together.
    uint32_t tpg = 1;
    while (tpg < 64 && tpg * 2 * a.G <= (uint32_t)kT) tpg *= 2;
    const bool quick = a.small && a.G <= (uint32_t)kT / tpg;
    double cA[kCarryR], cB[kCarryR];
    const uint32_t cjb = (t % tpg) * c / tpg, cje = (t % tpg + 1) * c / tpg;
    if (quick) {
        const uint32_t g = t / tpg, jb = cjb, je = cje;
#pragma unroll
        for (int r = 0; r < (int)kCarryR; r++) {
            const uint32_t j = jb + (uint32_t)r;
            cA[r] = -1.0;
            cB[r] = 0.0;
            if (g < a.G && j < je) {
                cA[r] = a.aggA[(uint64_t)j * a.G + g];
                cB[r] = a.aggB[(uint64_t)j * a.G + g];
            }
        }
    } else if (a.small) {
        for (uint32_t g = t; g < a.G; g += kT) {
            double v = a.s0[g];
            bool u = false;
            for (uint32_t j = 0; j < c; j++) {
                const double A = a.aggA[(uint64_t)j * a.G + g], B = a.aggB[(uint64_t)j * a.G + g];
                if (A >= 0.0) {
                    const double tt = A * v;
                    v = tt + B;
                    u = true;
                }
            }
            sv[g] = v;
            su[g] = (uint8_t)u;
        }
    } else {
        for (uint32_t g = t; g < a.G; g += kT) sv[g] = a.carry[(uint64_t)c * a.G + g];
    }
    const uint64_t c0 = (uint64_t)c * a.L;
    const uint64_t c1 = c0 + a.L < a.E ? c0 + a.L : a.E;
    const double nan = __builtin_nan("");
    double *tr = sh.b;
    Raw<kE> next;
    if (kPrefetch<kE> && c0 < c1) load_raw<kE>(a, (uint32_t)c0, (uint32_t)(c1 - c0 < kSub ? c1 - c0 : kSub), next);
    for (uint64_t s0 = c0; s0 < c1; s0 += kSub) {
        const uint32_t m = (uint32_t)(c1 - s0 < kSub ? c1 - s0 : kSub);
        Raw<kE> raw;
        fetch<kE>(a, s0, c1, m, raw, next);
        Sub<kE> sub;
        load_sort_scan<kE>(a, raw, m, sh, sub);
        if (quick && s0 == c0) {
            const uint32_t g = t / tpg, p = t % tpg;
            Map mp = {0u, 0u, 1.0, 0.0};
#pragma unroll
            for (int r = 0; r < (int)kCarryR; r++)
                if (cA[r] >= 0.0) mp = combine(mp, Map{0u, 1u, cA[r], cB[r]});
            for (uint32_t j0 = cjb + kCarryR; j0 < cje; j0 += kCarryR) {
#pragma unroll
                for (int r = 0; r < (int)kCarryR; r++) {
                    const uint32_t j = j0 + (uint32_t)r;
                    cA[r] = -1.0;
                    cB[r] = 0.0;
                    if (g < a.G && j < cje) {
                        cA[r] = a.aggA[(uint64_t)j * a.G + g];
                        cB[r] = a.aggB[(uint64_t)j * a.G + g];
                    }
                }
#pragma unroll
                for (int r = 0; r < (int)kCarryR; r++)
                    if (cA[r] >= 0.0) mp = combine(mp, Map{0u, 1u, cA[r], cB[r]});
            }
            for (uint32_t d = 1; d < tpg; d <<= 1) {
                Map o;
                o.f = 0u;
                o.u = (uint32_t)__shfl_down((int)mp.u, (int)d, 64);
                o.a = shfl_down_d(mp.a, (int)d);
                o.b = shfl_down_d(mp.b, (int)d);
                if (p % (2 * d) == 0) mp = combine(mp, o);
            }
            if (g < a.G && p == 0) {
                double v = a.s0[g];
                if (mp.u) {
                    const double tt = mp.a * v;
                    v = tt + mp.b;
                }
                sv[g] = v;
                su[g] = (uint8_t)mp.u;
            }
            lds_sync();
        }
        // the factor before this thread's first position: the group's factor
        // at the sub-tile start, through the earlier positions of its
        // segment (their composed map, if any of them is usable)
        double cv;
        {
            const uint32_t g0 = sub.key[0];
            const double base = g0 < a.G ? sv[g0] : nan;
            cv = base;
            if (!sub.flag[0] && sub.excl.u) {
                const double tt = sub.excl.a * base;
                cv = tt + sub.excl.b;
            }
        }
        double after[kE];
#pragma unroll
        for (int e = 0; e < kE; e++) {
            const uint32_t i = t * kE + (uint32_t)e;
            after[e] = cv;
            if (i >= m) continue;
            const uint32_t g = sub.key[e];
            if (sub.flag[e]) cv = g < a.G ? sv[g] : nan;
            trb[sub.slot[e]] = cv;
            if (a.small && sub.ok[e]) su[g] = 1;
            if (sub.ok[e]) {
                // the exact sequential update
                const double t1 = a.oma * cv;
                cv = t1 + sub.b[e];
            }
            tr[sub.slot[e]] = cv;
            after[e] = cv;
        }
        lds_sync();   // every read of sv above precedes the updates below
#pragma unroll
        for (int e = 0; e < kE; e++) {
            const uint32_t i = t * kE + (uint32_t)e;
            if (i >= m) break;
            const bool last = (i + 1 == m) || (e + 1 < kE ? sub.flag[e + 1] != 0u : sh.key[i + 1] != sh.key[i]);
            const uint32_t g = sub.key[e];
            if (last && g < a.G) sv[g] = after[e];
        }
        // the traces in event order
        for (uint32_t i = t; i < m; i += kT) {
            if (a.trace) a.trace[s0 + i] = tr[i];
            if (a.trace_before) a.trace_before[s0 + i] = trb[i];
        }
        lds_sync();
    }
    if (a.small && c + 1 == a.C) {
        // the factors after all events: the groups with a usable event in
        // some chunk (the others keep theirs untouched)
        for (uint32_t g = t; g < a.G; g += kT)
            if (su[g]) a.state[g] = sv[g];
    }
}

// ---- one launch for small tables of one sub-tile per chunk -------------------
//
// Each block publishes its chunk's maps M(c, g) as two 64-bit words per group
// (A, then B) as soon as it has formed them, and only then reads the words
// of the chunks before it, so a block never waits before publishing. Every
// word was set to kUnset (a signalling NaN) by k_calc_unset just before: A
// is -1 or in [0, 1] and B an arithmetic result (never a signalling NaN), so
// each word shows by itself whether it has been written, and no ordering
// between the stores of a block is needed.
constexpr uint64_t kUnset = 0x7FF4DEADBEEF0001ull;
constexpr uint32_t kOneChunks = 64;   // chunks of the one-launch path at most
constexpr uint32_t kOneR = 16;   // chunk maps per thread loaded at once

__device__ __forceinline__ uint64_t ld_relaxed64(const uint64_t *p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void st_relaxed64(uint64_t *p, uint64_t v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ __launch_bounds__(256) void k_calc_unset(uint64_t *w, uint32_t nw, uint32_t *wait_status)
{
    const uint32_t i = blockIdx.x * 256u + threadIdx.x;
    if (wait_status && i == 0) *wait_status = 0;
    for (uint32_t k = i; k < nw; k += gridDim.x * 256u) w[k] = kUnset;
}

template <int kE>
__global__ __launch_bounds__(kT) void k_calc_one(CalArgs a)
{
    constexpr uint32_t kSub = kT * kE;
    static_assert(kSub <= kG, "the trace_before staging shares sA");
    __shared__ SubShared<kE> sh;
    __shared__ double sA[kG], sB[kG];   // this chunk's map per group; sA then stages trace_before
    __shared__ double sv[kG];           // each group's factor (initial, then at the current point)
    __shared__ uint8_t su[kG];          // the group has a usable event so far
    const uint32_t t = threadIdx.x, c = blockIdx.x;
    // the initial factors are read before this block publishes anything: the
    // last block overwrites them only after every other block has published
    for (uint32_t g = t; g < a.G; g += kT) {
        sA[g] = -1.0;
        sB[g] = 0.0;
        sv[g] = a.state[g];
        su[g] = 0;
    }
    const uint64_t c0 = (uint64_t)c * kSub;
    const uint32_t m = (uint32_t)(a.E - c0 < kSub ? a.E - c0 : kSub);
    Raw<kE> raw;
    load_raw<kE>(a, (uint32_t)c0, m, raw);
    Sub<kE> sub;
    load_sort_scan<kE>(a, raw, m, sh, sub);   // (its first barrier orders the writes above)
    // which positions end their group's segment
    uint32_t lastm = 0;
#pragma unroll
    for (int e = 0; e < kE; e++) {
        const uint32_t i = t * kE + (uint32_t)e;
        if (i < m && ((i + 1 == m) || (e + 1 < kE ? sub.flag[e + 1] != 0u : sh.key[i + 1] != sh.key[i])))
            lastm |= 1u << e;
    }
    // this chunk's map of each group: its segment composed at its last position
    {
        Map run = sub.excl;
#pragma unroll
        for (int e = 0; e < kE; e++) {
            if (t * kE + (uint32_t)e >= m) break;
            Map mp;
            mp.f = sub.flag[e];
            mp.u = sub.ok[e];
            mp.a = sub.ok[e] ? a.oma : 1.0;
            mp.b = sub.ok[e] ? sub.b[e] : 0.0;
            mp.k = sub.ok[e];
            run = mp.f ? mp : combine(run, mp);
            const uint32_t g = sub.key[e];
            if (((lastm >> e) & 1u) && g < a.G && run.u) {
                sA[g] = run.a;
                sB[g] = run.b;
            }
        }
    }
    lds_sync();
    uint64_t *pubA = reinterpret_cast<uint64_t *>(a.aggA), *pubB = reinterpret_cast<uint64_t *>(a.aggB);
    if (c + 1 < a.C)   // the last chunk's maps are read by nobody
        for (uint32_t g = t; g < a.G; g += kT) {
            st_relaxed64(&pubA[(uint64_t)c * a.G + g], (uint64_t)__double_as_longlong(sA[g]));
            st_relaxed64(&pubB[(uint64_t)c * a.G + g], (uint64_t)__double_as_longlong(sB[g]));
        }
    // the carry of each group: the maps of chunks 0 .. c-1 composed in order
    // (tpg threads per group, each over a contiguous range of them, then an
    // ordered tree of shuffles), applied to the initial factor
    uint32_t tpg = 1;
    while (tpg < 64 && tpg * 2 * a.G <= (uint32_t)kT) tpg *= 2;
    const uint32_t p = t % tpg, jb = p * c / tpg, je = (p + 1) * c / tpg;
    bool gave_up = false;
    for (uint32_t g0 = 0; g0 < a.G; g0 += kT / tpg) {
        const uint32_t g = g0 + t / tpg;
        const bool gin = g < a.G;
        Map mp = {0u, 0u, 1.0, 0.0};
        if (c > 0 && a.no_wait) gave_up = true;
        for (uint32_t j0 = jb; gin && !gave_up && j0 < je; j0 += kOneR) {
            uint64_t A[kOneR], B[kOneR];
#pragma unroll
            for (uint32_t r = 0; r < kOneR; r++) {
                A[r] = 0;
                B[r] = 0;
                if (j0 + r < je) {
                    A[r] = ld_relaxed64(&pubA[(uint64_t)(j0 + r) * a.G + g]);
                    B[r] = ld_relaxed64(&pubB[(uint64_t)(j0 + r) * a.G + g]);
                }
            }
            // a word still unset is read again until it is written (bounded)
            uint32_t spins = 0;
            for (;;) {
                bool ready = true;
#pragma unroll
                for (uint32_t r = 0; r < kOneR; r++) ready = ready && A[r] != kUnset && B[r] != kUnset;
                if (ready) break;
                if (++spins > kSpinLimit) {
                    gave_up = true;
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
#pragma unroll
                for (uint32_t r = 0; r < kOneR; r++) {
                    if (A[r] == kUnset) A[r] = ld_relaxed64(&pubA[(uint64_t)(j0 + r) * a.G + g]);
                    if (B[r] == kUnset) B[r] = ld_relaxed64(&pubB[(uint64_t)(j0 + r) * a.G + g]);
                }
            }
#pragma unroll
            for (uint32_t r = 0; r < kOneR; r++) {
                const double av = __longlong_as_double((long long)A[r]);
                if (j0 + r < je && av >= 0.0)
                    mp = combine(mp, Map{0u, 1u, av, __longlong_as_double((long long)B[r])});
            }
        }
        for (uint32_t d = 1; d < tpg; d <<= 1) {
            Map o;
            o.f = 0u;
            o.u = (uint32_t)__shfl_down((int)mp.u, (int)d, 64);
            o.a = shfl_down_d(mp.a, (int)d);
            o.b = shfl_down_d(mp.b, (int)d);
            if (p % (2 * d) == 0) mp = combine(mp, o);
        }
        if (gin && p == 0 && mp.u) {
            const double tt = mp.a * sv[g];
            sv[g] = tt + mp.b;
            su[g] = 1;
        }
    }
    if (gave_up && a.status) atomicOr(a.status, 1u);
    lds_sync();
    // every event's exact update from its factor before (as in k_calc_apply)
    const double nan = __builtin_nan("");
    double *tr = sh.b, *trb = sA;
    double cv;
    {
        const uint32_t g0 = sub.key[0];
        const double base = g0 < a.G ? sv[g0] : nan;
        cv = base;
        if (!sub.flag[0] && sub.excl.u) {
            const double tt = sub.excl.a * base;
            cv = tt + sub.excl.b;
        }
    }
    double after[kE];
#pragma unroll
    for (int e = 0; e < kE; e++) {
        const uint32_t i = t * kE + (uint32_t)e;
        after[e] = cv;
        if (i >= m) continue;
        const uint32_t g = sub.key[e];
        if (sub.flag[e]) cv = g < a.G ? sv[g] : nan;
        trb[sub.slot[e]] = cv;
        if (sub.ok[e]) {
            su[g] = 1;
            const double t1 = a.oma * cv;
            cv = t1 + sub.b[e];
        }
        tr[sub.slot[e]] = cv;
        after[e] = cv;
    }
    lds_sync();   // every read of sv above precedes the updates below
#pragma unroll
    for (int e = 0; e < kE; e++) {
        const uint32_t g = sub.key[e];
        if (((lastm >> e) & 1u) && g < a.G) sv[g] = after[e];
    }
    for (uint32_t i = t; i < m; i += kT) {
        if (a.trace) a.trace[c0 + i] = tr[i];
        if (a.trace_before) a.trace_before[c0 + i] = trb[i];
    }
    if (c + 1 == a.C) {
        lds_sync();
        for (uint32_t g = t; g < a.G; g += kT)
            if (su[g]) a.state[g] = sv[g];
    }
}

// Events per thread of the one-launch path for E events and G groups (a
// chunk is one sub-tile of kT times that many events), or 0 when the chunks
// would be too many or their table of maps too large for it.
uint32_t one_e(uint64_t E, uint32_t G)
{
    for (uint32_t e = 1; e <= 4; e *= 2) {
        const uint64_t C = cdiv(E ? E : 1, (uint64_t)kT * e);
        if (C <= kOneChunks && C * G <= kSmallTable) return e;
    }
    return 0;
}

uint32_t sub_per_chunk(uint64_t E, uint32_t G, uint32_t kSub)
{
    uint64_t cmax = kMaxTable / (G ? G : 1);
    cmax = cmax < kMaxChunks ? cmax : kMaxChunks;
    cmax = cmax ? cmax : 1;
    const uint64_t subs = cdiv(E, kSub);
    return (uint32_t)(cdiv(subs, cmax) ? cdiv(subs, cmax) : 1);
}

}  // namespace

// Chunking for kE events per thread: events per chunk and chunks.
static void chunking(uint64_t n, uint32_t G, uint32_t e, uint32_t &L, uint32_t &C)
{
    const uint32_t sub = kT * e;
    L = sub * sub_per_chunk(n, G, sub);
    C = (uint32_t)cdiv(n ? n : 1, L);
}

size_t calc_ws_bytes(uint64_t n, uint32_t G)
{
    // the larger of the two chunkings' tables
    uint32_t L1, C1, L4, C4;
    chunking(n, G, 1, L1, C1);
    chunking(n, G, kBigE, L4, C4);
    const uint64_t C = C1 > C4 ? C1 : C4;
    const size_t base = 3 * align_up(C * G * 8, 256) + align_up((uint64_t)G * 8, 256);
    // the large tables' per-event maps and power tables (k_calc_ev)
    const bool large = one_e(n, G) == 0 && (uint64_t)C1 * G > kSmallTable;
    return large ? base + align_up(1024 * 8, 256) + align_up(n * 8, 256) + align_up(n * 4, 256) : base;
}

hipError_t calc_launch(const uint32_t *group, const double *est, const uint32_t *obs, uint32_t n,
                       double alpha, uint32_t G, double *state, double *trace, double *trace_before,
                       void *ws, hipStream_t s, WaitCfg wait)
{
    if (n == 0) return hipSuccess;
    if (G == 0 || G > kG) return hipErrorInvalidValue;
    CalArgs a;
    a.group = group;
    a.est = est;
    a.obs = obs;
    a.E = n;
    a.G = G;
    a.alpha = alpha;
    a.oma = 1.0 - alpha;
    // few chunks of one sub-tile each: one launch (after the unset words);
    // else sub-tiles of 512 events when the table of chunk maps stays small
    // (the carries are then formed in k_calc_apply), else of 4096
    const uint32_t one = one_e(n, G);
    if (one) {
        a.L = kT * one;
        a.C = (uint32_t)cdiv(n, a.L);
        a.small = 1;
    } else {
        chunking(n, G, 1, a.L, a.C);
        a.small = (uint64_t)a.C * G <= kSmallTable ? 1u : 0u;
        if (!a.small) chunking(n, G, kBigE, a.L, a.C);
    }
    a.passes = G < 256 ? 1u : 2u;   // keys 0..G fit in 8 or 16 bits
    a.keybits = 1;
    while ((1u << a.keybits) <= G) a.keybits++;
    uint8_t *p = static_cast<uint8_t *>(ws);
    const uint64_t tb = align_up((uint64_t)a.C * G * 8, 256);
    a.aggA = reinterpret_cast<double *>(p);
    a.aggB = reinterpret_cast<double *>(p + tb);
    a.carry = reinterpret_cast<double *>(p + 2 * tb);
    a.s0 = reinterpret_cast<double *>(p + 3 * tb);
    // per-event maps (large tables): after the other arrays, at the offsets
    // calc_ws_bytes reserves
    {
        uint32_t L1, C1, L4, C4;
        chunking(n, G, 1, L1, C1);
        chunking(n, G, kBigE, L4, C4);
        const uint64_t Cm = C1 > C4 ? C1 : C4;
        uint8_t *q = p + 3 * align_up(Cm * G * 8, 256) + align_up((uint64_t)G * 8, 256);
        a.pw = reinterpret_cast<double *>(q);
        q += align_up(1024 * 8, 256);
        a.xb = reinterpret_cast<double *>(q);
        q += align_up((uint64_t)n * 8, 256);
        a.xk = reinterpret_cast<uint32_t *>(q);
    }
    a.state = state;
    a.trace = trace;
    a.trace_before = trace_before;
    a.status = wait.status;
    a.clear = wait.clear ? 1u : 0u;
    a.no_wait = wait.no_wait ? 1u : 0u;
    a.incl = trace_before ? 0u : 1u;
    if (one) {
        // one sub-tile per chunk: the words the chunks publish are unset
        // first, then one launch does the rest
        const uint32_t nw = (uint32_t)(tb / 8 + (uint64_t)a.C * G);
        const uint32_t fb = (uint32_t)(cdiv(nw, 256) < 256 ? cdiv(nw, 256) : 256);
        hipLaunchKernelGGL(k_calc_unset, dim3(fb), dim3(256), 0, s, reinterpret_cast<uint64_t *>(a.aggA), nw,
                           a.clear ? a.status : nullptr);
        if (one == 1) hipLaunchKernelGGL(k_calc_one<1>, dim3(a.C), dim3(kT), 0, s, a);
        else if (one == 2) hipLaunchKernelGGL(k_calc_one<2>, dim3(a.C), dim3(kT), 0, s, a);
        else hipLaunchKernelGGL(k_calc_one<4>, dim3(a.C), dim3(kT), 0, s, a);
    } else if (a.small) {
        hipLaunchKernelGGL((k_calc_agg<1, false>), dim3(a.C), dim3(kT), 0, s, a);
        hipLaunchKernelGGL(k_calc_apply<1>, dim3(a.C), dim3(kT), 0, s, a);
    } else if (!trace && !trace_before) {
        // the final factors alone
        a.pw = nullptr;
        hipLaunchKernelGGL((k_calc_agg<kBigE, false>), dim3(a.C), dim3(kT), 0, s, a);
        hipLaunchKernelGGL(k_calc_scan, dim3((G + 63) / 64), dim3(64 * kScanW), 0, s, a);
    } else {
        hipLaunchKernelGGL((k_calc_agg<kBigE, true>), dim3(a.C), dim3(kT), 0, s, a);
        hipLaunchKernelGGL(k_calc_scan, dim3((G + 63) / 64), dim3(64 * kScanW), 0, s, a);
        hipLaunchKernelGGL(k_calc_ev, dim3((uint32_t)cdiv(n, 1024)), dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

}  // namespace ds
