// Smooth weighted round robin, a reading of Sec. "Weighted Scheduling" (the
// paper fixes the dispatch ratio and the cyclic service, not the order of
// the tiers inside a cycle): before each dispatch every non-empty queue's
// credit grows by its weight; the largest credit (the lowest tier on ties)
// is served and gives up the sum W of the non-empty queues' weights. A queue
// that runs empty leaves and the others keep their credits, as the
// published rule passes over an unavailable peer. (Internal to the library.)
//
// The sequence falls into phases, one per set of non-empty queues (a phase
// ends where a queue runs empty; at most one per tier). Within a phase the
// credits are a deterministic function of the previous ones on a finite
// set, so they become periodic; once the credits after W dispatches equal
// those before, the same W dispatches, w_q of them of queue q, repeat until
// the phase ends. From zero credits (the first phase) that holds at once;
// after a queue leaves with a non-zero credit there is a start-up stretch
// first. The plan records for each phase its first position, W, the length
// of its start-up stretch and each tier's dispatches in it (their positions,
// in tpos), each tier's dispatches before the phase, and the offsets of each
// tier's dispatches inside one period. The k-th request of tier q (FIFO
// order) is then served at, with i = k - (q's dispatches before the phase):
//   start + tpos[...]                                 if i < tcnt (start-up),
//   start + tlen + floor(i' / w_q) W + offset[i' mod w_q],  i' = i - tcnt, else.
#pragma once

#include "common.h"
#include "kernels.h"

namespace ds {

constexpr uint32_t kWrrTiers = 16;
constexpr uint32_t kWrrMaxOffsets = kWrrTiers * kWrrMaxWeightSum;

struct WrrPlanHead {
    uint32_t nph;                              // phases
    uint32_t start[kWrrTiers];                 // first position of each phase
    uint32_t W[kWrrTiers];                     // its period
    uint32_t tlen[kWrrTiers];                  // dispatches of its start-up stretch (before the period)
    uint32_t used[kWrrTiers][kWrrTiers];       // [phase][tier] dispatches before the phase
    uint32_t offbase[kWrrTiers][kWrrTiers];    // [phase][tier] first offset in off[]
};

struct WrrPlan {
    WrrPlanHead h;
    uint16_t off[kWrrMaxOffsets];              // dispatch offsets inside a period, ascending per tier
    uint32_t tcnt[kWrrTiers][kWrrTiers];       // [phase][tier] dispatches in the start-up stretch
    uint32_t tbase[kWrrTiers][kWrrTiers];      // [phase][tier] their first entry in tpos
};

// Reductions over the 16 lanes of each DPP row (the tiers are lanes 0..15,
// row 0): rotations by 8, 4, 2, 1 within the row; every lane of a row ends
// with its row's result.
template <int kRor>
__device__ __forceinline__ uint32_t row_ror(uint32_t x)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x120 + kRor, 0xF, 0xF, false);
}

__device__ __forceinline__ int32_t row_max_i32(int32_t x)
{
    int32_t o;
    o = (int32_t)row_ror<8>((uint32_t)x); x = o > x ? o : x;
    o = (int32_t)row_ror<4>((uint32_t)x); x = o > x ? o : x;
    o = (int32_t)row_ror<2>((uint32_t)x); x = o > x ? o : x;
    o = (int32_t)row_ror<1>((uint32_t)x); x = o > x ? o : x;
    return x;
}

__device__ __forceinline__ uint32_t row_sum_u32(uint32_t x)
{
    x += row_ror<8>(x);
    x += row_ror<4>(x);
    x += row_ror<2>(x);
    x += row_ror<1>(x);
    return x;
}

template <int kRor>
__device__ __forceinline__ uint64_t row_ror64(uint64_t x)
{
    return ((uint64_t)row_ror<kRor>((uint32_t)(x >> 32)) << 32) | row_ror<kRor>((uint32_t)x);
}

__device__ __forceinline__ uint64_t row_min_u64(uint64_t x)
{
    uint64_t o;
    o = row_ror64<8>(x); x = o < x ? o : x;
    o = row_ror64<4>(x); x = o < x ? o : x;
    o = row_ror64<2>(x); x = o < x ? o : x;
    o = row_ror64<1>(x); x = o < x ? o : x;
    return x;
}

// One dispatch of the smooth rule over the wave's lanes (lane q = tier q;
// only lanes 0..15 may be active): returns the served lane. total: the sum
// of the active lanes' weights.
__device__ __forceinline__ int wrr_pick(int32_t &credit, bool active, uint32_t wq, uint32_t total)
{
    if (active) credit += (int32_t)wq;
    const int32_t key = active ? credit : INT32_MIN;
    const int32_t mx = row_max_i32(key);   // row 0's maximum in lanes 0..15
    const int best = __ffsll((unsigned long long)__ballot(active && key == mx)) - 1;   // lowest tier
    if (lane_id() == best) credit -= (int32_t)total;
    return best;
}

// The plan for queue lengths len and weights wq held by lane q = tier q of
// one wave (lanes of absent tiers, and every lane from 16 on, pass len = 0;
// weights >= 1 for tiers with requests, their sum <= kWrrMaxWeightSum). per:
// LDS scratch of kWrrMaxWeightSum entries. tpos: global, room for one entry
// per request (the start-up stretches hold at most every request once). The
// plan goes to global memory, for later launches.
//
// Per phase, the wave first plays the rule block by block (W dispatches
// each) from the phase's credits until the credits after a block equal
// those before it (that block is the period) or a queue runs empty (the
// whole phase is then start-up stretch); then it plays the start-up
// stretch again from the same credits, writing each dispatch's position.
// The loops end: every dispatch serves one of the finitely many requests.
__device__ inline void wrr_plan_build(uint32_t len, uint32_t wq, uint16_t *per, WrrPlan *plan,
                                      uint32_t *tpos)
{
    const int lane = lane_id();
    bool active = len > 0u;
    uint32_t used = 0, pos = 0, ph = 0, offcur = 0, tcur = 0;
    int32_t credit = 0;   // kept across phases
    while (__ballot(active) != 0ull) {
        const uint32_t mine = active ? wq : 0u;
        const uint32_t W = readlane32(row_sum_u32(mine), 0);   // row 0 holds every active lane
        const uint32_t base = wave_incl_scan_dpp(mine) - mine;   // this tier's offsets in the period
        const uint32_t rem = active ? len - used : 0u;           // >= 1 when active
        // 1. blocks of W dispatches until one repeats the credits, or the
        //    phase ends
        const int32_t c_in = credit;
        uint32_t t = 0, got = 0;
        bool ended = false;
        for (;;) {
            const int32_t c0 = credit;
            uint32_t cnt = 0;
            for (uint32_t s = 0; s < W; s++) {
                const int b = wrr_pick(credit, active, wq, W);
                const bool me = lane == b;
                if (me) {
                    // a block that turns out to be the period serves w_q of
                    // tier q; the others' offsets are not used
                    if (cnt < wq) per[base + cnt] = (uint16_t)s;
                    cnt++;
                    got++;
                }
                t++;
                if (__ballot(me && got == rem) != 0ull) {
                    ended = true;
                    break;
                }
            }
            if (ended || __ballot(active && credit != c0) == 0ull) break;
        }
        // 2. the start-up stretch: every dispatch of the phase if it ended,
        //    else all but the last block (the period, w_q of tier q)
        const uint32_t tl = ended ? t : t - W;
        const uint32_t tc = ended ? got : (active ? got - wq : 0u);
        const uint32_t tb = tcur + wave_incl_scan_dpp(tc) - tc;
        credit = c_in;
        {
            uint32_t k = 0;
            for (uint32_t s = 0; s < tl; s++) {
                const int b = wrr_pick(credit, active, wq, W);
                if (lane == b) tpos[tb + k++] = s;
            }
        }
        if (lane == 0) {
            plan->h.start[ph] = pos;
            plan->h.W[ph] = W;
            plan->h.tlen[ph] = tl;
        }
        if ((uint32_t)lane < kWrrTiers) {
            plan->h.used[ph][lane] = used;
            plan->h.offbase[ph][lane] = offcur + base;
            plan->tcnt[ph][lane] = tc;
            plan->tbase[ph][lane] = tb;
        }
        uint64_t T;   // dispatches of the phase
        if (ended) {
            T = tl;
            used += tc;
        } else {
            // the period's offsets (each lane reads back only the ones it wrote)
            if (active)
                for (uint32_t i = 0; i < wq; i++) plan->off[offcur + base + i] = per[base + i];
            // the phase ends where the first queue runs empty: a queue's last
            // request is its (r - 1)-th after the start-up stretch
            uint64_t Tq = ~0ull;
            if (active) {
                const uint32_t r = rem - tc;   // >= 1: no queue ran empty in the stretch
                Tq = tl + (uint64_t)((r - 1u) / wq) * W + per[base + (r - 1u) % wq] + 1u;
            }
            T = readlane64(row_min_u64(Tq), 0);   // <= the requests left
            const uint32_t part = (uint32_t)((T - tl) % W);
            uint32_t inpart = 0;
            if (active)
                for (uint32_t i = 0; i < wq; i++) inpart += per[base + i] < part ? 1u : 0u;
            used += active ? tc + (uint32_t)((T - tl) / W) * wq + inpart : 0u;
            // the credits at the phase's end: those of the period's start
            // (now in credit) moved on by the part of a period
            for (uint32_t s = 0; s < part; s++) wrr_pick(credit, active, wq, W);
        }
        pos += (uint32_t)T;
        if (active && used == len) active = false;
        offcur += W;
        tcur += readlane32(row_sum_u32(tc), 0);   // lanes 16..63 hold 0
        ph++;
    }
    if (lane == 0) plan->h.nph = ph;
}

// Position of the k-th request (FIFO order) of tier q, and its round
// floor(k / w_q). head: the plan's header (a copy in LDS), plan: the plan
// (offsets and start-up counts), tpos: the start-up positions.
__device__ __forceinline__ uint64_t wrr_smooth_pos(const WrrPlanHead &head, const WrrPlan *plan,
                                                   const uint32_t *tpos, uint32_t wq, uint32_t q,
                                                   uint32_t k, uint32_t &rnd)
{
    wq = wq ? wq : 1u;
    rnd = k / wq;
    uint32_t ph = 0;
    for (uint32_t p = 1; p < head.nph; p++)
        if (head.used[p][q] <= k) ph = p;
    uint32_t i = k - head.used[ph][q];
    const uint32_t tc = plan->tcnt[ph][q];
    if (i < tc) return (uint64_t)head.start[ph] + tpos[plan->tbase[ph][q] + i];
    i -= tc;
    return (uint64_t)head.start[ph] + head.tlen[ph] + (uint64_t)(i / wq) * head.W[ph] +
           plan->off[head.offbase[ph][q] + i % wq];
}

// The blocked interleaving (the default reading of the same section): round
// r serves up to w_t requests of each tier t in tier order. The k-th request
// (FIFO order) of tier q runs in round r = floor(k / w_q), after
// sum_t min(n_t, r w_t) requests of the earlier rounds and, in round r,
// min(w_t, max(0, n_t - r w_t)) of each tier t < q. cnt(t) = n_t; weights of
// 0 count as 1 for the tier's own round.
template <typename Cnt>
__device__ __forceinline__ uint64_t wrr_blocked_pos(uint32_t q, uint64_t k, const uint32_t *w, uint32_t nq, Cnt cnt,
                                                    uint64_t &rnd)
{
    const uint64_t wq = w[q] ? w[q] : 1u;
    rnd = k / wq;
    uint64_t pos = k - rnd * wq;
    for (uint32_t t = 0; t < nq; t++) {
        const uint64_t nt = cnt(t), wt = w[t], full = rnd * wt;
        pos += nt < full ? nt : full;
        if (t < q) {
            const uint64_t left = nt > full ? nt - full : 0u;
            pos += left < wt ? left : wt;
        }
    }
    return pos;
}

// Stride scheduling, another reading of the same section: queue q's pass
// starts at its stride 1 / w_q and grows by it per dispatch; the smallest
// pass (the lowest tier on ties) is served. The k-th request (FIFO order)
// of tier q runs at pass (k + 1) / w_q, so its place is k plus, for every
// other tier t, the requests of t with a smaller pass, or an equal one when
// t < q: min(n_t, floor((k + 1) w_t / w_q)) for t < q and
// min(n_t, floor(((k + 1) w_t - 1) / w_q)) for t > q. cnt(t) = n_t; weights
// >= 1 below nq (the products stay below 2^62).
template <typename Cnt>
__device__ __forceinline__ uint64_t wrr_stride_pos(uint32_t q, uint64_t k, const uint32_t *w, uint32_t nq, Cnt cnt)
{
    const uint64_t wq = w[q] ? w[q] : 1u, k1 = k + 1u;
    uint64_t pos = k;
    for (uint32_t t = 0; t < nq; t++) {
        if (t == q) continue;
        const uint64_t x = k1 * (w[t] ? w[t] : 1u);
        const uint64_t c = (t < q ? x : x - 1u) / wq;
        const uint64_t nt = cnt(t);
        pos += c < nt ? c : nt;
    }
    return pos;
}

}  // namespace ds
