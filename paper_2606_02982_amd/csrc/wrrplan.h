// Smooth weighted round robin, a reading of Sec. "Weighted Scheduling" (the
// paper fixes the dispatch ratio and the cyclic service, not the order of
// the tiers inside a cycle): before each dispatch every non-empty queue's
// credit grows by its weight; the largest credit (the lowest tier on ties)
// is served and gives up the sum W of the non-empty queues' weights. When a
// queue runs empty a new cycle begins over the queues left, every credit
// back at 0. (Internal to the library.)
//
// From zero credits the rule serves queue q exactly w_q times in W
// dispatches and brings the credits back to 0, so the dispatches repeat with
// period W until a queue runs empty. The plan cuts the sequence into phases
// at those points (at most one per tier); for each phase it records its
// first position, W, every tier's dispatches before it, and the offsets of
// each tier's dispatches inside one period. The k-th request of tier q (FIFO
// order) is then served at
//   start + floor(i / w_q) W + offset[i mod w_q],  i = k - (q's dispatches before the phase).
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
    uint32_t used[kWrrTiers][kWrrTiers];       // [phase][tier] dispatches before the phase
    uint32_t offbase[kWrrTiers][kWrrTiers];    // [phase][tier] first offset in off[]
};

struct WrrPlan {
    WrrPlanHead h;
    uint16_t off[kWrrMaxOffsets];              // dispatch offsets inside a period, ascending per tier
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
// weights >= 1 for tiers with requests, their sum <= kWrrMaxWeightSum). per: LDS scratch of
// kWrrMaxWeightSum entries. The plan goes to global memory, for later
// launches.
__device__ inline void wrr_plan_build(uint32_t len, uint32_t wq, uint16_t *per, WrrPlan *plan)
{
    const int lane = lane_id();
    bool active = len > 0u;
    uint32_t used = 0, pos = 0, ph = 0, offcur = 0;
    while (__ballot(active) != 0ull) {
        const uint32_t mine = active ? wq : 0u;
        const uint32_t W = readlane32(row_sum_u32(mine), 0);   // row 0 holds every active lane
        const uint32_t base = wave_incl_scan_dpp(mine) - mine;   // this tier's offsets in the period
        if (lane == 0) {
            plan->h.start[ph] = pos;
            plan->h.W[ph] = W;
        }
        if ((uint32_t)lane < kWrrTiers) {
            plan->h.used[ph][lane] = used;
            plan->h.offbase[ph][lane] = offcur + base;
        }
        // one period from zero credits: the offsets of each tier's dispatches
        int32_t credit = 0;
        uint32_t cnt = 0;
        for (uint32_t t = 0; t < W; t++) {
            const int b = wrr_pick(credit, active, wq, W);
            if (lane == b) {
                per[base + cnt] = (uint16_t)t;
                plan->off[offcur + base + cnt] = (uint16_t)t;
                cnt++;
            }
        }
        // the phase ends where the first queue runs empty, after T
        // dispatches: a queue's last request is its (rem - 1)-th of the phase
        // (each lane reads back only the offsets it wrote itself)
        uint64_t Tq = ~0ull;
        if (active) {
            const uint32_t rem = len - used;   // >= 1
            Tq = (uint64_t)((rem - 1u) / wq) * W + per[base + (rem - 1u) % wq] + 1u;
        }
        const uint64_t T = readlane64(row_min_u64(Tq), 0);   // <= the requests left
        // each tier's dispatches among those T
        const uint32_t part = (uint32_t)(T % W);
        uint32_t inpart = 0;
        if (active)
            for (uint32_t i = 0; i < wq; i++) inpart += per[base + i] < part ? 1u : 0u;
        used += active ? (uint32_t)(T / W) * wq + inpart : 0u;
        pos += (uint32_t)T;
        if (active && used == len) active = false;
        offcur += W;
        ph++;
    }
    if (lane == 0) plan->h.nph = ph;
}

// Position of the k-th request (FIFO order) of tier q, and its round
// floor(k / w_q). head: the plan's header (a copy in LDS), off: its offsets.
__device__ __forceinline__ uint64_t wrr_smooth_pos(const WrrPlanHead &head, const uint16_t *off, uint32_t wq,
                                                   uint32_t q, uint32_t k, uint32_t &rnd)
{
    wq = wq ? wq : 1u;
    rnd = k / wq;
    uint32_t ph = 0;
    for (uint32_t p = 1; p < head.nph; p++)
        if (head.used[p][q] <= k) ph = p;
    const uint32_t i = k - head.used[ph][q];
    return (uint64_t)head.start[ph] + (uint64_t)(i / wq) * head.W[ph] + off[head.offbase[ph][q] + i % wq];
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
