// Priority and Weighted orders of up to kSsMaxN requests in one pass over
// the FIFO sequence (Sec. "Priority Scheduling", Sec. "Weighted
// Scheduling"); the tile body shared by k_part and the launch that also
// samples the SJF/Aging sorts (internal to the library).
//
// Both orders are stable partitions of the FIFO sequence by a digit of at
// most 4 bits: the priority class of the request's tier (Priority) or the
// tier (Weighted). Per tile of 2048 FIFO positions, a block
//   * adds up the tier counts of slices of the batch (made by an earlier
//     launch; they give each class's first position and the queue lengths of
//     the round-robin closed form),
//   * ranks its positions by digit with wave ballots,
//   * takes the digit's count over earlier tiles by decoupled look-back,
//   * and writes each request at its place: class start + rank in class,
//     or the round-robin position of the k-th request of its tier,
//     sum_t' min(n_t', r w_t') + sum_{t' < t} min(w_t', max(0, n_t' - r w_t'))
//     + (k - r w_t), r = floor(k / w_t).
// The look-back words are cleared by an earlier launch of the same call.
#pragma once

#include "common.h"
#include "kernels.h"
#include "lookback.h"
#include "tiercount.h"

namespace ds {

constexpr uint32_t kPTile = 2048;   // FIFO positions per tile
constexpr uint32_t kQ = 16;         // digits (tiers, classes)

struct PartJob {
    SortKind kind;             // Class (Priority) or Tier (Weighted)
    double *key_out;
    uint32_t *out;
    uint32_t *status;          // [tiles][kQ] look-back words, zero on entry
    uint32_t *error;           // set if a look-back wait ran out
};

struct PartBatch {
    SortInput in;
    uint32_t n;
    uint32_t tiles;
    uint32_t njobs;
    const uint32_t *tier_part;   // [nparts][16] tier counts of slices
    uint32_t nparts;
    PartJob job[2];
};

// The batch of one or two partition jobs (status: part_ws_bytes(n) bytes of
// look-back words per job, zeroed).
PartBatch part_batch(const SortInput &in, const SortJob *jobs, uint32_t njobs, uint32_t *status,
                     uint32_t *error, const uint32_t *tier_part, uint32_t nparts);

// Tile `tile` of job `job`, by a block of TPB threads.
template <int TPB>
__device__ void part_body(const PartBatch &b, uint32_t job, uint32_t tile)
{
    constexpr int kPR = (int)(kPTile / TPB);
    constexpr int kPWaves = TPB / 64;

    __shared__ uint32_t s_tot[kQ];          // requests per tier
    __shared__ uint32_t s_start[kQ];        // Priority: first position of each class
    __shared__ uint32_t wcnt[kPWaves][kQ];
    __shared__ uint32_t s_pre[kQ];          // digit count over earlier tiles

    const PartJob &J = b.job[job];
    const SortInput &in = b.in;
    const uint32_t t = threadIdx.x, n = b.n, nq = in.n_tiers;
    const int w = (int)(t >> 6), lane = lane_id();
    const uint32_t base = tile * kPTile;
    const uint32_t cnt = n - base < kPTile ? n - base : kPTile;
    const bool cls = J.kind == SortKind::Class;

    // this tile's requests (loads first) and their digits
    uint32_t id[kPR], qv[kPR], dg[kPR], rk[kPR];
#pragma unroll
    for (int r = 0; r < kPR; r++) {
        const uint32_t idx = (uint32_t)w * (64u * kPR) + (uint32_t)r * 64u + (uint32_t)lane;
        const uint32_t i = idx < cnt ? in.fifo[base + idx] : 0u;
        id[r] = i < n ? i : 0u;
    }
#pragma unroll
    for (int r = 0; r < kPR; r++) {
        const uint32_t idx = (uint32_t)w * (64u * kPR) + (uint32_t)r * 64u + (uint32_t)lane;
        const uint32_t q = in.ftier ? (idx < cnt ? in.ftier[base + idx] : 0u) : in.tier[id[r]];
        qv[r] = q < kQ ? q : kQ - 1u;
        dg[r] = cls ? in.cls[qv[r]] : qv[r];
    }

    // requests per tier: the sum of the slices' counts
    if (t < kQ) s_tot[t] = 0;
    __syncthreads();
    for (uint32_t i = t; i < b.nparts * kTierCounts; i += TPB) {
        const uint32_t c = b.tier_part[i];
        if (c) atomicAdd(&s_tot[i % kTierCounts], c);
    }
    // stable rank in the tile by digit, round by round
    if (t < kPWaves * kQ) (&wcnt[0][0])[t] = 0;
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kPR; r++) {
        const uint32_t idx = (uint32_t)w * (64u * kPR) + (uint32_t)r * 64u + (uint32_t)lane;
        const bool ok = idx < cnt;
        uint64_t peers = __ballot(ok);
#pragma unroll
        for (int bb = 0; bb < 4; bb++) {
            const bool bit = (dg[r] >> bb) & 1u;
            const uint64_t m = __ballot(bit);
            peers &= bit ? m : ~m;
        }
        const uint32_t below = (uint32_t)__popcll(peers & lanemask_lt());
        const uint32_t old = ok ? wcnt[w][dg[r]] : 0u;
        rk[r] = old + below;
        if (ok && below == 0) wcnt[w][dg[r]] = old + (uint32_t)__popcll(peers);
        __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();
    if (t < kQ) {
        uint32_t c[kPWaves], tc = 0;
#pragma unroll
        for (int q = 0; q < kPWaves; q++) c[q] = wcnt[q][t];
#pragma unroll
        for (int q = 0; q < kPWaves; q++) {
            wcnt[q][t] = tc;
            tc += c[q];
        }
        uint32_t *st = J.status;
        st_relaxed(&st[(uint64_t)tile * kQ + t], (tile == 0 ? kPre : kAgg) | tc);
        uint32_t prefix = 0;
        if (tile > 0) {
            prefix = look_back<kQ>(st, tile, t, J.error);
            st_relaxed(&st[(uint64_t)tile * kQ + t], kPre | (prefix + tc));
        }
        s_pre[t] = prefix;
    }
    __syncthreads();
    if (t < kQ) {
        // first position of class t: the requests of every tier of a lower class
        uint32_t s = 0;
        for (uint32_t q = 0; q < nq; q++) s += in.cls[q] < t ? s_tot[q] : 0u;
        s_start[t] = s;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kPR; r++) {
        const uint32_t idx = (uint32_t)w * (64u * kPR) + (uint32_t)r * 64u + (uint32_t)lane;
        if (idx >= cnt) continue;
        // rank of the request among its digit's requests in FIFO order
        const uint64_t k = (uint64_t)s_pre[dg[r]] + wcnt[w][dg[r]] + rk[r];
        const uint32_t q = qv[r];
        uint64_t pos;
        double key;
        if (cls) {
            pos = s_start[dg[r]] + k;
            key = in.prio[q];
        } else {
            const uint32_t wq = in.weight[q] ? in.weight[q] : 1u;
            const uint64_t rnd = (uint32_t)k / wq;   // k < n <= 2^18
            pos = k - rnd * wq;
            for (uint32_t u = 0; u < nq; u++) {
                const uint64_t nt = s_tot[u], wt = in.weight[u], full = rnd * wt;
                pos += nt < full ? nt : full;
                if (u < q) {
                    const uint64_t left = nt > full ? nt - full : 0u;
                    pos += left < wt ? left : wt;
                }
            }
            key = (double)rnd;
        }
        if (pos < n) J.out[pos] = id[r];   // always, for tiers < n_tiers
        if (J.key_out) J.key_out[id[r]] = key;
    }
}


}  // namespace ds
