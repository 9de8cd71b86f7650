// Requests per tier over a slice of the batch (internal to the library):
// block `part` of `nparts` counts the tiers of requests
// [part n / nparts, (part + 1) n / nparts) and writes 16 counts (tiers 0..15;
// a larger value counts as tier 15) to out[16 part ..]. The Priority and
// Weighted partitions add the slices up for the class starts and the queue
// lengths of the round-robin closed form.
#pragma once

#include "common.h"

namespace ds {

constexpr uint32_t kTierCounts = 16;

template <int TPB>
__device__ inline void tier_partial(const uint8_t *tier, uint32_t n, uint32_t part, uint32_t nparts,
                                    uint32_t *out, uint32_t *s_w /* [TPB / 64][16] LDS */)
{
    const uint32_t t = threadIdx.x, lane = (uint32_t)lane_id(), w = t >> 6;
    const uint32_t lo = (uint32_t)((uint64_t)part * n / nparts), hi = (uint32_t)((uint64_t)(part + 1) * n / nparts);
    uint32_t c[kTierCounts];
#pragma unroll
    for (uint32_t q = 0; q < kTierCounts; q++) c[q] = 0;
    for (uint32_t i = lo + t; i < hi; i += TPB) {
        uint32_t q = tier[i];
        q = q < kTierCounts ? q : kTierCounts - 1u;
#pragma unroll
        for (uint32_t qq = 0; qq < kTierCounts; qq++) c[qq] += q == qq ? 1u : 0u;
    }
#pragma unroll
    for (uint32_t q = 0; q < kTierCounts; q++) {
        const uint32_t s = wave_sum(c[q]);
        if (lane == 0) s_w[w * kTierCounts + q] = s;
    }
    __syncthreads();
    if (t < kTierCounts) {
        uint32_t s = 0;
        for (uint32_t q = 0; q < (uint32_t)(TPB / 64); q++) s += s_w[q * kTierCounts + t];
        out[(uint64_t)part * kTierCounts + t] = s;
    }
}

}  // namespace ds
