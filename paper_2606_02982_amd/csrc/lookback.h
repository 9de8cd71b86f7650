// Decoupled look-back over tiles and the digit scan used by the tile passes
// of the sorts (internal to the library).
//
// Tile t publishes, for each of 256 digits, a status word: flag bits in the
// top two bits (aggregate only, or inclusive prefix) and a 30-bit count.
#pragma once

#include "common.h"

namespace ds {

constexpr uint32_t kAgg = 1u << 30;          // the word holds this tile's count only
constexpr uint32_t kPre = 2u << 30;          // the word holds the inclusive prefix
constexpr uint32_t kValMask = (1u << 30) - 1u;
constexpr uint32_t kSpinLimit = 1u << 22;    // bounded waits (never reached in normal runs:
                                             // about 0.2 s of sleeps)

// Sum of digit t's counts over the tiles before `tile` (tile j's words at
// st[j * kStride + digit]). Tiles publish their own count as soon as they
// have ranked their keys, so by the time a tile looks back its predecessors'
// counts are normally all there: windows of 16 predecessors are loaded at
// once and summed back to the first inclusive prefix. The wait for an
// unpublished tile is bounded (spin_limit sleeps without progress) and
// reported through err; spin_limit 0 gives up before the first load, so that
// the error path can be exercised with every kernel still exiting normally.
template <uint32_t kStride = 256>
__device__ inline uint32_t look_back(const uint32_t *st, uint32_t tile, uint32_t t, uint32_t *err,
                                     uint32_t spin_limit = kSpinLimit)
{
    constexpr int kWin = 16;
    if (spin_limit == 0) {
        if (tile > 0) atomicOr(err, 1u);
        return 0;
    }
    uint32_t prefix = 0;
    int64_t j = (int64_t)tile - 1;   // nearest predecessor not yet summed
    uint32_t spins = 0;
    while (j >= 0) {
        uint32_t x[kWin];
#pragma unroll
        for (int k = 0; k < kWin; k++) {
            int64_t jj = j - k >= 0 ? j - k : 0;
            x[k] = ld_relaxed(&st[(uint64_t)jj * kStride + t]);
        }
        bool done = false, stop = false;
        int used = 0;
#pragma unroll
        for (int k = 0; k < kWin; k++) {
            const bool valid = !done && !stop && j - k >= 0;
            const uint32_t flag = x[k] & ~kValMask;
            stop = stop || (valid && flag == 0);                 // not published yet
            const bool take = valid && flag != 0;
            prefix += take ? (x[k] & kValMask) : 0u;
            used = take ? k + 1 : used;
            done = done || (take && flag == kPre);
        }
        if (done) break;
        j -= used;
        if (used == 0) {
            __builtin_amdgcn_s_sleep(1);
            if (++spins > spin_limit) {
                atomicOr(err, 1u);
                break;
            }
        }
    }
    return prefix;
}

// Exclusive scan of the values of threads 0..255 over a block of TPB >= 256
// threads (every thread calls it; the result is meaningful for t < 256).
template <int TPB>
__device__ inline uint32_t block_excl_scan_digits(uint32_t x, uint32_t *tmp4)
{
    const uint32_t incl = wave_incl_scan_dpp(x);
    const int w = threadIdx.x >> 6;
    if (lane_id() == 63 && w < 4) tmp4[w] = incl;
    __syncthreads();
    uint32_t off = 0;
    for (int k = 0; k < w && k < 4; k++) off += tmp4[k];
    __syncthreads();
    return off + incl - x;
}

// Stable rank of an 8-bit digit among the keys of one wave, round by round:
// `peers` is the set of lanes of this round holding the same digit, `below`
// the number of them in lower lanes.
__device__ __forceinline__ uint64_t digit_peers(uint32_t dg, bool ok)
{
    uint64_t peers = __ballot(ok);
#pragma unroll
    for (int bb = 0; bb < 8; bb++) {
        const bool bit = (dg >> bb) & 1u;
        const uint64_t m = __ballot(bit);
        peers &= bit ? m : ~m;
    }
    return peers;
}

}  // namespace ds
