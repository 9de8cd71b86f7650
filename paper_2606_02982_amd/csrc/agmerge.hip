// Aging Priority above the sample-sort limit as a merge of sorted runs
// (Sec. "Aging Priority Scheduling"; internal to the library).
//
// The aged score max(floor, p - rate * max(0, t_now - arrival)) is, for a
// fixed priority p, a non-decreasing function of the arrival: every
// operation (subtraction from t_now, the clamp at 0, the product, the
// subtraction from p, the clamp at the floor) is monotone and IEEE rounding
// keeps it so. Along the FIFO sequence the requests of one priority class
// (the tiers sharing a priority) are therefore already in Aging order, by
// (score, FIFO rank). The Aging order is the merge of those K <= 16 runs,
// with no comparison sort:
//   k_am_count  per tile of 4096 FIFO positions: each class's count
//   k_am_scan   one block: each tile's offset inside each class's run and
//               the runs' starts
//   k_am_place  per tile: each position's aged score (ordered bits) and FIFO
//               position go to its class run, stably
//   k_am_merge  ceil(log2 K) rounds (one when K = 1): adjacent runs are
//               merged pairwise by (score, FIFO position), merge-path
//               partitioned in output tiles of 2048 (a wave finds a tile's
//               split in about four 64-way probing steps, the block merges
//               in LDS); the last round writes the permutation and the key.
// Results are identical to sorting by (score, arrival, index): the scores
// are computed with the same operations as the other paths, and FIFO
// position order is (arrival, index) order.
#include <string.h>

#include "common.h"
#include "kernels.h"

namespace ds {
namespace {

constexpr int kAmTPB = 256;
constexpr uint32_t kAmTile = 4096;                 // FIFO positions per count/place block
constexpr uint32_t kAmRounds = kAmTile / kAmTPB;   // 16 positions per thread
constexpr uint32_t kAmCls = 16;
constexpr int kMgTPB = 256, kMgPer = 8;
constexpr uint32_t kMgTile = kMgTPB * kMgPer;       // outputs per merge block

struct AmArgs {
    SortInput in;            // arrival, tier, cls, prio, aging parameters; fifo = the FIFO permutation
    uint32_t n, tiles, K;
    uint32_t *cnt;           // [tiles][16]: counts, then each tile's offset in its class's run
    uint32_t *cstart;        // [17]: run starts (cstart[K..16] = n)
    uint64_t *rk[2];         // run keys (ping-pong)
    uint32_t *rp[2];         // run FIFO positions
    uint32_t *perm;
    double *key_out;         // per request, or null
    uint32_t *wait_status;   // zeroed by the first kernel (no waits here), or null
};

__device__ __forceinline__ uint32_t am_tier(const SortInput &in, uint32_t i)
{
    const uint32_t q = in.tier[i];
    return q < kAmCls ? q : kAmCls - 1u;
}

// The aged score, each operation rounded separately (no fused multiply-add).
__device__ __forceinline__ double am_aged(const SortInput &in, uint32_t i, uint32_t q)
{
    double w = in.t_now - in.arrival[i];
    if (w < 0.0) w = 0.0;
    const double d = in.aging_rate * w;
    double e = in.prio[q] - d;
    if (e < in.aging_floor) e = in.aging_floor;
    return e;
}

// Lanes of the wave holding the same 4-bit class (ok lanes only).
__device__ __forceinline__ uint64_t class_peers(uint32_t c, bool ok)
{
    uint64_t peers = __ballot(ok);
#pragma unroll
    for (int bb = 0; bb < 4; bb++) {
        const bool bit = (c >> bb) & 1u;
        const uint64_t m = __ballot(bit);
        peers &= bit ? m : ~m;
    }
    return peers;
}

__global__ __launch_bounds__(kAmTPB) void k_am_count(AmArgs a)
{
    __shared__ uint32_t c[kAmCls];
    const uint32_t t = threadIdx.x, tile = blockIdx.x;
    if (a.wait_status && tile == 0 && t == 0) *a.wait_status = 0;
    if (t < kAmCls) c[t] = 0;
    __syncthreads();
    const uint32_t base = tile * kAmTile;
    uint32_t cl[kAmRounds];
#pragma unroll
    for (uint32_t r = 0; r < kAmRounds; r++) {
        const uint32_t j = base + r * kAmTPB + t;
        uint32_t i = j < a.n ? a.in.fifo[j] : 0u;
        i = i < a.n ? i : 0u;
        cl[r] = j < a.n ? a.in.cls[am_tier(a.in, i)] : kAmCls;
    }
#pragma unroll
    for (uint32_t r = 0; r < kAmRounds; r++) {
        const bool ok = cl[r] < kAmCls;
        const uint64_t peers = class_peers(cl[r], ok);
        if (ok && (peers & lanemask_lt()) == 0) atomicAdd(&c[cl[r]], (uint32_t)__popcll(peers));
    }
    __syncthreads();
    if (t < kAmCls) a.cnt[tile * kAmCls + t] = c[t];
}

// Wave w handles class w: its total over the tiles first, then (with every
// class's total known, so with the class's start) the exclusive scan over
// the tiles. Each lane takes contiguous runs of 16 tiles, all their loads in
// flight together.
__global__ __launch_bounds__(1024) void k_am_scan(AmArgs a)
{
    constexpr uint32_t kPer = 16;   // tiles per lane and step
    __shared__ uint32_t tot[kAmCls];
    const uint32_t w = threadIdx.x >> 6;
    const int lane = lane_id();
    uint32_t sum = 0;
    for (uint32_t t0 = 0; t0 < a.tiles; t0 += 64 * kPer) {
        const uint32_t tl0 = t0 + (uint32_t)lane * kPer;
#pragma unroll
        for (uint32_t k = 0; k < kPer; k++) sum += tl0 + k < a.tiles ? a.cnt[(tl0 + k) * kAmCls + w] : 0u;
    }
    sum = wave_sum(sum);
    if (lane == 0) tot[w] = sum;
    __syncthreads();
    uint32_t run = 0;
    for (uint32_t k = 0; k < w; k++) run += tot[k];
    if (lane == 0) a.cstart[w] = run;
    if (threadIdx.x == 0) a.cstart[kAmCls] = a.n;
    for (uint32_t t0 = 0; t0 < a.tiles; t0 += 64 * kPer) {
        const uint32_t tl0 = t0 + (uint32_t)lane * kPer;
        uint32_t x[kPer];
#pragma unroll
        for (uint32_t k = 0; k < kPer; k++) x[k] = tl0 + k < a.tiles ? a.cnt[(tl0 + k) * kAmCls + w] : 0u;
        uint32_t part = 0;
#pragma unroll
        for (uint32_t k = 0; k < kPer; k++) part += x[k];
        const uint32_t incl = wave_incl_scan_dpp(part);
        uint32_t ex = run + incl - part;
#pragma unroll
        for (uint32_t k = 0; k < kPer; k++) {
            if (tl0 + k < a.tiles) a.cnt[(tl0 + k) * kAmCls + w] = ex;
            ex += x[k];
        }
        run += readlane32(incl, 63);
    }
}

__global__ __launch_bounds__(kAmTPB) void k_am_place(AmArgs a)
{
    constexpr int kWaves = kAmTPB / 64;
    // per round and wave, each class's count; then each one's offset in
    // its class's run (the tile's offset plus everything before it)
    __shared__ uint32_t pre[kAmRounds][kWaves][kAmCls];
    const uint32_t t = threadIdx.x, tile = blockIdx.x;
    const int w = (int)(t >> 6), lane = lane_id();
    const uint32_t base = tile * kAmTile;
    // the loads of all rounds first
    uint32_t cl[kAmRounds];
    uint64_t key[kAmRounds];
#pragma unroll
    for (uint32_t r = 0; r < kAmRounds; r++) {
        const uint32_t j = base + r * kAmTPB + t;
        uint32_t i = j < a.n ? a.in.fifo[j] : 0u;
        i = i < a.n ? i : 0u;
        const uint32_t q = am_tier(a.in, i);
        cl[r] = j < a.n ? a.in.cls[q] : kAmCls;
        key[r] = ordered_bits(am_aged(a.in, i, q));
    }
    uint32_t below[kAmRounds];
#pragma unroll
    for (uint32_t r = 0; r < kAmRounds; r++) {
        const bool ok = cl[r] < kAmCls;
        below[r] = (uint32_t)__popcll(class_peers(cl[r], ok) & lanemask_lt());
        uint32_t mine = 0;
#pragma unroll
        for (uint32_t k = 0; k < kAmCls; k++) {
            const uint32_t c = (uint32_t)__popcll(__ballot(cl[r] == k));
            mine = (uint32_t)lane == k ? c : mine;
        }
        if (lane < (int)kAmCls) pre[r][w][lane] = mine;
    }
    __syncthreads();
    if (t < kAmCls) {
        uint32_t s = a.cnt[tile * kAmCls + t];
        for (uint32_t r = 0; r < kAmRounds; r++)
            for (int v = 0; v < kWaves; v++) {
                const uint32_t x = pre[r][v][t];
                pre[r][v][t] = s;
                s += x;
            }
    }
    __syncthreads();
#pragma unroll
    for (uint32_t r = 0; r < kAmRounds; r++) {
        if (cl[r] < kAmCls) {
            const uint32_t pos = pre[r][w][cl[r]] + below[r];
            a.rk[0][pos] = key[r];
            a.rp[0][pos] = base + r * kAmTPB + t;
        }
    }
}

__device__ __forceinline__ bool am_less(uint64_t ka, uint32_t pa, uint64_t kb, uint32_t pb)
{
    return ka < kb || (ka == kb && pa < pb);
}

// Merge path: the number of A entries among the first d outputs of the merge
// of A (na entries) and B (nb), found by one wave in 64-way probing steps.
// Run-relative indices; A and B are the global arrays at their starts.
__device__ inline uint32_t merge_split(const uint64_t *ak, const uint32_t *ap, uint32_t na,
                                       const uint64_t *bk, const uint32_t *bp, uint32_t nb, uint32_t d)
{
    uint32_t lo = d > nb ? d - nb : 0u, hi = d < na ? d : na;
    const uint32_t lane = (uint32_t)lane_id();
    // smallest i in [lo, hi] with not (A[i] < B[d - 1 - i]); true for a prefix
    while (hi > lo) {
        const uint32_t span = hi - lo;
        const uint32_t m = lo + (uint32_t)(((uint64_t)span * lane) >> 6);   // lo <= m < hi
        // (the positions are read only on a tie of the keys)
        const uint64_t ka = ak[m], kb = bk[d - 1u - m];
        const bool p = ka < kb || (ka == kb && ap[m] < bp[d - 1u - m]);
        const uint32_t f = (uint32_t)__popcll(__ballot(p));   // probes 0..f-1 hold, f.. do not
        const uint32_t mf1 = f ? lo + (uint32_t)(((uint64_t)span * (f - 1u)) >> 6) : 0u;
        const uint32_t mf = f < 64u ? lo + (uint32_t)(((uint64_t)span * f) >> 6) : hi;
        const uint32_t nlo = f ? mf1 + 1u : lo;
        hi = f < 64u ? mf : hi;
        lo = nlo;
    }
    return lo;
}

// One round: run pairs of `span` classes each (run i covers classes
// [i span, (i + 1) span)); pair p merges runs 2p and 2p + 1 into
// [cstart[2p span], cstart[(2p + 2) span]). Blocks are handed to the pairs'
// output tiles in order; the grid covers every pair's tiles.
__global__ __launch_bounds__(kMgTPB) void k_am_merge(AmArgs a, uint32_t span, uint32_t src, uint32_t last)
{
    __shared__ uint64_t sk[kMgTile];
    __shared__ uint32_t sp[kMgTile];
    __shared__ uint64_t ok[kMgTile];
    __shared__ uint32_t op[kMgTile];
    __shared__ uint32_t s_split[2];
    const uint32_t t = threadIdx.x;
    const int w = (int)(t >> 6);
    uint32_t b = blockIdx.x, lo = 0, mid = 0, hi = 0;
    bool found = false;
    for (uint32_t p = 0; 2u * p * span < a.K; p++) {
        const uint32_t c0 = 2u * p * span, c1 = c0 + span, c2 = c0 + 2u * span;
        lo = a.cstart[c0 < a.K ? c0 : a.K];
        mid = a.cstart[c1 < a.K ? c1 : a.K];
        hi = a.cstart[c2 < a.K ? c2 : a.K];
        const uint32_t tiles = (hi - lo + kMgTile - 1u) / kMgTile;
        if (b < tiles) {
            found = true;
            break;
        }
        b -= tiles;
    }
    if (!found) return;   // the same for the whole block
    const uint32_t na = mid - lo, nb = hi - mid, len = hi - lo;
    const uint32_t d0 = b * kMgTile, d1 = d0 + kMgTile < len ? d0 + kMgTile : len;
    const uint64_t *rk = a.rk[src];
    const uint32_t *rp = a.rp[src];
    if (w < 2) {
        const uint32_t s = merge_split(rk + lo, rp + lo, na, rk + mid, rp + mid, nb, w == 0 ? d0 : d1);
        if (lane_id() == 0) s_split[w] = s;
    }
    __syncthreads();
    const uint32_t i0 = s_split[0], i1 = s_split[1];
    const uint32_t ta = i1 - i0, cnt = d1 - d0;   // tile: A[i0, i1), B[d0 - i0, d1 - i1)
    const uint32_t j0 = d0 - i0;
    for (uint32_t x = t; x < cnt; x += kMgTPB) {
        const uint32_t g = x < ta ? lo + i0 + x : mid + j0 + (x - ta);
        sk[x] = rk[g];
        sp[x] = rp[g];
    }
    __syncthreads();
    // each thread: outputs [dl, dl + kMgPer) of the tile
    const uint32_t dl = t * kMgPer;
    if (dl < cnt) {
        const uint32_t tb = cnt - ta;
        uint32_t l = dl > tb ? dl - tb : 0u, h = dl < ta ? dl : ta;
        while (l < h) {
            const uint32_t m = (l + h) >> 1;
            if (am_less(sk[m], sp[m], sk[ta + dl - 1u - m], sp[ta + dl - 1u - m])) l = m + 1u;
            else h = m;
        }
        uint32_t ia = l, ib = dl - l;
        const uint32_t e = dl + kMgPer < cnt ? dl + kMgPer : cnt;
        for (uint32_t o = dl; o < e; o++) {
            bool take_a;
            if (ia >= ta) take_a = false;
            else if (ib >= tb) take_a = true;
            else take_a = am_less(sk[ia], sp[ia], sk[ta + ib], sp[ta + ib]);
            const uint32_t s = take_a ? ia++ : ta + ib++;
            ok[o] = sk[s];
            op[o] = sp[s];
        }
    }
    __syncthreads();
    const uint32_t dst = src ^ 1u;
    for (uint32_t x = t; x < cnt; x += kMgTPB) {
        const uint32_t g = lo + d0 + x;
        if (last) {
            uint32_t i = a.in.fifo[op[x]];
            i = i < a.n ? i : 0u;
            a.perm[g] = i;
            if (a.key_out) a.key_out[i] = am_aged(a.in, i, am_tier(a.in, i));
        } else {
            a.rk[dst][g] = ok[x];
            a.rp[dst][g] = op[x];
        }
    }
}

// ceil(log2 K) merge rounds over the runs in a.rk[0] / a.rp[0] (one copying
// round when K = 1); the last one writes the permutation and the key.
void merge_rounds(const AmArgs &a, hipStream_t s)
{
    uint32_t rounds = 0;
    while ((1u << rounds) < a.K) rounds++;
    if (rounds == 0) rounds = 1;
    // blocks: every pair's tiles (at most n / kMgTile + one partial tile per pair)
    const uint32_t blocks = (uint32_t)cdiv(a.n, kMgTile) + (a.K + 1) / 2;
    uint32_t src = 0;
    for (uint32_t r = 0; r < rounds; r++) {
        hipLaunchKernelGGL(k_am_merge, dim3(blocks), dim3(kMgTPB), 0, s, a, 1u << r, src,
                           r + 1 == rounds ? 1u : 0u);
        src ^= 1u;
    }
}

}  // namespace

size_t am_partition_ws_bytes(uint64_t n)
{
    const uint64_t tiles = cdiv(n ? n : 1, kAmTile);
    return align_up(tiles * kAmCls * 4, 256) + align_up(n * 8, 256);
}

hipError_t am_partition(const SortInput &in, uint32_t *run_pos, uint32_t *run_start, void *ws, hipStream_t s)
{
    const uint32_t n = in.n;
    if (n == 0) return hipSuccess;
    if (n > kAmMaxN || !in.fifo) return hipErrorInvalidValue;
    AmArgs a;
    memset(&a, 0, sizeof(a));
    a.in = in;
    a.n = n;
    a.tiles = (uint32_t)cdiv(n, kAmTile);
    a.K = kAmCls;
    uint8_t *p = static_cast<uint8_t *>(ws);
    a.cnt = reinterpret_cast<uint32_t *>(p);
    p += align_up((uint64_t)a.tiles * kAmCls * 4, 256);
    a.rk[0] = reinterpret_cast<uint64_t *>(p);   // the scores are not used here
    a.rp[0] = run_pos;
    a.cstart = run_start;
    hipLaunchKernelGGL(k_am_count, dim3(a.tiles), dim3(kAmTPB), 0, s, a);
    hipLaunchKernelGGL(k_am_scan, dim3(1), dim3(1024), 0, s, a);
    hipLaunchKernelGGL(k_am_place, dim3(a.tiles), dim3(kAmTPB), 0, s, a);
    return hipGetLastError();
}

size_t am_ws_bytes(uint64_t n)
{
    const uint64_t tiles = cdiv(n ? n : 1, kAmTile);
    return align_up(tiles * kAmCls * 4, 256) + align_up((kAmCls + 1) * 4, 256) + 2 * align_up(n * 8, 256) +
           2 * align_up(n * 4, 256);
}

hipError_t am_launch(const SortInput &in, uint32_t n_classes, uint32_t *perm, double *key_out, void *ws,
                     hipStream_t s, uint32_t *wait_status)
{
    const uint32_t n = in.n;
    if (n == 0) return hipSuccess;
    if (n > kAmMaxN || !in.fifo || n_classes < 1 || n_classes > kAmCls) return hipErrorInvalidValue;
    AmArgs a;
    a.in = in;
    a.n = n;
    a.tiles = (uint32_t)cdiv(n, kAmTile);
    a.K = n_classes;
    uint8_t *p = static_cast<uint8_t *>(ws);
    a.cnt = reinterpret_cast<uint32_t *>(p);
    p += align_up((uint64_t)a.tiles * kAmCls * 4, 256);
    a.cstart = reinterpret_cast<uint32_t *>(p);
    p += align_up((kAmCls + 1) * 4, 256);
    for (int k = 0; k < 2; k++) {
        a.rk[k] = reinterpret_cast<uint64_t *>(p);
        p += align_up((uint64_t)n * 8, 256);
    }
    for (int k = 0; k < 2; k++) {
        a.rp[k] = reinterpret_cast<uint32_t *>(p);
        p += align_up((uint64_t)n * 4, 256);
    }
    a.perm = perm;
    a.key_out = key_out;
    a.wait_status = wait_status;
    hipLaunchKernelGGL(k_am_count, dim3(a.tiles), dim3(kAmTPB), 0, s, a);
    hipLaunchKernelGGL(k_am_scan, dim3(1), dim3(1024), 0, s, a);
    hipLaunchKernelGGL(k_am_place, dim3(a.tiles), dim3(kAmTPB), 0, s, a);
    merge_rounds(a, s);
    return hipGetLastError();
}

hipError_t am_merge_launch(const SortInput &in, uint32_t n_classes, uint32_t *cstart, uint64_t *const rk[2],
                           uint32_t *const rp[2], uint32_t *perm, double *key_out, hipStream_t s)
{
    const uint32_t n = in.n;
    if (n == 0) return hipSuccess;
    if (n > kAmMaxN || !in.fifo || n_classes < 1 || n_classes > kAmCls) return hipErrorInvalidValue;
    AmArgs a;
    memset(&a, 0, sizeof(a));
    a.in = in;
    a.n = n;
    a.K = n_classes;
    a.cstart = cstart;
    for (int k = 0; k < 2; k++) {
        a.rk[k] = rk[k];
        a.rp[k] = rp[k];
    }
    a.perm = perm;
    a.key_out = key_out;
    merge_rounds(a, s);
    return hipGetLastError();
}

}  // namespace ds
