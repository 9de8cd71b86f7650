// Dispatch orders of kSsMaxN < n <= kLsMaxN requests (Sec. "Scheduling
// Engine"): one sample sort per policy over a sequence of positions j, by
// the pair (key(j), j), which is the stable order by key. FIFO sorts the
// requests by arrival; SJF (and Aging) sort the FIFO sequence by budget (or
// aged score), so that ties keep FIFO order. Keys and values are those of
// produce() (keys.h).
//
//   k_ls_gather   the keys of S = 8 per bucket positions, one in each of S
//                 equal strata of [0, n) (so the sample is in sequence order),
//                 and each wave's 64 of them sorted (a bitonic network).
//   k_ls_sample   each sample's rank by counting the samples below it, the
//                 count of each group of 64 samples spread over four blocks
//                 (each staging a quarter of the sorted 64-sample blocks in
//                 LDS, one binary search per block).
//   k_ls_place    each sample at its rank (the four counts added): the
//                 sorted sample, of which every (S/B)-th pair is one of the
//                 B - 1 splitters.
//   k_ls_count    per tile of 4096 positions: each position's bucket (a
//                 descent of the splitters' search tree), stored, and the
//                 tile's count of each bucket; the per-request key output.
//   k_ls_scan     per bucket: exclusive prefix of its counts over the tiles
//                 (each tile's first slot in the bucket) and the bucket's size.
//   k_ls_scatter  per tile: the buckets' regions (exclusive scan of the
//                 sizes, in every block) and the tile's pairs grouped by
//                 bucket in LDS, then written in runs at the tile's slots. A
//                 bucket's pairs need no particular order inside it: the
//                 pair order is total (j is unique), so the bucket sort
//                 alone fixes the result.
//   k_ls_bucket   one block per bucket: a bucket of at most kLsCap pairs is
//                 ranked in LDS (bins over its key range, counting inside a
//                 bin; stable byte passes over j and then the key when a bin
//                 is crowded); a larger one (only for inputs arranged against
//                 the sampling) is sorted by the same byte passes through
//                 global memory, chunk by chunk. The values go to their
//                 places in the output.
// No atomics on global memory and no wait on another block; the bucket
// sizes are exact, so nothing overflows.
#include <string.h>

#include "common.h"
#include "kernels.h"
#include "keys.h"
#include "lookback.h"
#include "wrrplan.h"

namespace ds {
namespace {

constexpr uint32_t kLsAvg = 1024;                  // target pairs per bucket
constexpr uint32_t kLsMaxB = kLsMaxN / kLsAvg;     // 1024 buckets at most
constexpr uint32_t kLsOver = 8;                    // samples per bucket
constexpr uint32_t kLsMaxS = kLsMaxB * kLsOver;    // 8192
constexpr uint32_t kLsCap = 4096;                  // buckets ranked in LDS up to this size
constexpr uint32_t kJBits = 20;                    // positions j < 2^20
constexpr uint32_t kJMask = (1u << kJBits) - 1u;
static_assert(kLsMaxN <= (1u << kJBits), "a position fits its field");
static_assert(kLsMaxB <= (1u << (32 - kJBits)), "a bucket index fits above the position");

constexpr int kTT = 512, kTR = 8;                  // count and scatter tiles
constexpr uint32_t kTile = kTT * kTR;              // 4096 positions
constexpr int kBT = 512, kBW = kBT / 64, kBR = kLsCap / kBT;   // k_ls_bucket
constexpr uint32_t kBinBits = 11, kBins = 1u << kBinBits;
constexpr uint32_t kBinMax = 256;                  // larger bins: byte passes instead

constexpr uint32_t kLsMaxRows = 4;                 // sorts and partitions of one batch
constexpr uint32_t kQ = 16;                        // partition digits (tiers or classes)

// One row of a batch: a sort (Fifo, Budget, Aging: buckets by sampled
// splitters) or a partition (Class, Tier: the stable partition of the
// sequence by a digit below kQ, placed straight at the policy's positions).
struct LsRow {
    SortKind kind;
    uint32_t B;            // buckets, or kQ digits
    uint32_t S, hgt;       // sorts: samples and the splitter tree's height
    double *key_out;       // per-request key (or NULL)
    uint32_t *out;         // n values in order
    uint32_t *size;        // [B] pairs per bucket (requests per digit)
    uint32_t *start;       // [B] first place of each bucket's region (each digit's range)
    uint32_t *tcnt;        // [tiles][B] each tile's count of each bucket, then its first slot there
    uint16_t *bid;         // [n] bucket of each position (sorts)
    uint32_t by_req;       // the sample's keys are the budgets of the sampled requests
                           // (request index standing in for the FIFO position)
    uint64_t *raw_k;       // [S] the sample's keys in sample order
    uint32_t *rpart;       // [kSmP][S] each part's count of samples below each sample
    uint64_t *smp_k;       // [S] the sample in order
    uint32_t *smp_j;
    uint64_t *rk[2];       // [n] bucket regions, and the large-bucket path's second buffer
    uint32_t *rj[2];
    uint32_t *rv;          // [n] sorts over in.fifo: each region entry's value (or NULL)
    uint8_t *rt;           // [n] the FIFO sort, when it writes copies: each entry's tier
    double *rb;            //     and budget (or NULL)
};

struct LsArgs {
    SortInput in;
    LsCopies pf;           // the inputs in FIFO order (rows over in.fifo read them), or NULL:
                           // then the keys are gathered through in.fifo
    LsCopies cp;           // the FIFO sort writes those copies here (or NULL)
    LsRuns runs;           // the Class row lays out the Aging runs here (or NULL)
    uint32_t n, tiles;
    uint32_t nrows;        // rows [0, nsort) are sorts, the rest partitions
    uint32_t nsort;
    uint32_t nsamp;        // rows that draw their splitters in this call: r[srow[0 .. nsamp)]
    uint32_t srow[kLsMaxRows];
    WrrPlan *plan;         // Tier, smooth interleaving: the period table (built by the scan)
    uint32_t *tpos;        // its start-up positions
    LsRow r[kLsMaxRows];
};

__device__ __forceinline__ bool is_part(SortKind k) { return k == SortKind::Class || k == SortKind::Tier; }

// Position of sample s: in the s-th of S equal strata of [0, n), the offset
// picked by a fixed integer hash (so that sampling does not lock onto
// periodic inputs). Increasing in s.
__device__ __forceinline__ uint32_t ls_pos(uint32_t s, uint32_t n, uint32_t S)
{
    const uint32_t lo = (uint32_t)((uint64_t)s * n / S), hi = (uint32_t)((uint64_t)(s + 1) * n / S);
    uint32_t h = s * 0x9E3779B1u + 0x7F4A7C15u;
    h ^= h >> 15;
    h *= 0x85EBCA77u;
    h ^= h >> 13;
    return lo + h % (hi - lo);   // hi > lo since S <= n
}

// The aged score of a request with arrival x and tier q, each operation
// rounded separately (no fused multiply-add), as in produce().
__device__ __forceinline__ double ls_aged(const SortInput &in, double x, uint32_t q)
{
    double w = in.t_now - x;
    if (w < 0.0) w = 0.0;
    const double d = in.aging_rate * w;
    double e = in.prio[q] - d;
    if (e < in.aging_floor) e = in.aging_floor;
    return e;
}

// The key of position j of the row's sequence (the digit, for a partition).
__device__ __forceinline__ uint64_t ls_key(const LsArgs &a, const LsRow &R, uint32_t j)
{
    if (R.kind != SortKind::Fifo && a.pf.tier) {
        const uint32_t q0 = a.pf.tier[j], q = q0 < kQ ? q0 : kQ - 1u;
        switch (R.kind) {
        case SortKind::Budget: return ordered_bits(a.pf.bud[j]);
        case SortKind::Aging: return ordered_bits(ls_aged(a.in, a.pf.arr[j], q));
        case SortKind::Class: return a.in.cls[q];
        default: return q;   // Tier
        }
    }
    uint64_t k;
    uint32_t v;
    produce(a.in, R.kind, nullptr, a.n, j, k, v);
    return k;
}

// The per-request key output of request i (Weighted's round is written
// where the request is placed).
__device__ __forceinline__ void ls_key_out(const LsArgs &a, const LsRow &R, uint32_t i)
{
    const uint32_t q0 = R.kind == SortKind::Fifo || R.kind == SortKind::Budget ? 0u : a.in.tier[i];
    const uint32_t q = q0 < kQ ? q0 : kQ - 1u;
    switch (R.kind) {
    case SortKind::Fifo: R.key_out[i] = a.in.arrival[i]; break;
    case SortKind::Budget: R.key_out[i] = a.in.budget[i]; break;
    case SortKind::Aging: R.key_out[i] = ls_aged(a.in, a.in.arrival[i], q); break;
    case SortKind::Class: R.key_out[i] = a.in.prio[q]; break;
    default: break;
    }
}

// The value position j contributes to the output.
__device__ __forceinline__ uint32_t ls_value(const LsArgs &a, const LsRow &R, uint32_t j)
{
    if (R.kind == SortKind::Fifo) return j;
    const uint32_t i = a.in.fifo[j];
    return i < a.n ? i : 0u;
}

// A region entry's payload: its value, and for the FIFO sort's copies the
// request's tier and budget (carried from the scatter, or gathered).
struct LsPay {
    uint32_t v;
    uint8_t q;
    double b;
};

__device__ __forceinline__ LsPay ls_pay_region(const LsArgs &a, const LsRow &R, uint32_t g, uint32_t j)
{
    LsPay y;
    y.v = R.rv ? R.rv[g] : (R.kind == SortKind::Fifo ? j : 0u);
    y.q = R.rt ? R.rt[g] : 0;
    y.b = R.rb ? R.rb[g] : 0.0;
    return y;
}

__device__ __forceinline__ LsPay ls_pay_gather(const LsArgs &a, const LsRow &R, uint32_t j)
{
    LsPay y;
    y.v = ls_value(a, R, j);
    y.q = R.rt ? a.in.tier[j] : 0;
    y.b = R.rb ? a.in.budget[j] : 0.0;
    return y;
}

// Output place p of a sort gets an entry with key k: its value, and for the
// FIFO sort the request's inputs in FIFO order when they are wanted.
__device__ __forceinline__ void ls_emit(const LsArgs &a, const LsRow &R, uint32_t p, uint64_t k, const LsPay &y)
{
    R.out[p] = y.v;
    if (R.kind == SortKind::Fifo && a.cp.tier) {
        // the arrival back from its key (exact; a -0.0 comes back as +0.0,
        // which gives the same aged score)
        const uint64_t u = (k >> 63) ? (k & 0x7FFFFFFFFFFFFFFFull) : ~k;
        a.cp.arr[p] = __longlong_as_double((long long)u);
        a.cp.tier[p] = y.q;
        if (a.cp.bud) a.cp.bud[p] = y.b;
    }
}

__device__ __forceinline__ bool pair_less(uint64_t ka, uint32_t ja, uint64_t kb, uint32_t jb)
{
    return ka < kb || (ka == kb && ja < jb);
}

// Exclusive scan of one value per thread over a block of TPB threads
// (every thread calls it; wsum: TPB / 64 words of LDS). Ends with a barrier.
template <int TPB>
__device__ __forceinline__ uint32_t blk_excl_scan(uint32_t x, uint32_t *wsum)
{
    const int w = (int)(threadIdx.x >> 6);
    const uint32_t incl = wave_incl_scan_dpp(x);
    if (lane_id() == 63) wsum[w] = incl;
    __syncthreads();
    uint32_t off = 0;
    for (int q = 0; q < w; q++) off += wsum[q];
    __syncthreads();
    return off + incl - x;
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t x, int m)
{
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)x, m, 64);
    const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(x >> 32), m, 64);
    return ((uint64_t)hi << 32) | lo;
}

// The sample's keys in sample order (raw_k), and each wave's 64 samples
// sorted by (key, sample index) with a bitonic network across the lanes,
// stored as sorted blocks of 64 in smp_k / smp_j for the ranking (the
// placement overwrites them with the sorted sample).
__global__ __launch_bounds__(256) void k_ls_gather(LsArgs a)
{
    const LsRow &R = a.r[a.srow[blockIdx.y]];
    const uint32_t s = blockIdx.x * 256u + threadIdx.x;
    if (blockIdx.x * 256u + (threadIdx.x & ~63u) >= R.S) return;   // a whole wave past S (a multiple of 64)
    const uint32_t j = ls_pos(s, a.n, R.S);
    uint64_t k = R.by_req ? ordered_bits(a.in.budget[j]) : ls_key(a, R, j);
    R.raw_k[s] = k;
    uint32_t i = s;
    const uint32_t lane = (uint32_t)lane_id();
    for (uint32_t kk = 2; kk <= 64; kk <<= 1)
        for (uint32_t jj = kk >> 1; jj > 0; jj >>= 1) {
            const uint64_t pk = shfl_xor_u64(k, (int)jj);
            const uint32_t pi = (uint32_t)__shfl_xor((int)i, (int)jj, 64);
            const bool pl = pk < k || (pk == k && pi < i);   // the partner's pair is the smaller
            const bool up = (lane & kk) == 0, lower = (lane & jj) == 0;
            if (lower == up ? pl : !pl) {
                k = pk;
                i = pi;
            }
        }
    R.smp_k[s] = k;
    R.smp_j[s] = i;
}

constexpr int kSmT = 1024, kSmW = kSmT / 64;

// Ranks by counting, spread over kSmP blocks per group of 64 samples: block
// (g, p) stages part p of the sorted 64-sample blocks in LDS and counts, for
// each of the group's samples (one per lane), the part's samples below it
// by (key, sample index): one binary search per sorted block (each wave
// over a share of the part's blocks, the waves' counts added), stored as
// that part's count. Sample indices increase with the positions, so the
// order is the pair order by (key, position).
constexpr uint32_t kSmP = 4;

__global__ __launch_bounds__(kSmT) void k_ls_sample(LsArgs a)
{
    __shared__ uint64_t sk[kLsMaxS / kSmP];
    __shared__ uint16_t si[kLsMaxS / kSmP];
    __shared__ uint32_t part[kSmW][64];
    const LsRow &R = a.r[a.srow[blockIdx.y]];
    const uint32_t g = blockIdx.x / kSmP, pq = blockIdx.x % kSmP;
    if (g * 64u >= R.S) return;   // a row with a smaller sample than the grid is wide
    const uint32_t t = threadIdx.x, lane = (uint32_t)lane_id(), w = t >> 6, S = R.S;
    const uint32_t nb = S / 64u, b0 = pq * nb / kSmP, b1 = (pq + 1u) * nb / kSmP;   // sorted blocks [b0, b1)
    const uint32_t e0 = b0 * 64u, ne = (b1 - b0) * 64u;   // <= kLsMaxS / kSmP
    for (uint32_t x = t; x < ne; x += kSmT) {
        sk[x] = R.smp_k[e0 + x];
        si[x] = (uint16_t)R.smp_j[e0 + x];
    }
    const uint32_t s = g * 64u + lane;
    const uint64_t ks = R.raw_k[s];
    __syncthreads();
    uint32_t c = 0;
    for (uint32_t b = w; b < b1 - b0; b += kSmW) {
        // the block's pairs below (ks, s): steps of 32 .. 1, then the last one
        const uint32_t base = b * 64u;
        uint32_t pos = 0;
#pragma unroll
        for (uint32_t step = 32; step > 0; step >>= 1) {
            const uint32_t q = base + pos + step - 1u;
            const uint64_t x = sk[q];
            if (x < ks || (x == ks && si[q] < s)) pos += step;
        }
        const uint32_t q = base + pos;   // pos <= 63
        const uint64_t x = sk[q];
        if (x < ks || (x == ks && si[q] < s)) pos++;
        c += pos;
    }
    part[w][lane] = c;
    __syncthreads();
    if (w == 0) {
        uint32_t r = 0;
#pragma unroll
        for (int qq = 0; qq < kSmW; qq++) r += part[qq][lane];
        R.rpart[(uint64_t)pq * S + s] = r;
    }
}

// Each sample at its rank (the sum of its parts' counts).
__global__ __launch_bounds__(256) void k_ls_place(LsArgs a)
{
    const LsRow &R = a.r[a.srow[blockIdx.y]];
    const uint32_t s = blockIdx.x * 256u + threadIdx.x, S = R.S;
    if (s >= S) return;
    uint32_t r = 0;
#pragma unroll
    for (uint32_t p = 0; p < kSmP; p++) r += R.rpart[(uint64_t)p * S + s];
    R.smp_k[r] = R.raw_k[s];
    R.smp_j[r] = ls_pos(s, a.n, S);
}

// The splitters in breadth-first (Eytzinger) order of a complete search tree
// of height hgt: node e (1-based, depth d, p = e - 2^d) holds splitter
// i = (2 p + 1) 2^(hgt - d - 1) - 1, the sample of rank (i + 1) S / B;
// indices from B - 1 on hold the largest pair, above every real one.
__device__ __forceinline__ void ls_tree(const LsRow &R, uint64_t *tk, uint32_t *tj)
{
    const uint32_t nodes = 1u << R.hgt;
    for (uint32_t e = threadIdx.x + 1; e < nodes; e += blockDim.x) {
        const uint32_t d = 31u - (uint32_t)__clz((int)e), p = e - (1u << d);
        const uint32_t i = (2u * p + 1u) * (1u << (R.hgt - d - 1u)) - 1u;
        uint64_t k = ~0ull;
        uint32_t j = ~0u;
        if (i + 1u < R.B) {
            const uint32_t r = (i + 1u) * R.S / R.B;   // < S; (i + 1) S < 2^23
            k = R.smp_k[r];
            j = R.smp_j[r];
        }
        tk[e] = k;
        tj[e] = j;
    }
}

// A partition row's tile: the count of each digit, and the per-request keys
// (Priority: the tier's priority) in request order.
__device__ __forceinline__ void ls_count_part(const LsArgs &a, const LsRow &R, uint32_t *h)
{
    const uint32_t t = threadIdx.x, n = a.n, base = blockIdx.x * kTile;
    const uint32_t cnt = n - base < kTile ? n - base : kTile;
    uint32_t d[kTR];
#pragma unroll
    for (int r = 0; r < kTR; r++) {
        const uint32_t idx = (uint32_t)r * kTT + t;
        d[r] = idx < cnt ? (uint32_t)ls_key(a, R, base + idx) : kQ;   // kQ: no position
    }
    if (R.key_out && R.kind == SortKind::Class) {
#pragma unroll
        for (int r = 0; r < kTR; r++) {
            const uint32_t idx = (uint32_t)r * kTT + t;
            if (idx < cnt) ls_key_out(a, R, base + idx);
        }
    }
    if (t < kQ) h[t] = 0;
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kTR; r++)
        if (d[r] < kQ) atomicAdd(&h[d[r]], 1u);
    __syncthreads();
    if (t < kQ) R.tcnt[(uint64_t)blockIdx.x * kQ + t] = h[t];
}

__global__ __launch_bounds__(kTT) void k_ls_count(LsArgs a)
{
    __shared__ uint64_t tk[kLsMaxB];
    __shared__ uint32_t tj[kLsMaxB];
    __shared__ uint32_t h[kLsMaxB];
    const LsRow &R = a.r[blockIdx.y];
    const uint32_t t = threadIdx.x, n = a.n, base = blockIdx.x * kTile;
    const uint32_t cnt = n - base < kTile ? n - base : kTile;
    // (no waits here: the caller's status word is only cleared)
    if (blockIdx.x == 0 && blockIdx.y == 0 && t == 0 && a.in.wait.clear && a.in.wait.status)
        *a.in.wait.status = 0;
    if (is_part(R.kind)) {
        ls_count_part(a, R, h);
        return;
    }
    uint64_t k[kTR];
#pragma unroll
    for (int r = 0; r < kTR; r++) {
        const uint32_t idx = (uint32_t)r * kTT + t;
        const bool ok = idx < cnt;
        k[r] = ls_key(a, R, base + (ok ? idx : 0u));
    }
    // the per-request keys, in request order
    if (R.key_out) {
#pragma unroll
        for (int r = 0; r < kTR; r++)
            if ((uint32_t)r * kTT + t < cnt) ls_key_out(a, R, base + (uint32_t)r * kTT + t);
    }
    ls_tree(R, tk, tj);
    for (uint32_t i = t; i < R.B; i += kTT) h[i] = 0;
    __syncthreads();
    const uint32_t hgt = R.hgt;
    // bucket = splitters <= (key, j): hgt steps down the tree, the rounds
    // side by side so that their LDS reads overlap
    uint32_t node[kTR];
#pragma unroll
    for (int r = 0; r < kTR; r++) node[r] = 1;
    for (uint32_t l = 0; l < hgt; l++) {
#pragma unroll
        for (int r = 0; r < kTR; r++) {
            const uint32_t j = base + (uint32_t)r * kTT + t;
            node[r] = 2u * node[r] + (pair_less(k[r], j, tk[node[r]], tj[node[r]]) ? 0u : 1u);
        }
    }
#pragma unroll
    for (int r = 0; r < kTR; r++) {
        const uint32_t idx = (uint32_t)r * kTT + t;
        if (idx < cnt) {
            const uint32_t b = node[r] - (1u << hgt);
            R.bid[base + idx] = (uint16_t)b;
            atomicAdd(&h[b], 1u);
        }
    }
    __syncthreads();
    uint32_t *row = R.tcnt + (uint64_t)blockIdx.x * R.B;
    for (uint32_t b = t; b < R.B; b += kTT) row[b] = h[b];
}

// Block c: buckets 64 c .. 64 c + 63 over all tiles (at most 256), staged in
// LDS; wave w scans the columns w, w + 16, ... (four tiles per lane).
constexpr int kScT = 1024, kScW = kScT / 64;
constexpr uint32_t kMaxTiles = kLsMaxN / kTile;   // 256

__global__ __launch_bounds__(kScT) void k_ls_scan(LsArgs a)
{
    __shared__ uint32_t col[kMaxTiles][65];
    __shared__ uint32_t tot[64];
    __shared__ uint16_t per[kWrrMaxWeightSum];
    const LsRow &R = a.r[blockIdx.y];
    const uint32_t t = threadIdx.x, lane = (uint32_t)lane_id(), w = t >> 6;
    const uint32_t b0 = blockIdx.x * 64u, T = a.tiles, B = R.B;
    if (b0 >= B) return;   // a row with fewer buckets than the grid is wide
    constexpr int kPer = kMaxTiles * 64 / kScT;   // 16 loads per thread, in flight together
    {
        uint32_t x[kPer];
#pragma unroll
        for (int q = 0; q < kPer; q++) {
            const uint32_t i = (uint32_t)q * kScT + t, tl = i >> 6, bb = i & 63u;
            x[q] = tl < T && b0 + bb < B ? R.tcnt[(uint64_t)tl * B + b0 + bb] : 0u;
        }
#pragma unroll
        for (int q = 0; q < kPer; q++) {
            const uint32_t i = (uint32_t)q * kScT + t;
            col[i >> 6][i & 63u] = x[q];
        }
    }
    __syncthreads();
    for (uint32_t bb = w; bb < 64u; bb += kScW) {
        uint32_t v[4], sum = 0;
#pragma unroll
        for (int q = 0; q < 4; q++) {
            const uint32_t tl = 4u * lane + (uint32_t)q;
            v[q] = tl < T ? col[tl][bb] : 0u;
            sum += v[q];
        }
        const uint32_t incl = wave_incl_scan_dpp(sum);
        uint32_t ex = incl - sum;
#pragma unroll
        for (int q = 0; q < 4; q++) {
            const uint32_t tl = 4u * lane + (uint32_t)q;
            if (tl < T) col[tl][bb] = ex;
            ex += v[q];
        }
        if (lane == 63) {
            tot[bb] = incl;
            if (b0 + bb < B) R.size[b0 + bb] = incl;
        }
    }
    __syncthreads();
    if (is_part(R.kind) && w == 0) {
        // each digit's first place (Priority: the classes in order), and for
        // the smooth interleaving the period table of the tiers' counts
        const uint32_t x = lane < kQ ? tot[lane] : 0u;
        const uint32_t ex = wave_incl_scan_dpp(x) - x;
        if (lane <= kQ) R.start[lane] = ex;   // start[kQ] = n
        if (R.kind == SortKind::Tier && a.in.wrr_mode == kWrrSmooth) {
            const uint32_t nq = a.in.n_tiers < kWrrTiers ? a.in.n_tiers : kWrrTiers;
            const bool tl = lane < nq;
            wrr_plan_build(tl ? x : 0u, tl ? a.in.weight[lane] : 0u, per, a.plan, a.tpos);
        }
    }
#pragma unroll
    for (int q = 0; q < kPer; q++) {
        const uint32_t i = (uint32_t)q * kScT + t, tl = i >> 6, bb = i & 63u;
        if (tl < T && b0 + bb < B) R.tcnt[(uint64_t)tl * B + b0 + bb] = col[tl][bb];
    }
}

// A partition row's tile: each position's rank among the sequence's
// positions of its digit (the tile's first slot in the digit, from the scan,
// plus its stable rank in the tile: wave w holds the tile's positions
// 512 w .. 512 w + 511 in order, ranked round by round with ballots), then
// its place: Priority at the class's start plus that rank, Weighted at the
// round-robin position of the rank-th request of the tier.
__device__ __forceinline__ void ls_place_part(const LsArgs &a, const LsRow &R, uint32_t (*wc)[kQ], WrrPlanHead &wh)
{
    constexpr uint32_t kWK = 64u * kTR;
    const uint32_t t = threadIdx.x, n = a.n, base = blockIdx.x * kTile;
    const int w = (int)(t >> 6), lane = lane_id();
    const uint32_t cnt = n - base < kTile ? n - base : kTile;
    uint32_t d[kTR], v[kTR], rk[kTR];
#pragma unroll
    for (int r = 0; r < kTR; r++) {
        const uint32_t idx = (uint32_t)w * kWK + (uint32_t)r * 64u + (uint32_t)lane;
        const uint32_t j = base + (idx < cnt ? idx : 0u);
        d[r] = (uint32_t)ls_key(a, R, j);   // < kQ
        v[r] = ls_value(a, R, j);
    }
    if (t < (kTT / 64) * kQ) (&wc[0][0])[t] = 0;
    const bool smooth = R.kind == SortKind::Tier && a.in.wrr_mode == kWrrSmooth;
    if (smooth)
        for (uint32_t i = t; i < sizeof(WrrPlanHead) / 4; i += kTT)
            reinterpret_cast<uint32_t *>(&wh)[i] = reinterpret_cast<const uint32_t *>(&a.plan->h)[i];
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kTR; r++) {
        const uint32_t idx = (uint32_t)w * kWK + (uint32_t)r * 64u + (uint32_t)lane;
        const bool ok = idx < cnt;
        const uint64_t peers = digit_peers(d[r], ok);
        const uint32_t below = (uint32_t)__popcll(peers & lanemask_lt());
        const uint32_t old = ok ? wc[w][d[r]] : 0u;
        rk[r] = old + below;
        if (ok && below == 0) wc[w][d[r]] = old + (uint32_t)__popcll(peers);
        __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();
    if (t < kQ) {
        uint32_t acc = R.tcnt[(uint64_t)blockIdx.x * kQ + t];   // the tile's first slot in digit t
#pragma unroll
        for (int q = 0; q < kTT / 64; q++) {
            const uint32_t c = wc[q][t];
            wc[q][t] = acc;
            acc += c;
        }
    }
    __syncthreads();
    const uint32_t nq = a.in.n_tiers < kQ ? a.in.n_tiers : kQ;
#pragma unroll
    for (int r = 0; r < kTR; r++) {
        const uint32_t idx = (uint32_t)w * kWK + (uint32_t)r * 64u + (uint32_t)lane;
        if (idx >= cnt) continue;
        const uint32_t q = d[r], kd = wc[w][q] + rk[r];   // rank among the digit's requests
        if (R.kind == SortKind::Class) {
            const uint32_t pos = R.start[q] + kd;
            if (pos >= n) continue;
            if (R.out) R.out[pos] = v[r];
            if (a.runs.rk) {
                // the Aging run of the class: the aged score is monotone in
                // the arrival within a class, so the run is in Aging order
                const uint32_t j = base + idx;
                const uint32_t t0 = a.pf.tier ? a.pf.tier[j] : a.in.tier[v[r]];
                const double x = a.pf.arr ? a.pf.arr[j] : a.in.arrival[v[r]];
                a.runs.rk[pos] = ordered_bits(ls_aged(a.in, x, t0 < kQ ? t0 : kQ - 1u));
                a.runs.rp[pos] = j;
            }
            continue;
        }
        if (q >= nq) continue;   // a tier outside the contract: no place
        uint64_t pos, rnd;
        if (smooth) {
            uint32_t r32;
            pos = wrr_smooth_pos(wh, a.plan, a.tpos, a.in.weight[q], q, kd, r32);
            rnd = r32;
        } else if (a.in.wrr_mode == kWrrStride) {
            const uint32_t wq = a.in.weight[q] ? a.in.weight[q] : 1u;
            rnd = kd / wq;
            pos = wrr_stride_pos(q, kd, a.in.weight, nq, [&](uint32_t u) { return R.size[u]; });
        } else {
            pos = wrr_blocked_pos(q, kd, a.in.weight, nq, [&](uint32_t u) { return R.size[u]; }, rnd);
        }
        if (pos < n) R.out[pos] = v[r];
        if (R.key_out) R.key_out[v[r]] = (double)rnd;
    }
}

__global__ __launch_bounds__(kTT) void k_ls_scatter(LsArgs a)
{
    static_assert(2 * kTT == kLsMaxB, "two buckets per thread");
    __shared__ uint32_t h[kLsMaxB], texcl[kLsMaxB], gb[kLsMaxB];
    __shared__ uint64_t lk[kTile];
    __shared__ uint32_t lj[kTile];
    __shared__ uint16_t lb[kTile];
    __shared__ uint32_t wsum[kTT / 64];
    __shared__ uint32_t pwc[kTT / 64][kQ];
    __shared__ WrrPlanHead wh;
    const LsRow &R = a.r[blockIdx.y];
    if (is_part(R.kind)) {
        ls_place_part(a, R, pwc, wh);
        return;
    }
    const uint32_t t = threadIdx.x, n = a.n, B = R.B, base = blockIdx.x * kTile;
    const uint32_t cnt = n - base < kTile ? n - base : kTile;
    uint64_t k[kTR];
    uint32_t b[kTR], sl[kTR];
#pragma unroll
    for (int r = 0; r < kTR; r++) {
        const uint32_t idx = (uint32_t)r * kTT + t;
        const uint32_t j = base + (idx < cnt ? idx : 0u);
        k[r] = ls_key(a, R, j);
        b[r] = R.bid[j];
    }
    // the regions: exclusive scan of the sizes (thread t: buckets 2t, 2t + 1)
    const uint32_t b0 = 2u * t, b1 = b0 + 1u;
    const uint32_t z0 = b0 < B ? R.size[b0] : 0u, z1 = b1 < B ? R.size[b1] : 0u;
    h[b0] = 0;
    h[b1] = 0;
    const uint32_t rs = blk_excl_scan<kTT>(z0 + z1, wsum);   // (its barriers order the clears)
#pragma unroll
    for (int r = 0; r < kTR; r++) {
        const uint32_t idx = (uint32_t)r * kTT + t;
        sl[r] = idx < cnt ? atomicAdd(&h[b[r]], 1u) : 0u;
    }
    __syncthreads();
    const uint32_t h0 = h[b0], h1 = h[b1];
    const uint32_t te = blk_excl_scan<kTT>(h0 + h1, wsum);
    texcl[b0] = te;
    texcl[b1] = te + h0;
    if (blockIdx.x == 0) {
        if (b0 < B) R.start[b0] = rs;
        if (b1 < B) R.start[b1] = rs + z0;
    }
    const uint32_t *row = R.tcnt + (uint64_t)blockIdx.x * B;
    gb[b0] = rs + (b0 < B ? row[b0] : 0u);
    gb[b1] = rs + z0 + (b1 < B ? row[b1] : 0u);
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kTR; r++) {
        const uint32_t idx = (uint32_t)r * kTT + t;
        if (idx < cnt) {
            const uint32_t p = texcl[b[r]] + sl[r];
            lk[p] = k[r];
            lj[p] = (base + idx) | (b[r] << kJBits);
        }
    }
    __syncthreads();
    const bool pay = R.rv || R.rt;
    for (uint32_t s = t; s < cnt; s += kTT) {
        const uint32_t x = lj[s], bb = x >> kJBits;
        const uint32_t g = gb[bb] + (s - texcl[bb]);   // < n: a region holds its bucket's pairs
        R.rk[0][g] = lk[s];
        R.rj[0][g] = x & kJMask;
        if (pay) lb[s] = (uint16_t)bb;
    }
    if (!pay) return;
    // the payloads ride along the same way (read in sequence order, staged
    // in the same places, written in the same runs), so that the bucket sort
    // gathers nothing: the value of a sort over in.fifo, or the FIFO sort's
    // tier and budget
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kTR; r++) {
        const uint32_t idx = (uint32_t)r * kTT + t;
        if (idx < cnt) {
            const uint32_t p = texcl[b[r]] + sl[r], j = base + idx;
            if (R.rv) {
                lj[p] = ls_value(a, R, j);
            } else {
                lj[p] = a.in.tier[j];
                if (R.rb) lk[p] = (uint64_t)__double_as_longlong(a.in.budget[j]);
            }
        }
    }
    __syncthreads();
    for (uint32_t s = t; s < cnt; s += kTT) {
        const uint32_t bb = lb[s], g = gb[bb] + (s - texcl[bb]);
        if (R.rv) {
            R.rv[g] = lj[s];
        } else {
            R.rt[g] = (uint8_t)lj[s];
            if (R.rb) R.rb[g] = __longlong_as_double((long long)lk[s]);
        }
    }
}

struct BkLs {
    uint32_t bin[kBins + 1];
    uint64_t lk[kLsCap];
    uint32_t lj[kLsCap];
    uint32_t wc[kBW][256];        // per-wave digit counters of a byte pass
    uint32_t texcl[256];
    uint32_t dtot[256];
    uint32_t base[256];           // large bucket: each digit's next place
    uint32_t wsum[kBW];
    uint32_t wmax[kBW];
    uint64_t red[4][kBW];
};

enum class Red { Min, Max, Or };

template <Red R>
__device__ __forceinline__ uint64_t red_op(uint64_t a, uint64_t b)
{
    if constexpr (R == Red::Min) return a < b ? a : b;
    if constexpr (R == Red::Max) return a > b ? a : b;
    return a | b;
}

// Block reductions of four 64-bit values, each with its own operation (every
// thread gets the results). Ends with a barrier.
template <Red R0, Red R1, Red R2, Red R3>
__device__ __forceinline__ void blk_reduce(BkLs &sh, uint64_t &v0, uint64_t &v1, uint64_t &v2, uint64_t &v3)
{
    const int w = (int)(threadIdx.x >> 6);
#pragma unroll
    for (int sft = 32; sft >= 1; sft >>= 1) {
        v0 = red_op<R0>(v0, shfl_xor_u64(v0, sft));
        v1 = red_op<R1>(v1, shfl_xor_u64(v1, sft));
        v2 = red_op<R2>(v2, shfl_xor_u64(v2, sft));
        v3 = red_op<R3>(v3, shfl_xor_u64(v3, sft));
    }
    if (lane_id() == 0) {
        sh.red[0][w] = v0;
        sh.red[1][w] = v1;
        sh.red[2][w] = v2;
        sh.red[3][w] = v3;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kBW; q++) {
        v0 = red_op<R0>(v0, sh.red[0][q]);
        v1 = red_op<R1>(v1, sh.red[1][q]);
        v2 = red_op<R2>(v2, sh.red[2][q]);
        v3 = red_op<R3>(v3, sh.red[3][q]);
    }
    __syncthreads();
}

// One stable pass of the block's pairs (wave-major: entry w * 64 reff + r * 64
// + lane, valid when below m) by the byte of `sel ? j : k` at bit `sh8`:
// pos[r] = the entry's place among the m in the pass order; sh.texcl: the
// digits' exclusive starts, sh.dtot: their counts. sh.wc must be zero on
// entry and is left zero. Ends with a barrier.
__device__ __forceinline__ void ls_byte_rank(BkLs &sh, const uint64_t *k, const uint32_t *j, bool sel,
                                             uint32_t sh8, uint32_t reff, uint32_t m, uint32_t *pos)
{
    const uint32_t t = threadIdx.x;
    const int w = (int)(t >> 6), lane = lane_id();
    const uint32_t wk = 64u * reff;
    uint32_t rk[kBR], dg[kBR];
#pragma unroll
    for (int r = 0; r < kBR; r++) {
        rk[r] = 0;
        dg[r] = 0;
        if ((uint32_t)r < reff) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            const bool ok = idx < m;
            dg[r] = (uint32_t)((sel ? (uint64_t)j[r] : k[r]) >> sh8) & 255u;
            const uint64_t peers = digit_peers(dg[r], ok);
            const uint32_t below = (uint32_t)__popcll(peers & lanemask_lt());
            const uint32_t old = ok ? sh.wc[w][dg[r]] : 0u;
            rk[r] = old + below;
            if (ok && below == 0) sh.wc[w][dg[r]] = old + (uint32_t)__popcll(peers);
            __builtin_amdgcn_wave_barrier();
        }
    }
    __syncthreads();
    // thread t < 256 = digit t: per-wave exclusive offsets and the total
    uint32_t tot = 0;
    if (t < 256) {
        uint32_t c[kBW];
#pragma unroll
        for (int q = 0; q < kBW; q++) c[q] = sh.wc[q][t];
#pragma unroll
        for (int q = 0; q < kBW; q++) {
            sh.wc[q][t] = tot;
            tot += c[q];
        }
    }
    const uint32_t ex = blk_excl_scan<kBT>(t < 256 ? tot : 0u, sh.wsum);
    if (t < 256) {
        sh.texcl[t] = ex;
        sh.dtot[t] = tot;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kBR; r++)
        if ((uint32_t)r < reff) pos[r] = sh.texcl[dg[r]] + sh.wc[w][dg[r]] + rk[r];
    __syncthreads();
    for (uint32_t i = t; i < kBW * 256u; i += kBT) (&sh.wc[0][0])[i] = 0;
    __syncthreads();
}

// A bucket of m > kLsCap pairs at [off, off + m): stable byte passes through
// global memory (the varying bytes of j, then those of the key), chunk by
// chunk of kLsCap pairs in order; then the values out.
__device__ void ls_big_bucket(const LsArgs &a, const LsRow &R, BkLs &sh, uint32_t off, uint32_t m)
{
    const uint32_t t = threadIdx.x;
    const int w = (int)(t >> 6), lane = lane_id();
    // the bits that vary (against the first pair)
    const uint64_t k0 = R.rk[0][off];
    const uint32_t j0 = R.rj[0][off];
    uint64_t kor = 0, jor = 0, z0 = 0, z1 = 0;
    for (uint32_t i = t; i < m; i += kBT) {
        kor |= R.rk[0][off + i] ^ k0;
        jor |= (uint64_t)(R.rj[0][off + i] ^ j0);
    }
    blk_reduce<Red::Or, Red::Or, Red::Or, Red::Or>(sh, kor, jor, z0, z1);
    for (uint32_t i = t; i < kBW * 256u; i += kBT) (&sh.wc[0][0])[i] = 0;
    uint32_t src = 0;
    for (uint32_t pass = 0; pass < 11; pass++) {
        const bool sel = pass < 3;   // three bytes of j (< 2^20), then eight of the key
        const uint32_t sh8 = 8u * (sel ? pass : pass - 3u);
        if ((((sel ? jor : kor) >> sh8) & 255u) == 0) continue;   // the same in every pair
        // digit counts over the bucket, then their exclusive starts
        if (t < 256) sh.base[t] = 0;
        __syncthreads();
        for (uint32_t i = t; i < m; i += kBT) {
            const uint64_t x = sel ? (uint64_t)R.rj[src][off + i] : R.rk[src][off + i];
            atomicAdd(&sh.base[(uint32_t)(x >> sh8) & 255u], 1u);
        }
        __syncthreads();
        {
            const uint32_t c = t < 256 ? sh.base[t] : 0u;
            const uint32_t ex = blk_excl_scan<kBT>(c, sh.wsum);
            if (t < 256) sh.base[t] = ex;
            __syncthreads();
        }
        // chunks in order: stable places inside the chunk, after the digit's
        // places taken by earlier chunks
        for (uint32_t c0 = 0; c0 < m; c0 += kLsCap) {
            const uint32_t cm = m - c0 < kLsCap ? m - c0 : kLsCap;
            const uint32_t reff = (cm + kBT - 1) / kBT, wk = 64u * reff;
            uint64_t k[kBR];
            uint32_t j[kBR], pos[kBR];
#pragma unroll
            for (int r = 0; r < kBR; r++) {
                const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
                const bool ok = (uint32_t)r < reff && idx < cm;
                k[r] = ok ? R.rk[src][off + c0 + idx] : 0ull;
                j[r] = ok ? R.rj[src][off + c0 + idx] : 0u;
            }
            ls_byte_rank(sh, k, j, sel, sh8, reff, cm, pos);
#pragma unroll
            for (int r = 0; r < kBR; r++) {
                const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
                if ((uint32_t)r < reff && idx < cm) {
                    const uint32_t d = (uint32_t)((sel ? (uint64_t)j[r] : k[r]) >> sh8) & 255u;
                    const uint32_t g = sh.base[d] + (pos[r] - sh.texcl[d]);
                    R.rk[src ^ 1u][off + g] = k[r];
                    R.rj[src ^ 1u][off + g] = j[r];
                }
            }
            __syncthreads();
            if (t < 256) sh.base[t] += sh.dtot[t];
            __syncthreads();
        }
        src ^= 1u;
    }
    for (uint32_t i = t; i < m; i += kBT)
        ls_emit(a, R, off + i, R.rk[src][off + i], ls_pay_gather(a, R, R.rj[src][off + i]));
}

__global__ __launch_bounds__(kBT) void k_ls_bucket(LsArgs a)
{
    __shared__ BkLs sh;
    const LsRow &R = a.r[blockIdx.y];
    const uint32_t t = threadIdx.x, bkt = blockIdx.x;
    if (bkt >= R.B) return;   // a row with fewer buckets than the grid is wide
    const int w = (int)(t >> 6), lane = lane_id();
    const uint32_t m = R.size[bkt], off = R.start[bkt];
    for (uint32_t i = t; i <= kBins; i += kBT) sh.bin[i] = 0;
    for (uint32_t i = t; i < kBW * 256u; i += kBT) (&sh.wc[0][0])[i] = 0;
    __syncthreads();
    if (m > kLsCap) {
        ls_big_bucket(a, R, sh, off, m);
        return;
    }
    const uint32_t reff = (m + kBT - 1) / kBT, wk = 64u * reff;
    uint64_t k[kBR];
    uint32_t j[kBR], rank[kBR];
    uint64_t kmn = ~0ull, kmx = 0, jmn = ~0ull, jmx = 0;
#pragma unroll
    for (int r = 0; r < kBR; r++) {
        const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
        const bool ok = (uint32_t)r < reff && idx < m;
        k[r] = ok ? R.rk[0][off + idx] : 0ull;
        j[r] = ok ? R.rj[0][off + idx] : 0u;
        rank[r] = 0;
        if (ok) {
            kmn = k[r] < kmn ? k[r] : kmn;
            kmx = k[r] > kmx ? k[r] : kmx;
            jmn = j[r] < jmn ? j[r] : jmn;
            jmx = j[r] > jmx ? j[r] : jmx;
        }
    }
    blk_reduce<Red::Min, Red::Max, Red::Min, Red::Max>(sh, kmn, kmx, jmn, jmx);
    // the primary key of the bins: the key, or j when every key is equal
    const bool byj = kmn == kmx;
    bool permuted = false;   // the byte passes moved the entries (their payloads are gathered)
    if (m <= 1) {
        // nothing to order
    } else {
        const uint64_t pmn = byj ? jmn : kmn, pmx = byj ? jmx : kmx;
        const uint64_t span = pmx - pmn;   // > 0: the pairs differ in p when m > 1
        const uint32_t bl = 64u - (uint32_t)__clzll((long long)span);
        const uint32_t shift = bl > kBinBits ? bl - kBinBits : 0u;
        uint32_t db[kBR];
#pragma unroll
        for (int r = 0; r < kBR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            db[r] = 0;
            if ((uint32_t)r < reff && idx < m) {
                const uint64_t p = byj ? (uint64_t)j[r] : k[r];
                const uint32_t q = (uint32_t)((p - pmn) >> shift);   // < kBins
                db[r] = q | (atomicAdd(&sh.bin[q], 1u) << kBinBits);
            }
        }
        __syncthreads();
        // bin starts: thread t owns bins 4t .. 4t + 3
        uint32_t maxbin;
        {
            uint32_t hv[4], sum = 0, mx = 0;
#pragma unroll
            for (int e = 0; e < 4; e++) {
                hv[e] = sh.bin[4 * t + e];
                sum += hv[e];
                mx = hv[e] > mx ? hv[e] : mx;
            }
#pragma unroll
            for (int sft = 32; sft >= 1; sft >>= 1) {
                const uint32_t o = (uint32_t)__shfl_xor((int)mx, sft, 64);
                mx = o > mx ? o : mx;
            }
            if (lane == 0) sh.wmax[w] = mx;
            uint32_t ex = blk_excl_scan<kBT>(sum, sh.wsum);
#pragma unroll
            for (int e = 0; e < 4; e++) {
                sh.bin[4 * t + e] = ex;
                ex += hv[e];
            }
            if (t == 0) sh.bin[kBins] = m;
            maxbin = 0;
#pragma unroll
            for (int q = 0; q < kBW; q++) maxbin = sh.wmax[q] > maxbin ? sh.wmax[q] : maxbin;
            __syncthreads();
        }
        if (maxbin <= kBinMax) {
            // each pair in its bin, then its rank = the bin's start + the
            // pairs of the bin below it
#pragma unroll
            for (int r = 0; r < kBR; r++) {
                const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
                if ((uint32_t)r < reff && idx < m) {
                    const uint32_t p = sh.bin[db[r] & (kBins - 1u)] + (db[r] >> kBinBits);
                    sh.lk[p] = k[r];
                    sh.lj[p] = j[r];
                }
            }
            __syncthreads();
#pragma unroll
            for (int r = 0; r < kBR; r++) {
                const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
                if ((uint32_t)r < reff && idx < m) {
                    const uint32_t q = db[r] & (kBins - 1u);
                    const uint32_t s0 = sh.bin[q], s1 = sh.bin[q + 1];
                    uint32_t rk = s0, u = s0;
                    for (; u + 4u <= s1; u += 4u) {
                        uint64_t xk[4];
                        uint32_t xj[4];
#pragma unroll
                        for (int q = 0; q < 4; q++) {
                            xk[q] = sh.lk[u + q];
                            xj[q] = sh.lj[u + q];
                        }
#pragma unroll
                        for (int q = 0; q < 4; q++) rk += pair_less(xk[q], xj[q], k[r], j[r]) ? 1u : 0u;
                    }
                    for (; u < s1; u++) rk += pair_less(sh.lk[u], sh.lj[u], k[r], j[r]) ? 1u : 0u;
                    rank[r] = rk;
                }
            }
        } else {
            // crowded bins (many equal or clustered keys): stable byte
            // passes over the bytes of j that vary in the bucket, then those
            // of the key; the pairs end in order, place = rank
            // the bits that vary: some pair differs there from the minimum
            uint64_t kor = 0, jor = 0, z0 = 0, z1 = 0;
#pragma unroll
            for (int r = 0; r < kBR; r++) {
                const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
                if ((uint32_t)r < reff && idx < m) {
                    kor |= k[r] ^ kmn;
                    jor |= (uint64_t)j[r] ^ jmn;
                }
            }
            blk_reduce<Red::Or, Red::Or, Red::Or, Red::Or>(sh, kor, jor, z0, z1);
            for (uint32_t pass = 0; pass < 11; pass++) {
                const bool sel = pass < 3;
                const uint32_t sh8 = 8u * (sel ? pass : pass - 3u);
                if ((((sel ? jor : kor) >> sh8) & 255u) == 0) continue;
                uint32_t pos[kBR];
                ls_byte_rank(sh, k, j, sel, sh8, reff, m, pos);
#pragma unroll
                for (int r = 0; r < kBR; r++) {
                    const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
                    if ((uint32_t)r < reff && idx < m) {
                        sh.lk[pos[r]] = k[r];
                        sh.lj[pos[r]] = j[r];
                    }
                }
                __syncthreads();
#pragma unroll
                for (int r = 0; r < kBR; r++) {
                    const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
                    if ((uint32_t)r < reff && idx < m) {
                        k[r] = sh.lk[idx];
                        j[r] = sh.lj[idx];
                    }
                }
                __syncthreads();
            }
#pragma unroll
            for (int r = 0; r < kBR; r++) rank[r] = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            permuted = true;
        }
    }
#pragma unroll
    for (int r = 0; r < kBR; r++) {
        const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
        if ((uint32_t)r < reff && idx < m)
            ls_emit(a, R, off + rank[r], k[r],
                    permuted ? ls_pay_gather(a, R, j[r]) : ls_pay_region(a, R, off + idx, j[r]));
    }
}

struct LsLayout {
    uint32_t B, S, hgt, tiles;
};

LsLayout ls_layout(uint64_t n)
{
    LsLayout l;
    l.B = (uint32_t)cdiv(n, kLsAvg);
    if (l.B < 2) l.B = 2;
    l.hgt = 0;
    while ((1u << l.hgt) < l.B) l.hgt++;
    const uint64_t s = align_up((uint64_t)kLsOver * l.B, 64);
    l.S = (uint32_t)(s < kLsMaxS ? s : kLsMaxS);
    l.tiles = (uint32_t)cdiv(n, kTile);
    return l;
}

}  // namespace

size_t lsort_sample_bytes(uint64_t n)
{
    if (n <= kSsMaxN || n > kLsMaxN) return 0;
    const LsLayout l = ls_layout(n);
    return 2 * align_up(l.S * 8, 256) + align_up(l.S * 4, 256) + align_up(kSmP * l.S * 4, 256);
}

LsSample lsort_sample_at(uint64_t n, void *p)
{
    const LsLayout l = ls_layout(n > kSsMaxN ? n : kSsMaxN + 1);
    uint8_t *q = static_cast<uint8_t *>(p);
    LsSample y;
    y.raw_k = reinterpret_cast<uint64_t *>(q);
    q += align_up(l.S * 8, 256);
    y.smp_k = reinterpret_cast<uint64_t *>(q);
    q += align_up(l.S * 8, 256);
    y.smp_j = reinterpret_cast<uint32_t *>(q);
    q += align_up(l.S * 4, 256);
    y.rpart = reinterpret_cast<uint32_t *>(q);
    y.draw = true;
    return y;
}

size_t lsort_ws_bytes(uint64_t n, uint32_t nsort, uint32_t npart)
{
    if (n <= kSsMaxN || n > kLsMaxN) return 0;
    const LsLayout l = ls_layout(n);
    const uint64_t sort = 2 * align_up(l.B * 4, 256) + align_up((uint64_t)l.tiles * l.B * 4, 256) +
                          2 * align_up(l.S * 8, 256) + align_up(l.S * 4, 256) + align_up(kSmP * l.S * 4, 256) +
                          align_up(n * 2, 256) +
                          2 * (align_up(n * 8, 256) + align_up(n * 4, 256)) +
                          align_up(n * 4, 256) + align_up(n, 256) + align_up(n * 8, 256);   // payloads
    const uint64_t part = 2 * align_up((kQ + 1) * 4, 256) + align_up((uint64_t)l.tiles * kQ * 4, 256);
    const uint64_t wrr = npart ? align_up(sizeof(WrrPlan), 256) + align_up(n * 4, 256) : 0;
    return (size_t)(nsort * sort + npart * part + wrr);
}

hipError_t lsort_launch(const SortInput &in, const SortJob *jobs, uint32_t njobs, void *ws, hipStream_t s,
                        const LsCopies *fifo_in_copies, const LsCopies *fifo_out_copies, const LsRuns *aging_runs,
                        const LsSample *sjf)
{
    const uint64_t n = in.n;
    if (n <= kSsMaxN || n > kLsMaxN || njobs == 0 || njobs > kLsMaxRows) return hipErrorInvalidValue;
    const LsLayout l = ls_layout(n);
    LsArgs a;
    memset(&a, 0, sizeof(a));
    a.in = in;
    if (fifo_in_copies) a.pf = *fifo_in_copies;
    if (fifo_out_copies) a.cp = *fifo_out_copies;
    if (aging_runs) a.runs = *aging_runs;
    a.n = (uint32_t)n;
    a.tiles = l.tiles;
    uint8_t *p = static_cast<uint8_t *>(ws);
    auto take = [&](uint64_t bytes) {
        uint8_t *q = p;
        p += align_up(bytes, 256);
        return q;
    };
    // the sorts first, then the partitions
    uint32_t npart = 0;
    for (int pass = 0; pass < 2; pass++)
        for (uint32_t i = 0; i < njobs; i++) {
            const SortKind k = jobs[i].kind;
            const bool part = k == SortKind::Class || k == SortKind::Tier;
            if (part != (pass == 1)) continue;
            if (!jobs[i].out && !(k == SortKind::Class && aging_runs)) return hipErrorInvalidValue;
            if (k != SortKind::Fifo && !in.fifo) return hipErrorInvalidValue;
            if (k != SortKind::Fifo && k != SortKind::Budget && k != SortKind::Aging && !part)
                return hipErrorInvalidValue;
            LsRow &R = a.r[a.nrows++];
            R.kind = k;
            R.key_out = jobs[i].key_out;
            R.out = jobs[i].out;
            if (part) {
                npart++;
                R.B = kQ;
                R.size = reinterpret_cast<uint32_t *>(take(kQ * 4));
                R.start = reinterpret_cast<uint32_t *>(take((kQ + 1) * 4));
                if (k == SortKind::Class && aging_runs) R.start = aging_runs->cstart;
                R.tcnt = reinterpret_cast<uint32_t *>(take((uint64_t)l.tiles * kQ * 4));
                continue;
            }
            a.nsort++;
            R.B = l.B;
            R.S = l.S;
            R.hgt = l.hgt;
            R.size = reinterpret_cast<uint32_t *>(take(l.B * 4));
            R.start = reinterpret_cast<uint32_t *>(take(l.B * 4));
            R.tcnt = reinterpret_cast<uint32_t *>(take((uint64_t)l.tiles * l.B * 4));
            R.raw_k = reinterpret_cast<uint64_t *>(take(l.S * 8));
            R.rpart = reinterpret_cast<uint32_t *>(take(kSmP * l.S * 4));
            R.smp_k = reinterpret_cast<uint64_t *>(take(l.S * 8));
            R.smp_j = reinterpret_cast<uint32_t *>(take(l.S * 4));
            if (k == SortKind::Budget && sjf && !sjf->draw) {
                // splitters drawn beside the FIFO sort
                R.smp_k = sjf->smp_k;
                R.smp_j = sjf->smp_j;
            } else {
                a.srow[a.nsamp++] = a.nrows - 1;
            }
            R.bid = reinterpret_cast<uint16_t *>(take(n * 2));
            for (int e = 0; e < 2; e++) {
                R.rk[e] = reinterpret_cast<uint64_t *>(take(n * 8));
                R.rj[e] = reinterpret_cast<uint32_t *>(take(n * 4));
            }
            if (k != SortKind::Fifo) R.rv = reinterpret_cast<uint32_t *>(take(n * 4));
            if (k == SortKind::Fifo && fifo_out_copies) {
                R.rt = reinterpret_cast<uint8_t *>(take(n));
                if (fifo_out_copies->bud) R.rb = reinterpret_cast<double *>(take(n * 8));
            }
        }
    if (npart) {
        a.plan = reinterpret_cast<WrrPlan *>(take(sizeof(WrrPlan)));
        a.tpos = reinterpret_cast<uint32_t *>(take(n * 4));
    }
    if (sjf && sjf->draw) {
        // a row after the others, sampled only: SJF's splitters by request
        // index, so that the batch over the FIFO sequence skips its sampling
        if (a.nrows >= kLsMaxRows) return hipErrorInvalidValue;
        LsRow &R = a.r[a.nrows];
        R.kind = SortKind::Budget;
        R.by_req = 1;
        R.B = l.B;
        R.S = l.S;
        R.hgt = l.hgt;
        R.raw_k = sjf->raw_k;
        R.rpart = sjf->rpart;
        R.smp_k = sjf->smp_k;
        R.smp_j = sjf->smp_j;
        a.srow[a.nsamp++] = a.nrows;
    }
    const uint32_t maxb = a.nsort ? l.B : kQ;
    if (a.nsamp) {
        hipLaunchKernelGGL(k_ls_gather, dim3(cdiv(l.S, 256), a.nsamp), dim3(256), 0, s, a);
        hipLaunchKernelGGL(k_ls_sample, dim3(l.S / 64 * kSmP, a.nsamp), dim3(kSmT), 0, s, a);
        hipLaunchKernelGGL(k_ls_place, dim3(cdiv(l.S, 256), a.nsamp), dim3(256), 0, s, a);
    }
    hipLaunchKernelGGL(k_ls_count, dim3(l.tiles, a.nrows), dim3(kTT), 0, s, a);
    hipLaunchKernelGGL(k_ls_scan, dim3(cdiv(maxb, 64), a.nrows), dim3(kScT), 0, s, a);
    hipLaunchKernelGGL(k_ls_scatter, dim3(l.tiles, a.nrows), dim3(kTT), 0, s, a);
    if (a.nsort) hipLaunchKernelGGL(k_ls_bucket, dim3(l.B, a.nsort), dim3(kBT), 0, s, a);
    return hipGetLastError();
}

}  // namespace ds
