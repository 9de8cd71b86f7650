// Dispatch orders of up to 2^18 requests as one batch of sample sorts
// (Sec. "Scheduling Engine"): three launches for any set of policies.
//
// Every policy ends ties in FIFO order, and FIFO order is the order of
// (arrival, index). So SJF and Aging order the requests by a composite key
// (k1, k2, i): k1 the policy's own key, k2 the arrival, i the request index,
// compared in that order; neither needs the FIFO permutation as an input,
// and they sort side by side with the FIFO sort:
//   Fifo    k1 = arrival (no k2)
//   Budget  k1 = budget                                     (SJF)
//   Aging   k1 = aged score max(floor, p - rate * max(0, t_now - arrival))
// Keys are doubles compared through ordered_bits (so -0.0 ties with +0.0).
// Priority and Weighted are stable partitions of the FIFO sequence by a
// digit of at most 4 bits (the priority class of the tier, or the tier).
// The FIFO row's bucket blocks place them: a bucket holds a contiguous run
// of the FIFO sequence, so a request's rank among its digit's requests is
// the count over earlier buckets (decoupled look-back over the buckets'
// digit counts) plus its rank in the bucket. Priority puts it at its class's
// first position plus that rank; Weighted at the round-robin position of
// the k-th request of tier t, blocked:
//   sum_t' min(n_t', r w_t') + sum_{t' < t} min(w_t', max(0, n_t' - r w_t'))
//   + (k - r w_t),  r = floor(k / w_t);
// smooth: from the period table of the smooth interleaving (wrrplan.h),
// built by the FIFO row's last scatter tile; stride: from the closed form
// of the passes (k + 1) / w_t.
//
//   k_ss_sample   S triples (1024 up to 2^17 requests, else 2048) at
//                 stratified random positions; each of S/8 blocks stages all
//                 of them in LDS, finds the rank of 8 of them by counting the
//                 smaller ones and stores each at its rank: the sorted
//                 sample, of which every (S/B)-th triple is one of B - 1
//                 splitters. Also clears the look-back words, the overflow
//                 flag and the tier totals.
//   k_ss_scatter  per tile of 2048 requests: makes the keys (and the
//                 per-request key output; the FIFO row adds its tier counts
//                 to the totals), finds each request's bucket by
//                 descending a search tree of the splitters, ranks the tile
//                 by bucket (wave ballots), takes the bucket's count over
//                 earlier tiles by decoupled look-back and writes the keys
//                 and index into the bucket's fixed-capacity region, so that
//                 a bucket holds its requests in index order.
//   k_ss_bucket   one block per bucket (its offset: the sizes of the buckets
//                 before it). A rank pass orders the bucket by one 64-bit key,
//                 stably in the current order: by bins over the key range and
//                 counting inside a bin, or stable LSD passes when a bin is
//                 crowded. Two-key sorts take a pass by k2, then one by k1
//                 (skipped when k1 is the same for the whole bucket), which
//                 together order by (k1, k2, index).
// A bucket that outgrows its region (only for inputs arranged against the
// sampling) sets the overflow flag; k_ss_bucket then sorts the whole batch
// in one workgroup with LSD passes over global memory.
#include <string.h>

#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "lookback.h"
#include "wrrplan.h"

namespace ds {
namespace {

constexpr uint32_t kSamples = 2048;      // triples sampled per sort (at most)
constexpr uint32_t kCap = 4096;          // requests per bucket region
constexpr uint32_t kMaxBuckets = 256;
constexpr uint32_t kBucketAvg = 1024;    // target requests per bucket
constexpr uint32_t kBucketAvgFifo = 512; // the same for the FIFO row, which does the most per bucket
constexpr int kScTPB = 512, kScR = 4;    // scatter tile: 2048 requests
constexpr uint32_t kScTile = kScTPB * kScR;
constexpr int kBkTPB = 512, kBkR = kCap / kBkTPB;
constexpr uint32_t kBinBits = 11, kBins = 1u << kBinBits;   // in-bucket bins
constexpr uint32_t kBinMax = 128;        // larger bins: LSD passes instead
constexpr uint32_t kBinMax2 = 32;        // the same for a pass by two keys
constexpr int kSmpTPB = 256;             // k_ss_sample: threads per block,
constexpr uint32_t kSmpThr = 32;         // threads per sample ranked,
constexpr uint32_t kSmpPerBlock = kSmpTPB / kSmpThr;   // samples ranked per block
constexpr uint32_t kQ = 16;              // tiers (a larger tier value counts as the last)
// FIFO row with the partitions: a bucket entry's index carries its request's
// tier in the top byte (written by the scatter, which loads the tiers
// anyway), so that the bucket blocks need not gather them
constexpr uint32_t kIdxBits = 24, kIdxMask = (1u << kIdxBits) - 1u;
static_assert(kSsMaxN <= (1u << kIdxBits), "request index and tier share a word");

struct SsCtl {
    uint32_t overflow;
    uint32_t lb_err;       // a bounded look-back wait over the buckets ran out
    uint32_t tiles_done;   // FIFO row, smooth round robin: scatter tiles whose tier counts are in
    uint32_t pad[61];
};

struct SsDesc {
    SortKind kind;
    uint32_t nb;           // buckets of this row, 1..kMaxBuckets
    uint32_t two;          // k2 (the arrival) is part of the key
    double *key_out;
    uint32_t *out;
    SsCtl *ctl;
    uint64_t *smp_k1;      // [kSamples] the sample in sorted order
    uint64_t *smp_k2;
    uint32_t *smp_j;
    uint32_t *status;      // [tiles][256] look-back words
    uint64_t *bk1;         // [buckets][kCap] bucket regions
    uint64_t *bk2;
    uint32_t *bj;
    uint32_t *tot;         // [kQ] requests per tier (FIFO row with partitions; added up by the scatter tiles)
    uint32_t *bstat;       // [buckets][2 kQ] look-back words of the digit counts
    uint32_t *pw_out[2];   // FIFO row: Priority and Weighted orders (or NULL)
    double *pw_key[2];
    uint64_t *fk1[2];      // [n] x 2: single-workgroup sort
    uint64_t *fk2[2];
    uint32_t *fj[2];
};

struct SsBatch {
    SortInput in;
    uint32_t n;
    uint32_t tiles;        // scatter tiles
    uint32_t nb;           // the most buckets of a row (grid width of the bucket launch)
    uint32_t ns;           // samples, 1..kSamples
    uint32_t serial;       // sort in one workgroup regardless of the buckets
    uint32_t nsorts;       // sorts of the batch (grid rows)
    uint32_t nsb;          // blocks of k_ss_sample per sort
    WrrPlan *plan;         // smooth round robin: the period table (built by the scatter)
    uint32_t *tpos;        // [n] its start-up positions
    SsDesc s[kSsMaxSorts];
};

// Position of sample s: uniform in the s-th of S equal strata of [0, n)
// (a fixed integer hash picks the offset), so that sampling does not lock
// onto periodic arrangements of the input.
// (32-bit arithmetic: s n < 2^29 for n <= 2^18 and s < 2048.)
__device__ __forceinline__ uint32_t sample_pos(uint32_t s, uint32_t n, uint32_t S)
{
    const uint32_t lo = s * n / S, hi = (s + 1) * n / S;
    uint32_t h = s * 0x9E3779B1u + 0x7F4A7C15u;
    h ^= h >> 15;
    h *= 0x85EBCA77u;
    h ^= h >> 13;
    return lo + h % (hi - lo);   // hi > lo since S <= n
}

// The double whose ordered_bits is k (+0.0 for the key of both zeros).
__device__ __forceinline__ double from_ordered(uint64_t k)
{
    const uint64_t u = (k >> 63) ? (k & 0x7FFFFFFFFFFFFFFFull) : ~k;
    return __longlong_as_double((long long)u);
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t x, int m)
{
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)x, m, 64);
    const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(x >> 32), m, 64);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ bool key_less(uint64_t a1, uint64_t a2, uint32_t ja, uint64_t b1, uint64_t b2,
                                         uint32_t jb)
{
    return a1 < b1 || (a1 == b1 && (a2 < b2 || (a2 == b2 && ja < jb)));
}

// The sort key (k1, k2) of request i, and the per-request key output (the
// policy's primary key). The
// aged score rounds each operation separately (no fused multiply-add). Only
// loads and arithmetic: a caller that unrolls several requests gets all
// their loads in flight before the first use.
template <SortKind K>
__device__ __forceinline__ void ss_key(const SortInput &in, uint32_t i, uint64_t &k1, uint64_t &k2, double &kv)
{
    const double a = in.arrival[i];
    if constexpr (K == SortKind::Fifo) {
        kv = a;
        k1 = ordered_bits(a);
        k2 = 0;
    } else if constexpr (K == SortKind::Budget) {
        kv = in.budget[i];
        k1 = ordered_bits(kv);
        k2 = ordered_bits(a);
    } else {   // Aging
        uint32_t q = in.tier[i];
        q = q < kQ ? q : kQ - 1u;
        k2 = ordered_bits(a);
        double w = in.t_now - a;
        if (w < 0.0) w = 0.0;
        const double d = in.aging_rate * w;
        double e = in.prio[q] - d;
        if (e < in.aging_floor) e = in.aging_floor;
        kv = e;
        k1 = ordered_bits(e);
    }
}

// Run `body` with the sort kind as a compile-time constant.
template <typename F>
__device__ __forceinline__ void with_kind(SortKind kind, F &&body)
{
    switch (kind) {
    case SortKind::Fifo: body(std::integral_constant<SortKind, SortKind::Fifo>()); break;
    case SortKind::Budget: body(std::integral_constant<SortKind, SortKind::Budget>()); break;
    default: body(std::integral_constant<SortKind, SortKind::Aging>()); break;
    }
}

struct SmpShared {
    uint64_t k1[kSamples];
    uint64_t k2[kSamples];
    uint32_t j[kSamples];
};

template <SortKind K>
__device__ __forceinline__ void sample_body(const SsBatch &b, const SsDesc &d, SmpShared &sh)
{
    const uint32_t t = threadIdx.x, n = b.n, S = b.ns;
    const uint32_t stride = b.nsb * kSmpTPB;
    for (uint32_t i = blockIdx.x * kSmpTPB + t; i < b.tiles * 256u; i += stride) d.status[i] = 0;
    if (d.pw_out[0] || d.pw_out[1])
        for (uint32_t i = blockIdx.x * kSmpTPB + t; i < d.nb * 2u * kQ; i += stride) d.bstat[i] = 0;
    if (blockIdx.x == 0 && t == 0) {
        d.ctl->overflow = b.serial;
        d.ctl->lb_err = 0;
        if (blockIdx.y == 0 && b.in.wait.clear && b.in.wait.status) *b.in.wait.status = 0;
        d.ctl->tiles_done = 0;
    }
    if (blockIdx.x == 0 && t < kQ && (d.pw_out[0] || d.pw_out[1])) d.tot[t] = 0;
    {
        // all loads in flight before the first LDS store
        constexpr int kPer = kSamples / kSmpTPB;
        uint64_t k1[kPer], k2[kPer];
        uint32_t j[kPer];
#pragma unroll
        for (int r = 0; r < kPer; r++) {
            const uint32_t s = (uint32_t)r * kSmpTPB + t;
            j[r] = s < S ? sample_pos(s, n, S) : 0u;
            double kv;
            ss_key<K>(b.in, j[r], k1[r], k2[r], kv);
        }
#pragma unroll
        for (int r = 0; r < kPer; r++) {
            // unused slots hold the largest triple, below no sample
            const uint32_t s = (uint32_t)r * kSmpTPB + t;
            sh.k1[s] = s < S ? k1[r] : ~0ull;
            sh.k2[s] = s < S ? k2[r] : ~0ull;
            sh.j[s] = s < S ? j[r] : ~0u;
        }
    }
    __syncthreads();
    // kSmpThr threads per sample: thread q of sample s counts the samples
    // u = q, q + kSmpThr, ... below s (neighbouring lanes read neighbouring
    // words); the partial counts are added by shuffles
    const uint32_t s = blockIdx.x * kSmpPerBlock + t / kSmpThr, q = t % kSmpThr;
    uint32_t below = 0;
    {
        const uint32_t sc = s < S ? s : 0u;
        const uint64_t a1 = sh.k1[sc], a2 = sh.k2[sc];
        const uint32_t ja = sh.j[sc];
        uint32_t part[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        const uint32_t Sp = (S + 8 * kSmpThr - 1) / (8 * kSmpThr) * (8 * kSmpThr);   // <= kSamples
        for (uint32_t u0 = 0; u0 < Sp; u0 += 8 * kSmpThr) {
            uint64_t u1[8], u2[8];
            uint32_t ju[8];
#pragma unroll
            for (uint32_t e = 0; e < 8; e++) {
                u1[e] = sh.k1[u0 + e * kSmpThr + q];
                u2[e] = sh.k2[u0 + e * kSmpThr + q];
                ju[e] = sh.j[u0 + e * kSmpThr + q];
            }
#pragma unroll
            for (uint32_t e = 0; e < 8; e++) part[e] += key_less(u1[e], u2[e], ju[e], a1, a2, ja) ? 1u : 0u;
        }
#pragma unroll
        for (uint32_t e = 0; e < 8; e++) below += part[e];
    }
#pragma unroll
    for (int m = kSmpThr / 2; m >= 1; m >>= 1) below += (uint32_t)__shfl_xor((int)below, m, 64);
    if (s < S && q == 0) {
        d.smp_k1[below] = sh.k1[s];
        d.smp_k2[below] = sh.k2[s];
        d.smp_j[below] = sh.j[s];
    }
}

__global__ __launch_bounds__(kSmpTPB) void k_ss_sample(SsBatch b)
{
    __shared__ SmpShared sh;
    const SsDesc &d = b.s[blockIdx.y];
    with_kind(d.kind, [&](auto K) { sample_body<decltype(K)::value>(b, d, sh); });
}

// The keys of this thread's kScR requests of the tile (loads first, then the
// per-request key output).
template <SortKind K>
__device__ __forceinline__ void scatter_keys(const SsBatch &b, const SsDesc &d, uint32_t base, uint32_t cnt,
                                             uint64_t *k1, uint64_t *k2, uint32_t *jj)
{
    const int w = (int)(threadIdx.x >> 6), lane = lane_id();
    double kv[kScR];
#pragma unroll
    for (int r = 0; r < kScR; r++) {
        const uint32_t idx = (uint32_t)w * (64u * kScR) + (uint32_t)r * 64u + (uint32_t)lane;
        jj[r] = base + (idx < cnt ? idx : 0u);
        ss_key<K>(b.in, jj[r], k1[r], k2[r], kv[r]);
    }
    if (d.key_out) {
#pragma unroll
        for (int r = 0; r < kScR; r++) {
            const uint32_t idx = (uint32_t)w * (64u * kScR) + (uint32_t)r * 64u + (uint32_t)lane;
            if (idx < cnt) d.key_out[base + idx] = kv[r];
        }
    }
}

__global__ __launch_bounds__(kScTPB) void k_ss_scatter(SsBatch b)
{
    constexpr int kWaves = kScTPB / 64;
    constexpr uint32_t kWaveKeys = 64u * kScR;
    __shared__ uint64_t s_k1[kMaxBuckets];   // [1, 2^hgt): the search tree
    __shared__ uint64_t s_k2[kMaxBuckets];
    __shared__ uint32_t s_j[kMaxBuckets];
    __shared__ uint32_t wcnt[kWaves][256];
    __shared__ uint32_t texcl[256];
    __shared__ uint32_t gbase[256];
    __shared__ uint32_t tmp4[4];
    __shared__ uint64_t lk1[kScTile];
    __shared__ uint64_t lk2[kScTile];
    __shared__ uint32_t lj[kScTile];
    __shared__ uint8_t lb[kScTile];
    __shared__ uint32_t s_tq[kQ];
    __shared__ uint32_t s_last;

    const SsDesc &d = b.s[blockIdx.y];
    const uint32_t t = threadIdx.x, n = b.n, nsp = d.nb - 1;
    const int w = (int)(t >> 6), lane = lane_id();
    const uint32_t tile = blockIdx.x, base = tile * kScTile;
    const uint32_t cnt = n - base < kScTile ? n - base : kScTile;
    const bool digit_thread = t < 256;
    const bool pw = d.pw_out[0] || d.pw_out[1];   // FIFO row with the partitions: count the tiers

    uint64_t k1[kScR], k2[kScR];
    uint32_t jj[kScR], bk[kScR], rk[kScR], tq[kScR];
    with_kind(d.kind, [&](auto K) { scatter_keys<decltype(K)::value>(b, d, base, cnt, k1, k2, jj); });
    if (pw) {
#pragma unroll
        for (int r = 0; r < kScR; r++) {
            const uint32_t idx = (uint32_t)w * kWaveKeys + (uint32_t)r * 64u + (uint32_t)lane;
            tq[r] = idx < cnt ? b.in.tier[base + idx] : kQ;   // kQ: no request
        }
        if (t < kQ) s_tq[t] = 0;
    }
    // splitters in breadth-first (Eytzinger) order of a complete search tree
    // of height hgt: node e (1-based) holds the splitter of in-order index
    // (2 p + 1) 2^(hgt - d - 1) - 1 (d = depth of e, p = e - 2^d); splitter i
    // is the sample of rank floor((i + 1) S / B), and in-order indices from
    // B - 1 on are padded with the largest triple. The first levels of every
    // search then read the same few LDS words in all lanes.
    uint32_t hgt = 0;
    while ((1u << hgt) < d.nb) hgt++;
    for (uint32_t e = t + 1; e < (1u << hgt); e += kScTPB) {
        const uint32_t dpt = 31u - (uint32_t)__clz((int)e), pp = e - (1u << dpt);
        const uint32_t i = (2u * pp + 1u) * (1u << (hgt - dpt - 1u)) - 1u;
        uint64_t a1 = ~0ull, a2 = ~0ull;
        uint32_t jv = ~0u;
        if (i < nsp) {
            const uint32_t r = (i + 1) * b.ns / d.nb;   // < ns; (i + 1) ns < 2^19
            a1 = d.smp_k1[r];
            a2 = d.smp_k2[r];
            jv = d.smp_j[r];
        }
        s_k1[e] = a1;
        s_k2[e] = a2;
        s_j[e] = jv;
    }
    for (uint32_t i = t; i < kWaves * 256u; i += kScTPB) (&wcnt[0][0])[i] = 0;
    __syncthreads();   // splitters and counters ready
    if (pw) {
#pragma unroll
        for (int r = 0; r < kScR; r++)
            if (tq[r] != kQ) atomicAdd(&s_tq[tq[r] < kQ ? tq[r] : kQ - 1u], 1u);
    }
    // bucket = number of splitters <= (k1, k2, i): hgt steps down the tree
    // (the rounds advance together, so that their LDS reads overlap)
    uint32_t node[kScR];
#pragma unroll
    for (int r = 0; r < kScR; r++) node[r] = 1;
    for (uint32_t lvl = 0; lvl < hgt; lvl++) {
        uint64_t a1[kScR], a2[kScR];
        uint32_t aj[kScR];
#pragma unroll
        for (int r = 0; r < kScR; r++) {
            a1[r] = s_k1[node[r]];
            a2[r] = s_k2[node[r]];
            aj[r] = s_j[node[r]];
        }
#pragma unroll
        for (int r = 0; r < kScR; r++)
            node[r] = 2u * node[r] + (key_less(k1[r], k2[r], jj[r], a1[r], a2[r], aj[r]) ? 0u : 1u);
    }
#pragma unroll
    for (int r = 0; r < kScR; r++) bk[r] = node[r] - (1u << hgt);
    // stable rank within the wave by bucket, round by round
#pragma unroll
    for (int r = 0; r < kScR; r++) {
        const uint32_t idx = (uint32_t)w * kWaveKeys + (uint32_t)r * 64u + (uint32_t)lane;
        const bool ok = idx < cnt;
        const uint32_t dg = bk[r];
        const uint64_t peers = digit_peers(dg, ok);
        const uint32_t below = (uint32_t)__popcll(peers & lanemask_lt());
        const uint32_t old = ok ? wcnt[w][dg] : 0u;
        rk[r] = old + below;
        if (ok && below == 0) wcnt[w][dg] = old + (uint32_t)__popcll(peers);
        __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();
    uint32_t tc = 0;
    if (digit_thread) {
        uint32_t c[kWaves];
#pragma unroll
        for (int q = 0; q < kWaves; q++) c[q] = wcnt[q][t];
#pragma unroll
        for (int q = 0; q < kWaves; q++) {
            wcnt[q][t] = tc;
            tc += c[q];
        }
    }
    // the tile's requests per tier join the row's totals (read by the bucket launch)
    if (pw && t < kQ && s_tq[t]) atomicAdd(&d.tot[t], s_tq[t]);
    uint32_t *st = d.status;
    if (digit_thread) st_relaxed(&st[(uint64_t)tile * 256u + t], (tile == 0 ? kPre : kAgg) | tc);
    const uint32_t tex = block_excl_scan_digits<kScTPB>(tc, tmp4);
    if (digit_thread) {
        texcl[t] = tex;
        uint32_t prefix = 0;
        if (tile > 0) {
            // a wait that runs out sends the sort to the single-workgroup path
            prefix = look_back(st, tile, t, &d.ctl->overflow, b.in.wait.no_wait ? 0u : kSpinLimit);
            st_relaxed(&st[(uint64_t)tile * 256u + t], kPre | (prefix + tc));
        }
        gbase[t] = prefix;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kScR; r++) {
        const uint32_t idx = (uint32_t)w * kWaveKeys + (uint32_t)r * 64u + (uint32_t)lane;
        if (idx < cnt) {
            const uint32_t dg = bk[r];
            const uint32_t lp = texcl[dg] + wcnt[w][dg] + rk[r];
            lk1[lp] = k1[r];
            lk2[lp] = k2[r];
            lj[lp] = pw ? jj[r] | (tq[r] << kIdxBits) : jj[r];   // tq[r] < 256 here
            lb[lp] = (uint8_t)dg;
        }
    }
    __syncthreads();
    bool over = false;
    for (uint32_t s = t; s < cnt; s += kScTPB) {
        const uint32_t dg = lb[s];
        const uint32_t g = gbase[dg] + s - texcl[dg];
        if (g < kCap) {
            const uint64_t o = (uint64_t)dg * kCap + g;
            d.bk1[o] = lk1[s];
            if (d.two) d.bk2[o] = lk2[s];
            d.bj[o] = lj[s];
        } else {
            over = true;
        }
    }
    if (over) atomicOr(&d.ctl->overflow, 1u);
    if (pw && d.pw_out[1] && b.in.wrr_mode == kWrrSmooth) {
        // the smooth interleaving's period table needs every tile's tier
        // counts: the last tile to be done builds it, with one wave (its
        // keys are out, so lj serves as scratch)
        if (t < kQ) __threadfence();   // this tile's counts are in before its ticket
        __syncthreads();
        if (t == 0) s_last = atomicAdd(&d.ctl->tiles_done, 1u) == b.tiles - 1u ? 1u : 0u;
        __syncthreads();
        if (s_last && w == 0) {
            __threadfence();
            const uint32_t nq = b.in.n_tiers < kQ ? b.in.n_tiers : kQ;
            const bool tl = (uint32_t)lane < nq;
            wrr_plan_build(tl ? ld_relaxed(&d.tot[lane]) : 0u, tl ? b.in.weight[lane] : 0u,
                           reinterpret_cast<uint16_t *>(lj), b.plan, b.tpos);
        }
    }
}

// Priority and Weighted: requests per tier, each class's first position,
// and the digit counts (classes 0..15, then tiers 16..31).
struct PwTable {
    double prio[kQ];                 // per tier: priority, class, weight (copies of
    uint32_t cls[kQ];                // the launch parameters, indexed per lane)
    uint32_t weight[kQ];
    uint32_t tot[kQ];
    uint32_t cstart[kQ];
    uint32_t cnt[2 * kQ];            // this bucket's (or chunk's) digit counts
    uint32_t pre[2 * kQ];            // the digits' counts before it
    uint32_t wd[kBkTPB / 64][2 * kQ];   // per-wave digit counters
    WrrPlanHead wh;                  // smooth round robin: the phases of the period table
};

// The round-robin position of the k-th request (in FIFO order) of tier q,
// and its round.
__device__ __forceinline__ uint64_t weighted_pos(const PwTable &pt, uint32_t n_tiers, uint32_t q, uint32_t k,
                                                 uint32_t &rnd)
{
    const uint32_t wq = pt.weight[q] ? pt.weight[q] : 1u;
    rnd = k / wq;
    uint64_t p = k - rnd * wq;
    for (uint32_t u = 0; u < n_tiers; u++) {
        const uint64_t nt = pt.tot[u], wt = pt.weight[u], full = (uint64_t)rnd * wt;
        p += nt < full ? nt : full;
        if (u < q) {
            const uint64_t left = nt > full ? nt - full : 0u;
            p += left < wt ? left : wt;
        }
    }
    return p;
}

// Requests at FIFO positions in a run: their Priority and Weighted places.
// qd: tier (clamped), j: request, rc/rt: rank among the run's requests of
// the same class/tier before it, pre: counts of the digits before the run.
__device__ __forceinline__ void pw_place(const SsBatch &b, const SsDesc &d, const PwTable &pt, uint32_t q,
                                         uint32_t j, uint32_t kc, uint32_t kt)
{
    if (d.pw_out[0]) {
        const uint32_t c = pt.cls[q];
        const uint64_t pos = (uint64_t)pt.cstart[c] + kc;
        if (pos < b.n) d.pw_out[0][pos] = j;   // always, for tiers < n_tiers
        if (d.pw_key[0]) d.pw_key[0][j] = pt.prio[q];
    }
    if (d.pw_out[1]) {
        uint32_t rnd;
        const uint32_t nq = b.in.n_tiers < kQ ? b.in.n_tiers : kQ;
        uint64_t pos;
        if (b.in.wrr_mode == kWrrSmooth) {
            pos = wrr_smooth_pos(pt.wh, b.plan, b.tpos, pt.weight[q], q, kt, rnd);
        } else if (b.in.wrr_mode == kWrrStride) {
            rnd = kt / (pt.weight[q] ? pt.weight[q] : 1u);
            pos = wrr_stride_pos(q, kt, pt.weight, nq, [&](uint32_t u) { return pt.tot[u]; });
        } else {
            pos = weighted_pos(pt, nq, q, kt, rnd);
        }
        if (pos < b.n) d.pw_out[1][pos] = j;
        if (d.pw_key[1]) d.pw_key[1][j] = (double)rnd;
    }
}

// LDS scratch of the bucket sort (also used by the single-workgroup sort).
// The bin histogram and the LSD digit counters are never live together and
// share their words, so that two blocks fit a CU.
struct BkShared {
    union {
        uint32_t bin[kBins + 1];              // bin histogram, then bin starts
        uint32_t wcnt[2][kBkTPB / 64][256];   // per-wave digit counters, two passes' worth
    };
    uint32_t texcl[256];
    uint32_t dcnt[256];
    uint32_t offs[256];
    uint32_t tmp4[4];
    uint32_t redu[kBkTPB / 64];
    uint32_t wsum[kBkTPB / 64];
    uint32_t wmax[kBkTPB / 64];
    uint64_t kmin[kBkTPB / 64], kmax[kBkTPB / 64], kmin2[kBkTPB / 64];
    uint64_t kmin1[kBkTPB / 64], kmax1[kBkTPB / 64];
    PwTable pt;
    uint64_t lkey[kCap];
    uint64_t lkey2[kCap];
    uint32_t lj[kCap + 1];
    uint16_t lslot[kCap];
    uint8_t lq[kCap];
};

// One stable LSD pass on byte p of the keys of m entries held R_eff per
// thread (wave-major positions w * 64 R_eff + r * 64 + lane): returns each
// entry's place in the pass order through pos, leaves the digits' exclusive
// starts in sh.texcl and, for thread t < 256, digit t's count in tc. Counters
// buffer `cur` must be zero on entry; buffer cur ^ 1 is cleared for the next
// pass. Ends with a barrier; the caller's reads of pos-ordered data need
// another.
__device__ __forceinline__ void lds_rank(BkShared &sh, uint32_t cur, const uint64_t *k, uint32_t reff,
                                         uint32_t m, uint32_t p, uint32_t *pos, uint32_t &tc)
{
    constexpr int kWaves = kBkTPB / 64;
    const uint32_t t = threadIdx.x;
    const int w = (int)(t >> 6), lane = lane_id();
    const uint32_t wk = 64u * reff;
    uint32_t (*wc)[256] = sh.wcnt[cur];
    uint32_t rk[kBkR];
#pragma unroll
    for (int r = 0; r < kBkR; r++) {
        rk[r] = 0;
        if ((uint32_t)r < reff) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            const bool ok = idx < m;
            const uint32_t dg = (uint32_t)(k[r] >> (8 * p)) & 255u;
            const uint64_t peers = digit_peers(dg, ok);
            const uint32_t below = (uint32_t)__popcll(peers & lanemask_lt());
            const uint32_t old = ok ? wc[w][dg] : 0u;
            rk[r] = old + below;
            if (ok && below == 0) wc[w][dg] = old + (uint32_t)__popcll(peers);
            __builtin_amdgcn_wave_barrier();
        }
    }
    for (uint32_t i = t; i < kWaves * 256u; i += kBkTPB) (&sh.wcnt[cur ^ 1u][0][0])[i] = 0;
    __syncthreads();
    // wave 0: digits 4 l .. 4 l + 3 per lane l: per-wave exclusive offsets,
    // digit totals and their exclusive scan
    if (w == 0) {
        uint32_t c[4][kWaves], tot[4];
#pragma unroll
        for (int e = 0; e < 4; e++)
#pragma unroll
            for (int q = 0; q < kWaves; q++) c[e][q] = wc[q][4u * (uint32_t)lane + (uint32_t)e];
#pragma unroll
        for (int e = 0; e < 4; e++) {
            const uint32_t dgt = 4u * (uint32_t)lane + (uint32_t)e;
            uint32_t acc = 0;
#pragma unroll
            for (int q = 0; q < kWaves; q++) {
                wc[q][dgt] = acc;
                acc += c[e][q];
            }
            tot[e] = acc;
        }
        const uint32_t sum = tot[0] + tot[1] + tot[2] + tot[3];
        uint32_t ex = wave_incl_scan_dpp(sum) - sum;
#pragma unroll
        for (int e = 0; e < 4; e++) {
            const uint32_t dgt = 4u * (uint32_t)lane + (uint32_t)e;
            sh.texcl[dgt] = ex;
            sh.dcnt[dgt] = tot[e];
            ex += tot[e];
        }
    }
    __syncthreads();
    tc = t < 256 ? sh.dcnt[t] : 0u;
#pragma unroll
    for (int r = 0; r < kBkR; r++) {
        if ((uint32_t)r < reff) {
            const uint32_t dg = (uint32_t)(k[r] >> (8 * p)) & 255u;
            pos[r] = sh.texcl[dg] + wc[w][dg] + rk[r];
        }
    }
}

// Key ranges of the m entries of a bucket: of k, and of k2 when given
// (every thread gets them). Ends with a barrier.
__device__ __forceinline__ void block_range(BkShared &sh, const uint64_t *k, const uint64_t *k2, uint32_t reff,
                                            uint32_t m, uint64_t &kmn, uint64_t &kmx, uint64_t &kmn2,
                                            uint64_t &kmx2)
{
    constexpr int kWaves = kBkTPB / 64;
    const int w = (int)(threadIdx.x >> 6), lane = lane_id();
    const uint32_t wk = 64u * reff;
    kmn = ~0ull;
    kmx = 0;
    kmn2 = ~0ull;
    kmx2 = 0;
#pragma unroll
    for (int r = 0; r < kBkR; r++) {
        const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
        if ((uint32_t)r < reff && idx < m) {
            kmn = k[r] < kmn ? k[r] : kmn;
            kmx = k[r] > kmx ? k[r] : kmx;
            if (k2) {
                kmn2 = k2[r] < kmn2 ? k2[r] : kmn2;
                kmx2 = k2[r] > kmx2 ? k2[r] : kmx2;
            }
        }
    }
#pragma unroll
    for (int sft = 32; sft >= 1; sft >>= 1) {
        uint64_t a = shfl_xor_u64(kmn, sft), c2 = shfl_xor_u64(kmx, sft);
        kmn = a < kmn ? a : kmn;
        kmx = c2 > kmx ? c2 : kmx;
        if (k2) {
            a = shfl_xor_u64(kmn2, sft);
            c2 = shfl_xor_u64(kmx2, sft);
            kmn2 = a < kmn2 ? a : kmn2;
            kmx2 = c2 > kmx2 ? c2 : kmx2;
        }
    }
    if (lane == 0) {
        sh.kmin[w] = kmn;
        sh.kmax[w] = kmx;
        sh.kmin1[w] = kmn2;
        sh.kmax1[w] = kmx2;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kWaves; q++) {
        kmn = sh.kmin[q] < kmn ? sh.kmin[q] : kmn;
        kmx = sh.kmax[q] > kmx ? sh.kmax[q] : kmx;
        kmn2 = sh.kmin1[q] < kmn2 ? sh.kmin1[q] : kmn2;
        kmx2 = sh.kmax1[q] > kmx2 ? sh.kmax1[q] : kmx2;
    }
}

// Exclusive scan of one value per thread over the block (every thread
// calls it; sh.wsum is used). Ends with a barrier.
__device__ __forceinline__ uint32_t block_excl_scan(BkShared &sh, uint32_t x)
{
    const int w = (int)(threadIdx.x >> 6);
    const uint32_t incl = wave_incl_scan_dpp(x);
    if (lane_id() == 63) sh.wsum[w] = incl;
    __syncthreads();
    uint32_t off = 0;
    for (int q = 0; q < w; q++) off += sh.wsum[q];
    __syncthreads();
    return off + incl - x;
}

// Rank pass: the place rank[r] of each of the m entries (entry idx =
// w * 64 R_eff + r * 64 + lane) in the order of key k, ties in entry order;
// kmn, kmx: the keys' range. Every thread of the block calls it; sh.bin,
// sh.lkey, sh.lj and sh.lslot are used, and k is left in an unspecified
// order.
//
// With k2 (not NULL) it ranks by (k, k2, entry) in one pass if it can: all
// entries (the smallest key included) go to the bins, and when no bin holds
// more than kBinMax2 of them each is ranked by counting inside its bin by
// (k, k2, entry). Otherwise it returns false without ranks, k unchanged
// (the caller then ranks by k2 and by k in two passes). The outcome is the
// same in every thread.
//
// Entries with the smallest key (the common heavy tie: aged scores clamped to
// the floor, or the lowest class of a bucket) come first, in entry order:
// their rank is the number of such entries before them, from ballots. The
// others go to bins, monotone in the key, over the range [x2, xmax] of the
// keys above the minimum: for a finite range, kBins equal intervals
// ((x - x2) * (kBins / (xmax - x2)), each step rounded, so monotone);
// otherwise the kBinBits bits of key - key2 below its highest varying bit.
// Their rank = entries at the minimum + bin start + rank inside the bin by
// (key, entry). A bin of more than kBinMax entries sends the whole bucket
// through stable LSD passes on the key bytes that vary in it instead.
__device__ __forceinline__ bool rank_pass(BkShared &sh, uint64_t *k, const uint64_t *k2, uint32_t reff, uint32_t m,
                                          uint64_t kmn, uint64_t kmx, uint32_t *rank, bool bins_zero = false)
{
    constexpr int kWaves = kBkTPB / 64;
    const uint32_t t = threadIdx.x;
    const int w = (int)(t >> 6), lane = lane_id();
    const uint32_t wk = 64u * reff;
    if (kmn >= kmx) {
        // one key (or no entry): entry order is the order
#pragma unroll
        for (int r = 0; r < kBkR; r++) rank[r] = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
        return !k2;   // one key: the order is by k2 alone
    }
    if (!bins_zero)
        for (uint32_t i = t; i <= kBins; i += kBkTPB) sh.bin[i] = 0;
    // excl: the minimum-key entries are ranked apart (one key only).
    // rank[r] first holds the number of minimum-key entries before entry r
    // (its rank if it has the minimum key; the valid entries are a prefix,
    // so entry idx has idx - rank[r] entries above the minimum before it)
    const bool excl = !k2;
    uint32_t nlow = 0;
    uint64_t kmn2 = excl ? ~0ull : kmn;   // smallest key of the binned entries
    if (excl) {
        uint32_t run = 0;
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            if ((uint32_t)r >= reff) break;
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            const bool valid = (uint32_t)r < reff && idx < m;
            const bool low = valid && k[r] == kmn;
            const uint64_t bl = __ballot(low);
            rank[r] = run + (uint32_t)__popcll(bl & lanemask_lt());
            run += (uint32_t)__popcll(bl);
            if (valid && !low && k[r] < kmn2) kmn2 = k[r];
        }
#pragma unroll
        for (int sft = 32; sft >= 1; sft >>= 1) {
            const uint64_t a = shfl_xor_u64(kmn2, sft);
            kmn2 = a < kmn2 ? a : kmn2;
        }
        if (lane == 0) {
            sh.wsum[w] = run;
            sh.kmin2[w] = kmn2;
        }
        __syncthreads();
        uint32_t before_w = 0;
        nlow = 0;
#pragma unroll
        for (int q = 0; q < kWaves; q++) {
            before_w += q < w ? sh.wsum[q] : 0u;
            nlow += sh.wsum[q];
            kmn2 = sh.kmin2[q] < kmn2 ? sh.kmin2[q] : kmn2;
        }
#pragma unroll
        for (int r = 0; r < kBkR; r++) rank[r] += before_w;
        __syncthreads();   // sh.wsum is reused by the bin scan
    } else if (!bins_zero) {
        __syncthreads();   // the bins are zero before any count goes in
    }
    if (kmn2 >= kmx) {
        // two distinct keys: each in entry order
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            if (k[r] != kmn) rank[r] = nlow + (idx - rank[r]);
        }
        return true;
    }
    // bins over [kmn2, kmx] for the binned entries
    const int hb = 63 - __clzll((long long)(kmn2 ^ kmx));
    const uint32_t shift = hb >= (int)kBinBits ? (uint32_t)hb - (kBinBits - 1u) : 0u;
    const double xmn = from_ordered(kmn2), xmx = from_ordered(kmx);
    const double span = xmx - xmn;
    const bool linear = isfinite(span) && span > 0.0 && isfinite((double)kBins / span);
    const double scale = linear ? (double)kBins / span : 0.0;
    // bin (low kBinBits bits) and slot in the bin (above them) of each entry
    uint32_t db[kBkR];
#pragma unroll
    for (int r = 0; r < kBkR; r++) {
        const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
        db[r] = 0;
        if ((uint32_t)r < reff && idx < m && (!excl || k[r] != kmn)) {
            uint32_t q;
            if (linear) {
                const double f = (from_ordered(k[r]) - xmn) * scale;   // in [0, kBins]
                q = f < (double)kBins ? (uint32_t)f : kBins - 1u;
            } else {
                q = (uint32_t)((k[r] - kmn2) >> shift);   // < kBins
            }
            db[r] = q | (atomicAdd(&sh.bin[q], 1u) << kBinBits);
        }
    }
    __syncthreads();
    // bin starts: thread t owns bins 4t .. 4t + 3
    {
        uint32_t hv[4], sum = 0, mx = 0;
#pragma unroll
        for (int e = 0; e < 4; e++) {
            hv[e] = sh.bin[4 * t + e];
            sum += hv[e];
            mx = hv[e] > mx ? hv[e] : mx;
        }
        const uint32_t incl = wave_incl_scan_dpp(sum);
#pragma unroll
        for (int sft = 32; sft >= 1; sft >>= 1) {
            const uint32_t o = (uint32_t)__shfl_xor((int)mx, sft, 64);
            mx = o > mx ? o : mx;
        }
        if (lane == 63) sh.wsum[w] = incl;
        if (lane == 0) sh.wmax[w] = mx;
        __syncthreads();
        uint32_t ex = incl - sum;
        for (int q = 0; q < w; q++) ex += sh.wsum[q];
#pragma unroll
        for (int e = 0; e < 4; e++) {
            sh.bin[4 * t + e] = ex;
            ex += hv[e];
        }
        if (t == 0) sh.bin[kBins] = m - nlow;
    }
    uint32_t maxbin = 0;
#pragma unroll
    for (int q = 0; q < kWaves; q++) maxbin = sh.wmax[q] > maxbin ? sh.wmax[q] : maxbin;
    __syncthreads();
    if (maxbin <= (excl ? kBinMax : kBinMax2)) {
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            if ((uint32_t)r < reff && idx < m && (!excl || k[r] != kmn)) {
                const uint32_t q = sh.bin[db[r] & (kBins - 1u)] + (db[r] >> kBinBits);
                sh.lkey[q] = k[r];
                if (k2) sh.lkey2[q] = k2[r];
                sh.lslot[q] = (uint16_t)idx;
            }
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            if ((uint32_t)r < reff && idx < m && (!excl || k[r] != kmn)) {
                const uint32_t bn = db[r] & (kBins - 1u);
                const uint32_t s0 = sh.bin[bn], s1 = sh.bin[bn + 1];
                uint32_t rk = nlow + s0;
                if (k2) {
                    for (uint32_t u = s0; u < s1; u++) {
                        const uint64_t ku = sh.lkey[u], k2u = sh.lkey2[u];
                        rk += key_less(ku, k2u, sh.lslot[u], k[r], k2[r], idx) ? 1u : 0u;
                    }
                } else {
                    for (uint32_t u = s0; u < s1; u++) {
                        const uint64_t ku = sh.lkey[u];
                        rk += (ku < k[r] || (ku == k[r] && sh.lslot[u] < idx)) ? 1u : 0u;
                    }
                }
                rank[r] = rk;
            }
        }
        __syncthreads();   // sh.lkey, sh.lkey2, sh.lslot are free again
        return true;
    }
    if (linear) {
        // crowded bins (keys in clusters with gaps between them, which the
        // equal-width bins spread over): bin b of c_b entries is cut into c_b
        // equal sub-intervals, one sub-bin each, by the fraction of the key
        // inside the bin (the same rounded operations, so monotone). The
        // sub-bins of bin b start at the bin's start; their counts and starts
        // use sh.lj.
        const uint32_t nb2 = m - nlow;   // sub-bins, one per binned entry
        for (uint32_t i = t; i <= nb2; i += kBkTPB) sh.lj[i] = 0;
        __syncthreads();
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            if ((uint32_t)r < reff && idx < m && (!excl || k[r] != kmn)) {
                const uint32_t bn = db[r] & (kBins - 1u);
                const uint32_t s0 = sh.bin[bn], cb = sh.bin[bn + 1] - s0;
                const double f = (from_ordered(k[r]) - xmn) * scale - (double)bn;   // in [0, 1)
                uint32_t sub = f > 0.0 ? (uint32_t)(f * (double)cb) : 0u;
                sub = sub < cb ? sub : cb - 1u;
                const uint32_t sb = s0 + sub;
                db[r] = sb | (atomicAdd(&sh.lj[sb], 1u) << 12);
            }
        }
        __syncthreads();
        // sub-bin starts: thread t scans sub-bins 8t .. 8t + 7
        uint32_t hv[kCap / kBkTPB], sum = 0, mx = 0;
#pragma unroll
        for (int e = 0; e < (int)(kCap / kBkTPB); e++) {
            const uint32_t i = (uint32_t)t * (kCap / kBkTPB) + (uint32_t)e;
            hv[e] = i < nb2 ? sh.lj[i] : 0u;
            sum += hv[e];
            mx = hv[e] > mx ? hv[e] : mx;
        }
#pragma unroll
        for (int sft = 32; sft >= 1; sft >>= 1) {
            const uint32_t o = (uint32_t)__shfl_xor((int)mx, sft, 64);
            mx = o > mx ? o : mx;
        }
        if (lane == 0) sh.wmax[w] = mx;
        uint32_t ex = block_excl_scan(sh, sum);
#pragma unroll
        for (int e = 0; e < (int)(kCap / kBkTPB); e++) {
            const uint32_t i = (uint32_t)t * (kCap / kBkTPB) + (uint32_t)e;
            if (i < nb2) sh.lj[i] = ex;
            ex += hv[e];
        }
        if (t == 0) sh.lj[nb2] = nb2;
        uint32_t maxsub = 0;
#pragma unroll
        for (int q = 0; q < kWaves; q++) maxsub = sh.wmax[q] > maxsub ? sh.wmax[q] : maxsub;
        __syncthreads();
        if (maxsub <= (excl ? kBinMax : kBinMax2)) {
#pragma unroll
            for (int r = 0; r < kBkR; r++) {
                const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
                if ((uint32_t)r < reff && idx < m && (!excl || k[r] != kmn)) {
                    const uint32_t q = sh.lj[db[r] & 4095u] + (db[r] >> 12);
                    sh.lkey[q] = k[r];
                    sh.lkey2[q] = k2 ? k2[r] : 0ull;
                    sh.lslot[q] = (uint16_t)idx;
                }
            }
            __syncthreads();
#pragma unroll
            for (int r = 0; r < kBkR; r++) {
                const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
                if ((uint32_t)r < reff && idx < m && (!excl || k[r] != kmn)) {
                    const uint32_t sb = db[r] & 4095u;
                    const uint32_t s0 = sh.lj[sb], s1 = sh.lj[sb + 1];
                    const uint64_t e2 = k2 ? k2[r] : 0ull;
                    uint32_t rk = nlow + s0;
                    for (uint32_t u = s0; u < s1; u++)
                        rk += key_less(sh.lkey[u], sh.lkey2[u], sh.lslot[u], k[r], e2, idx) ? 1u : 0u;
                    rank[r] = rk;
                }
            }
            __syncthreads();
            return true;
        }
    }
    if (k2) return false;
    // crowded bins (many equal or near-equal keys): stable LSD passes over
    // all the entries, on the key bytes up to the highest bit that varies in
    // the bucket (minimum included); the entries carry their index along,
    // and the final order gives each its rank
    const int hba = 63 - __clzll((long long)(kmn ^ kmx));
    const uint64_t diff = hba == 63 ? ~0ull : ((1ull << (hba + 1)) - 1ull);
    for (uint32_t i = t; i < 2u * kWaves * 256u; i += kBkTPB) (&sh.wcnt[0][0][0])[i] = 0;
    uint64_t *kk = k;
    uint32_t slot[kBkR], pos[kBkR];
#pragma unroll
    for (int r = 0; r < kBkR; r++) slot[r] = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
    __syncthreads();
    uint32_t cur = 0;
    for (uint32_t p = 0; p < 8; p++) {
        if (((diff >> (8 * p)) & 255u) == 0) continue;   // uniform
        uint32_t tc;
        lds_rank(sh, cur, kk, reff, m, p, pos, tc);
        cur ^= 1u;
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            if ((uint32_t)r < reff && idx < m) {
                sh.lkey[pos[r]] = kk[r];
                sh.lj[pos[r]] = slot[r];
            }
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            if ((uint32_t)r < reff && idx < m) {
                kk[r] = sh.lkey[idx];
                slot[r] = sh.lj[idx];
            }
        }
        __syncthreads();
    }
    // entry slot[r] is now at place idx
#pragma unroll
    for (int r = 0; r < kBkR; r++) {
        const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
        if ((uint32_t)r < reff && idx < m) sh.lslot[slot[r]] = (uint16_t)idx;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kBkR; r++) {
        const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
        rank[r] = (uint32_t)r < reff && idx < m ? sh.lslot[idx] : 0u;
    }
    __syncthreads();
    return true;
}

// Requests per tier and each class's first position, into sh.pt; clears the
// digit counters. Every thread calls pw_params, then (after a barrier)
// pw_starts; load_pw does both.
__device__ __forceinline__ void pw_params(const SsBatch &b, const SsDesc &d, BkShared &sh)
{
    const uint32_t t = threadIdx.x;
    if (t < kQ) {
        sh.pt.tot[t] = d.tot[t];
        sh.pt.prio[t] = b.in.prio[t];
        sh.pt.cls[t] = b.in.cls[t];
        sh.pt.weight[t] = b.in.weight[t];
    }
    if (t < 2 * kQ) sh.pt.cnt[t] = 0;
    for (uint32_t i = t; i < (kBkTPB / 64) * 2 * kQ; i += kBkTPB) (&sh.pt.wd[0][0])[i] = 0;
    if (d.pw_out[1] && b.in.wrr_mode == kWrrSmooth)
        for (uint32_t i = t; i < sizeof(WrrPlanHead) / 4; i += kBkTPB)
            reinterpret_cast<uint32_t *>(&sh.pt.wh)[i] = reinterpret_cast<const uint32_t *>(&b.plan->h)[i];
}

__device__ __forceinline__ void pw_starts(const SsBatch &b, BkShared &sh)
{
    const uint32_t t = threadIdx.x;
    if (t < kQ) {
        uint32_t s = 0;
        for (uint32_t q = 0; q < b.in.n_tiers && q < kQ; q++) s += sh.pt.cls[q] < t ? sh.pt.tot[q] : 0u;
        sh.pt.cstart[t] = s;
    }
}

__device__ __forceinline__ void load_pw(const SsBatch &b, const SsDesc &d, BkShared &sh)
{
    pw_params(b, d, sh);
    __syncthreads();
    pw_starts(b, sh);
}

// Stable ranks of this thread's entries (wave-major, entry idx =
// w * 64 R_eff + r * 64 + lane, valid below m) among the entries of the
// same class (rc) and of the same tier (rt) of the run, from ballots and
// the per-wave counters sh.pt.wd (zero on entry; afterwards each wave's
// exclusive start per digit). Ends with a barrier.
__device__ __forceinline__ void pw_rank(const SsBatch &b, BkShared &sh, const uint32_t *q, uint32_t reff, uint32_t m,
                                        uint32_t *rc, uint32_t *rt)
{
    constexpr int kWaves = kBkTPB / 64;
    const uint32_t t = threadIdx.x;
    const int w = (int)(t >> 6), lane = lane_id();
    const uint32_t wk = 64u * reff;
#pragma unroll
    for (int r = 0; r < kBkR; r++) {
        rc[r] = 0;
        rt[r] = 0;
        if ((uint32_t)r < reff) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            const bool ok = idx < m;
            const uint32_t dc = sh.pt.cls[q[r]], dt = q[r];
            uint64_t pc = __ballot(ok), pt = pc;
#pragma unroll
            for (int bb = 0; bb < 4; bb++) {
                const bool xc = (dc >> bb) & 1u, xt = (dt >> bb) & 1u;
                const uint64_t mc = __ballot(xc), mt = __ballot(xt);
                pc &= xc ? mc : ~mc;
                pt &= xt ? mt : ~mt;
            }
            const uint32_t bc = (uint32_t)__popcll(pc & lanemask_lt()), bt = (uint32_t)__popcll(pt & lanemask_lt());
            const uint32_t oc = ok ? sh.pt.wd[w][dc] : 0u, ot = ok ? sh.pt.wd[w][kQ + dt] : 0u;
            rc[r] = oc + bc;
            rt[r] = ot + bt;
            if (ok && bc == 0) sh.pt.wd[w][dc] = oc + (uint32_t)__popcll(pc);
            if (ok && bt == 0) sh.pt.wd[w][kQ + dt] = ot + (uint32_t)__popcll(pt);
            __builtin_amdgcn_wave_barrier();
        }
    }
    __syncthreads();
    if (t < 2 * kQ) {
        uint32_t acc = 0;
#pragma unroll
        for (int v = 0; v < kWaves; v++) {
            const uint32_t c = sh.pt.wd[v][t];
            sh.pt.wd[v][t] = acc;
            acc += c;
        }
        sh.pt.cnt[t] = acc;   // the run's digit counts
    }
    __syncthreads();
}

// The whole batch sorted by one workgroup: stable LSD passes over global
// ping-pong buffers, in chunks of kCap entries taken in order; by k2 first
// (two-key sorts), then by k1.
__device__ __forceinline__ void serial_sort(const SsBatch &b, const SsDesc &d, BkShared &sh)
{
    const uint32_t n = b.n, t = threadIdx.x;
    const int w = (int)(t >> 6), lane = lane_id();
    for (uint32_t i = t; i < 2u * (kBkTPB / 64) * 256u; i += kBkTPB) (&sh.wcnt[0][0][0])[i] = 0;
    uint32_t cur = 0;
    for (uint32_t j = t; j < n; j += kBkTPB) {
        uint64_t k1, k2;
        double kv;
        with_kind(d.kind, [&](auto K) { ss_key<decltype(K)::value>(b.in, j, k1, k2, kv); });
        d.fk1[0][j] = k1;
        d.fk2[0][j] = k2;
        d.fj[0][j] = j;
        if (d.key_out) d.key_out[j] = kv;
    }
    __syncthreads();
    uint32_t src = 0;
    for (uint32_t pass = 0; pass < 16; pass++) {
        // bytes 0..7 of k2, then of k1; a pass whose digit is the same for
        // all keys is skipped
        const bool on_k1 = pass >= 8;
        const uint32_t p = pass & 7u;
        if (!on_k1 && !d.two) continue;
        const uint64_t *ksrc = on_k1 ? d.fk1[src] : d.fk2[src];
        if (t < 256) sh.offs[t] = 0;
        __syncthreads();
        for (uint32_t j = t; j < n; j += kBkTPB) atomicAdd(&sh.offs[(uint32_t)(ksrc[j] >> (8 * p)) & 255u], 1u);
        __syncthreads();
        const uint32_t h = t < 256 ? sh.offs[t] : 0u;
        const int constant = __syncthreads_or(t < 256 && h == n);
        if (constant) continue;
        const uint32_t ex = block_excl_scan_digits<kBkTPB>(h, sh.tmp4);
        if (t < 256) sh.offs[t] = ex;
        __syncthreads();
        for (uint32_t c0 = 0; c0 < n; c0 += kCap) {
            const uint32_t m = n - c0 < kCap ? n - c0 : kCap;
            const uint32_t reff = (m + kBkTPB - 1) / kBkTPB;
            const uint32_t wk = 64u * reff;
            uint64_t k[kBkR];
            uint32_t pos[kBkR];
#pragma unroll
            for (int r = 0; r < kBkR; r++) {
                const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
                k[r] = (uint32_t)r < reff && idx < m ? ksrc[c0 + idx] : 0ull;
            }
            uint32_t tc;
            lds_rank(sh, cur, k, reff, m, p, pos, tc);
            cur ^= 1u;
#pragma unroll
            for (int r = 0; r < kBkR; r++) {
                const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
                if ((uint32_t)r < reff && idx < m) {
                    const uint32_t dg = (uint32_t)(k[r] >> (8 * p)) & 255u;
                    // rank in the chunk minus the chunk's digit start, plus
                    // the digit's running offset
                    const uint32_t g = sh.offs[dg] + pos[r] - sh.texcl[dg];
                    d.fk1[src ^ 1u][g] = d.fk1[src][c0 + idx];
                    d.fk2[src ^ 1u][g] = d.fk2[src][c0 + idx];
                    d.fj[src ^ 1u][g] = d.fj[src][c0 + idx];
                }
            }
            __syncthreads();
            if (t < 256) sh.offs[t] += tc;
            __syncthreads();
        }
        src ^= 1u;
    }
    if (d.out)
        for (uint32_t i = t; i < n; i += kBkTPB) d.out[i] = d.fj[src][i];
    if (!d.pw_out[0] && !d.pw_out[1]) return;
    // Priority and Weighted over the FIFO sequence, a chunk of kBkTPB
    // positions at a time (one per thread), with running digit counts
    load_pw(b, d, sh);
    if (t < 2 * kQ) sh.pt.pre[t] = 0;
    __syncthreads();
    for (uint32_t c0 = 0; c0 < n; c0 += kBkTPB) {
        const uint32_t m = n - c0 < kBkTPB ? n - c0 : kBkTPB;
        uint32_t q[kBkR], rc[kBkR], rt[kBkR];
        uint32_t j = 0;
#pragma unroll
        for (int r = 0; r < kBkR; r++) q[r] = 0;
        if (t < m) {
            j = d.fj[src][c0 + t];
            j = j < n ? j : 0u;
            const uint32_t qq = b.in.tier[j];
            q[0] = qq < kQ ? qq : kQ - 1u;
        }
        pw_rank(b, sh, q, 1u, m, rc, rt);
        if (t < m) {
            const uint32_t c = sh.pt.cls[q[0]];
            pw_place(b, d, sh.pt, q[0], j, sh.pt.pre[c] + sh.pt.wd[w][c] + rc[0],
                     sh.pt.pre[kQ + q[0]] + sh.pt.wd[w][kQ + q[0]] + rt[0]);
        }
        __syncthreads();
        if (t < 2 * kQ) sh.pt.pre[t] += sh.pt.cnt[t];
        for (uint32_t i = t; i < (kBkTPB / 64) * 2 * kQ; i += kBkTPB) (&sh.pt.wd[0][0])[i] = 0;
        __syncthreads();
    }
}

__global__ __launch_bounds__(kBkTPB) void k_ss_bucket(SsBatch b)
{
    constexpr int kWaves = kBkTPB / 64;
    __shared__ BkShared sh;
    const SsDesc &d = b.s[blockIdx.y];
    const uint32_t t = threadIdx.x, bkt = blockIdx.x, n = b.n;
    const int w = (int)(t >> 6), lane = lane_id();
    if (ld_relaxed(&d.ctl->overflow)) {
        if (bkt == 0) serial_sort(b, d, sh);
        return;
    }
    if (bkt >= d.nb) return;   // a row with fewer buckets than the grid is wide
    const bool pw = d.pw_out[0] || d.pw_out[1];   // FIFO row with the partitions
    const uint64_t *src1 = d.bk1 + (uint64_t)bkt * kCap;
    const uint64_t *src2 = d.bk2 + (uint64_t)bkt * kCap;
    const uint32_t *srcj = d.bj + (uint64_t)bkt * kCap;
    const bool two = d.two != 0;
    // the first kPreSlots slots are loaded before the size is known, four
    // per thread, and staged in LDS, from where each thread takes its entries
    // in the layout the size gives (a bucket of at most kPreSlots requests,
    // twice the average, needs no other global load)
    constexpr uint32_t kPreR = 4, kPreSlots = kPreR * kBkTPB;
    static_assert(kPreSlots <= kCap, "staged slots lie in the region");
    uint64_t pa[kPreR], pb[kPreR];
    uint32_t pj[kPreR];
#pragma unroll
    for (uint32_t i = 0; i < kPreR; i++) {
        const uint32_t s = t + i * kBkTPB;
        pa[i] = src1[s];
        pb[i] = two ? src2[s] : 0ull;
        pj[i] = srcj[s];
    }
    // the partitions' parameters (their loads in flight with the slots'),
    // and the bins of the first rank pass cleared, before the size barrier
    if (pw) pw_params(b, d, sh);
    for (uint32_t i = t; i <= kBins; i += kBkTPB) sh.bin[i] = 0;
    // bucket sizes: the last tile's inclusive prefixes
    const uint32_t *last = d.status + (uint64_t)(b.tiles - 1) * 256u;
    const uint32_t c = t < d.nb ? (last[t] & kValMask) : 0u;
    const uint32_t before = wave_sum(t < bkt ? c : 0u);
    if (lane == 0) sh.redu[w] = before;
    if (t == bkt) sh.offs[0] = c;
#pragma unroll
    for (uint32_t i = 0; i < kPreR; i++) {
        const uint32_t s = t + i * kBkTPB;
        sh.lkey[s] = pa[i];
        if (two) sh.lkey2[s] = pb[i];
        sh.lj[s] = pj[i];
    }
    __syncthreads();
    uint32_t off = 0;
#pragma unroll
    for (int q = 0; q < kWaves; q++) off += sh.redu[q];
    const uint32_t m = sh.offs[0];   // <= kCap: no region overflowed
    const uint32_t reff = (m + kBkTPB - 1) / kBkTPB;
    const uint32_t wk = 64u * reff;

    // the entries (index order within the bucket) and the keys' ranges
    if (pw) pw_starts(b, sh);
    uint64_t k[kBkR], k2[kBkR];
    uint32_t jv[kBkR], rank[kBkR], q[kBkR];
#pragma unroll
    for (int r = 0; r < kBkR; r++) {
        const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
        k[r] = 0;
        k2[r] = 0;
        jv[r] = 0;
        q[r] = 0;
        if ((uint32_t)r < reff && idx < m) {
            if (idx < kPreSlots) {
                k[r] = sh.lkey[idx];
                if (two) k2[r] = sh.lkey2[idx];
                jv[r] = sh.lj[idx];
            } else {
                k[r] = src1[idx];
                if (two) k2[r] = src2[idx];
                jv[r] = srcj[idx];
            }
        }
    }
    if (pw) {
        // the bucket's digit counts (order-free), published before its own
        // ranking so that later buckets need not wait for it
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            if ((uint32_t)r < reff && idx < m) {
                const uint32_t qq = jv[r] >> kIdxBits;   // the tier, packed by the scatter
                jv[r] &= kIdxMask;
                q[r] = qq < kQ ? qq : kQ - 1u;
                atomicAdd(&sh.pt.cnt[sh.pt.cls[q[r]]], 1u);
                atomicAdd(&sh.pt.cnt[kQ + q[r]], 1u);
            }
        }
    }
    uint64_t mn1, mx1, mn2, mx2;
    // (two calls, so that k2 is never behind a pointer chosen at run time,
    // which would move the array out of registers)
    if (two)
        block_range(sh, k, k2, reff, m, mn1, mx1, mn2, mx2);
    else
        block_range(sh, k, nullptr, reff, m, mn1, mx1, mn2, mx2);
    if (pw && t < 2 * kQ)
        st_relaxed(&d.bstat[(uint64_t)bkt * 2 * kQ + t], (bkt == 0 ? kPre : kAgg) | sh.pt.cnt[t]);
    // One pass by (k1, k2, index) where the bucket allows it; FIFO takes it
    // too, with k2 = 0 (every entry binned, no separate pass for the ties
    // at the minimum). Otherwise stable passes: by arrival (ties: index
    // order, which is entry order), then by k1 with the entries laid out in
    // arrival order (skipped when the bucket holds one k1); FIFO: one pass
    // by arrival.
    const bool both = two && mn1 < mx1;
    bool done = (both || (!two && mn1 < mx1)) && rank_pass(sh, k, k2, reff, m, mn1, mx1, rank, true);
    if (!done) {
        const uint32_t npass = both ? 2u : 1u;
        for (uint32_t ps = 0; ps < npass; ps++) {
            uint64_t lo = mn1, hi = mx1;
            if (ps == 0 && two) {
#pragma unroll
                for (int r = 0; r < kBkR; r++) k[r] = k2[r];
                lo = mn2;
                hi = mx2;
            }
            if (ps == 1) {
#pragma unroll
                for (int r = 0; r < kBkR; r++) {
                    const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
                    if ((uint32_t)r < reff && idx < m) {
                        sh.lkey[rank[r]] = src1[idx];
                        sh.lj[rank[r]] = jv[r];
                    }
                }
                __syncthreads();
#pragma unroll
                for (int r = 0; r < kBkR; r++) {
                    const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
                    k[r] = 0;
                    jv[r] = 0;
                    if ((uint32_t)r < reff && idx < m) {
                        k[r] = sh.lkey[idx];
                        jv[r] = sh.lj[idx];
                    }
                }
                __syncthreads();
            }
            rank_pass(sh, k, nullptr, reff, m, lo, hi, rank);
        }
    }
    if (pw) {
        // the bucket's requests in FIFO order, and the digits' counts over
        // the buckets before it
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            if ((uint32_t)r < reff && idx < m) {
                sh.lq[rank[r]] = (uint8_t)q[r];
                sh.lj[rank[r]] = jv[r];
            }
        }
        if (t < 2 * kQ) {
            uint32_t pre = 0;
            if (bkt > 0) {
                pre = look_back<2 * kQ>(d.bstat, bkt, t,
                                        b.in.wait.status ? b.in.wait.status : &d.ctl->lb_err,
                                        b.in.wait.no_wait ? 0u : kSpinLimit);
                st_relaxed(&d.bstat[(uint64_t)bkt * 2 * kQ + t], kPre | (pre + sh.pt.cnt[t]));
            }
            sh.pt.pre[t] = pre;
        }
        __syncthreads();
        uint32_t jf[kBkR], rc[kBkR], rt[kBkR];
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            const bool ok = (uint32_t)r < reff && idx < m;
            q[r] = ok ? sh.lq[idx] : 0u;
            jf[r] = ok ? sh.lj[idx] : 0u;
        }
        pw_rank(b, sh, q, reff, m, rc, rt);
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            if ((uint32_t)r < reff && idx < m) {
                const uint32_t c = sh.pt.cls[q[r]];
                pw_place(b, d, sh.pt, q[r], jf[r], sh.pt.pre[c] + sh.pt.wd[w][c] + rc[r],
                         sh.pt.pre[kQ + q[r]] + sh.pt.wd[w][kQ + q[r]] + rt[r]);
            }
        }
    }
    if (d.out) {
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            if ((uint32_t)r < reff && idx < m && off + rank[r] < n) d.out[off + rank[r]] = jv[r];
        }
    }
}

uint32_t n_buckets(uint64_t n, uint32_t avg = kBucketAvg)
{
    const uint64_t b = cdiv(n, avg);
    return (uint32_t)(b < 1 ? 1 : (b > kMaxBuckets ? kMaxBuckets : b));
}

uint32_t n_samples(uint64_t n)
{
    // 1024 samples up to 2^17 requests, 2048 above: 8 to 16 per bucket of
    // the SJF and Aging rows (an average bucket of at most a quarter of the
    // region), 4 to 8 per bucket of the FIFO row (at most an eighth)
    const uint64_t smax = n <= (1u << 17) ? kSamples / 2 : kSamples;
    return (uint32_t)(n < smax ? n : smax);
}

uint32_t sample_blocks(uint64_t n)
{
    const uint32_t ns = n_samples(n);
    return (uint32_t)cdiv(ns ? ns : 1, kSmpPerBlock);
}

uint64_t region_bytes(uint64_t n)
{
    const uint64_t tiles = cdiv(n, kScTile);
    const uint64_t nb = n_buckets(n, kBucketAvgFifo);   // every row's regions hold the most buckets
    return align_up(sizeof(SsCtl), 256) + 2 * align_up(kSamples * 8, 256) + align_up(kSamples * 4, 256) +
           align_up(tiles * 256 * 4, 256) + 2 * align_up(nb * kCap * 8, 256) + align_up(nb * kCap * 4, 256) +
           align_up(kQ * 4, 256) + align_up(nb * 2 * kQ * 4, 256) + 4 * align_up(n * 8, 256) +
           2 * align_up(n * 4, 256);
}

void carve(uint8_t *p, uint64_t n, SsDesc &d)
{
    const uint64_t tiles = cdiv(n, kScTile);
    const uint64_t nb = n_buckets(n, kBucketAvgFifo);
    auto take = [&](uint64_t bytes) {
        uint8_t *q = p;
        p += align_up(bytes, 256);
        return q;
    };
    d.ctl = reinterpret_cast<SsCtl *>(take(sizeof(SsCtl)));
    d.smp_k1 = reinterpret_cast<uint64_t *>(take(kSamples * 8));
    d.smp_k2 = reinterpret_cast<uint64_t *>(take(kSamples * 8));
    d.smp_j = reinterpret_cast<uint32_t *>(take(kSamples * 4));
    d.status = reinterpret_cast<uint32_t *>(take(tiles * 256 * 4));
    d.bk1 = reinterpret_cast<uint64_t *>(take(nb * kCap * 8));
    d.bk2 = reinterpret_cast<uint64_t *>(take(nb * kCap * 8));
    d.bj = reinterpret_cast<uint32_t *>(take(nb * kCap * 4));
    d.tot = reinterpret_cast<uint32_t *>(take(kQ * 4));
    d.bstat = reinterpret_cast<uint32_t *>(take(nb * 2 * kQ * 4));
    for (int i = 0; i < 2; i++) d.fk1[i] = reinterpret_cast<uint64_t *>(take(n * 8));
    for (int i = 0; i < 2; i++) d.fk2[i] = reinterpret_cast<uint64_t *>(take(n * 8));
    for (int i = 0; i < 2; i++) d.fj[i] = reinterpret_cast<uint32_t *>(take(n * 4));
}


}  // namespace

size_t ssort_ws_bytes(uint64_t n, uint32_t nsorts)
{
    return n <= kSsMaxN ? (size_t)(align_up(sizeof(WrrPlan), 256) + align_up(n * 4, 256) +
                                   (uint64_t)nsorts * region_bytes(n))
                        : 0;
}

hipError_t ssort_launch(const SortInput &in, const SortJob *jobs, uint32_t nsorts, bool serial, void *ws,
                        hipStream_t s, const SsPartitions *parts)
{
    if (in.n == 0 || nsorts == 0) return hipSuccess;
    if (nsorts > kSsMaxSorts || in.n > kSsMaxN) return hipErrorInvalidValue;
    SsBatch b;
    memset(&b, 0, sizeof(b));
    b.in = in;
    b.n = in.n;
    b.tiles = (uint32_t)cdiv(in.n, kScTile);
    b.nb = 1;
    b.ns = n_samples(in.n);
    b.serial = serial ? 1u : 0u;
    b.nsorts = nsorts;
    b.nsb = sample_blocks(in.n);
    uint8_t *p = static_cast<uint8_t *>(ws);
    b.plan = reinterpret_cast<WrrPlan *>(p);
    p += align_up(sizeof(WrrPlan), 256);
    b.tpos = reinterpret_cast<uint32_t *>(p);
    p += align_up((uint64_t)in.n * 4, 256);
    for (uint32_t i = 0; i < nsorts; i++) {
        SsDesc &d = b.s[i];
        const SortKind k = jobs[i].kind;
        if (k != SortKind::Fifo && k != SortKind::Budget && k != SortKind::Aging) return hipErrorInvalidValue;
        d.kind = k;
        d.nb = n_buckets(in.n, k == SortKind::Fifo ? kBucketAvgFifo : kBucketAvg);
        b.nb = d.nb > b.nb ? d.nb : b.nb;
        if (k == SortKind::Fifo && parts && (parts->perm[0] || parts->perm[1])) {
            for (int e = 0; e < 2; e++) {
                d.pw_out[e] = parts->perm[e];
                d.pw_key[e] = parts->perm[e] ? parts->key[e] : nullptr;
            }
        }
        d.two = k != SortKind::Fifo;
        d.key_out = jobs[i].key_out;
        d.out = jobs[i].out;
        carve(p, in.n, d);
        p += region_bytes(in.n);
    }
    hipLaunchKernelGGL(k_ss_sample, dim3(b.nsb, nsorts), dim3(kSmpTPB), 0, s, b);
    hipLaunchKernelGGL(k_ss_scatter, dim3(b.tiles, nsorts), dim3(kScTPB), 0, s, b);
    hipLaunchKernelGGL(k_ss_bucket, dim3(b.nb, nsorts), dim3(kBkTPB), 0, s, b);
    return hipGetLastError();
}

}  // namespace ds
