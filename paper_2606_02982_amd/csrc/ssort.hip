// Sample sort of (64-bit key, position) pairs for batches of up to 2^18
// requests, where the dispatch orders are latency-bound: three launches per
// batch of sorts instead of one launch per 8-bit digit.
//
// Every sort orders positions j = 0..n-1 of a sequence by (key_j, j); its
// output is the value of each position in that order (j itself for the FIFO
// sort, the j-th request of the FIFO sequence for SJF and Aging). Since the
// pairs are distinct, the result is the unique stable order whatever the
// intermediate arrangement.
//
//   k_ss_sample   produces S pairs (1024 up to 2^17 keys, else 2048) at
//                 stratified random positions;
//                 each of S/8 blocks stages all of them in LDS and finds the
//                 rank of 8 of them by counting the smaller ones, and stores
//                 each at its rank: the sorted sample, of which every
//                 (S/B)-th pair is one of B - 1 splitters. Also clears the
//                 look-back words and the overflow flag.
//   k_ss_scatter  per tile of 2048 positions: produces the pairs (and the
//                 per-request key output), finds each pair's bucket by binary
//                 search over the splitters, ranks the tile by bucket (wave
//                 ballots), takes the bucket prefix of earlier tiles by
//                 decoupled look-back and writes each key with its output
//                 value into the bucket's fixed-capacity region, so that a
//                 bucket holds its pairs in position order.
//   k_ss_bucket   one block per bucket (its offset: the sizes of the
//                 buckets before it): bins the pairs into 2048 intervals of
//                 the bucket's key range (an LDS histogram and its scan), and
//                 ranks each pair inside its bin by (key, position) by
//                 counting; a bucket with a bin of more than 64 pairs runs
//                 stable LSD passes over its varying key bytes instead.
// A bucket that outgrows its region (only for inputs arranged against the
// sampling) sets the overflow flag; k_ss_bucket then sorts the whole
// sequence in one workgroup with the same LSD passes over global memory.
#include <string.h>

#include "common.h"
#include "kernels.h"
#include "keys.h"
#include "lookback.h"
#include "partbody.h"
#include "tiercount.h"

namespace ds {
namespace {

constexpr uint32_t kSamples = 2048;      // pairs sampled per sort (at most)
constexpr uint32_t kCap = 4096;          // pairs per bucket region
constexpr uint32_t kMaxBuckets = 256;
constexpr uint32_t kBucketAvg = 256;     // target pairs per bucket
constexpr int kScTPB = 512, kScR = 4;    // scatter tile: 2048 positions
constexpr uint32_t kScTile = kScTPB * kScR;
constexpr int kBkTPB = 512, kBkR = kCap / kBkTPB;
constexpr uint32_t kBinBits = 11, kBins = 1u << kBinBits;   // in-bucket bins
constexpr uint32_t kBinMax = 64;         // larger bins: LSD passes instead
constexpr int kSmpTPB = 256;            // k_ss_sample: threads per block,
constexpr uint32_t kSmpThr = 32;         // threads per sample ranked,
constexpr uint32_t kSmpPerBlock = kSmpTPB / kSmpThr;   // samples ranked per block

struct SsCtl {
    uint32_t overflow;
    uint32_t pad[63];
};

struct SsDesc {
    SortKind kind;
    double *key_out;
    uint32_t *out;
    SsCtl *ctl;
    uint64_t *smp_k;       // [kSamples] the sample in sorted order
    uint32_t *smp_j;
    uint32_t *status;      // [tiles][256] look-back words
    uint64_t *bkey;        // [buckets][kCap] bucket regions: keys and output values
    uint32_t *bj;
    uint64_t *fkey[2];     // [n] x 2: single-workgroup sort
    uint32_t *fj[2];
};

struct SsBatch {
    SortInput in;
    uint32_t n;
    uint32_t tiles;        // scatter tiles
    uint32_t nb;           // buckets, 1..kMaxBuckets
    uint32_t ns;           // samples, 1..kSamples
    uint32_t serial;       // sort in one workgroup regardless of the buckets
    uint32_t nsorts;       // sorts of the batch (grid rows 0 .. nsorts - 1)
    uint32_t nsb;          // blocks of k_ss_sample per sort
    SsSide side;           // side work for the launches after this sort
    PartBatch part;        // Priority/Weighted tiles run by k_ss_sample (rows nsorts ..)
    SsDesc s[kMaxSorts];
};

// Value emitted for position j: the FIFO sort reorders the requests
// themselves; SJF and Aging reorder the FIFO sequence.
__device__ __forceinline__ uint32_t value_of(const SortInput &in, SortKind kind, uint32_t n, uint32_t j)
{
    if (kind == SortKind::Fifo) return j;
    const uint32_t i = in.fifo[j < n ? j : 0];
    return i < n ? i : 0u;
}

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

__device__ __forceinline__ bool pair_less(uint64_t ka, uint32_t ja, uint64_t kb, uint32_t jb)
{
    return ka < kb || (ka == kb && ja < jb);
}

template <SortKind K>
__device__ __forceinline__ void sample_body(const SsBatch &b, const SsDesc &d, uint64_t *sk, uint32_t *sj)
{
    const uint32_t t = threadIdx.x, n = b.n, S = b.ns;
    const uint32_t stride = b.nsb * kSmpTPB;
    for (uint32_t i = blockIdx.x * kSmpTPB + t; i < b.tiles * 256u; i += stride) d.status[i] = 0;
    if (blockIdx.x == 0 && t == 0) d.ctl->overflow = b.serial;
    if (blockIdx.y == 0) {
        for (uint32_t i = blockIdx.x * kSmpTPB + t; i < b.side.clear_words; i += stride) b.side.clear[i] = 0;
        if (b.side.tier_part)
            tier_partial<kSmpTPB>(b.in.tier, n, blockIdx.x, b.nsb, b.side.tier_part,
                                  reinterpret_cast<uint32_t *>(sk));
        __syncthreads();   // sk is reused below
    }
    {
        // all gathers in flight before the first LDS store
        constexpr int kPer = kSamples / kSmpTPB;
        double kv[kPer];
        uint32_t j[kPer];
#pragma unroll
        for (int r = 0; r < kPer; r++) {
            const uint32_t s = (uint32_t)r * kSmpTPB + t;
            j[r] = s < S ? sample_pos(s, n, S) : 0u;
            uint32_t v;
            kv[r] = primary_key<K>(b.in, n, j[r], v);
        }
#pragma unroll
        for (int r = 0; r < kPer; r++) {
            // unused slots hold the largest pair, below no sample
            const uint32_t s = (uint32_t)r * kSmpTPB + t;
            sk[s] = s < S ? ordered_bits(kv[r]) : ~0ull;
            sj[s] = s < S ? j[r] : ~0u;
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
        const uint64_t ks = sk[sc];
        const uint32_t js = sj[sc];
        uint32_t part[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        const uint32_t Sp = (S + 8 * kSmpThr - 1) / (8 * kSmpThr) * (8 * kSmpThr);   // <= kSamples
        for (uint32_t u0 = 0; u0 < Sp; u0 += 8 * kSmpThr) {
            uint64_t ku[8];
            uint32_t ju[8];
#pragma unroll
            for (uint32_t e = 0; e < 8; e++) {
                ku[e] = sk[u0 + e * kSmpThr + q];
                ju[e] = sj[u0 + e * kSmpThr + q];
            }
#pragma unroll
            for (uint32_t e = 0; e < 8; e++) part[e] += pair_less(ku[e], ju[e], ks, js) ? 1u : 0u;
        }
#pragma unroll
        for (uint32_t e = 0; e < 8; e++) below += part[e];
    }
#pragma unroll
    for (int m = kSmpThr / 2; m >= 1; m >>= 1) below += (uint32_t)__shfl_xor((int)below, m, 64);
    if (s < S && q == 0) {
        d.smp_k[below] = sk[s];
        d.smp_j[below] = sj[s];
    }
}

__global__ __launch_bounds__(kSmpTPB) void k_ss_sample(SsBatch b)
{
    __shared__ uint64_t sk[kSamples];
    __shared__ uint32_t sj[kSamples];
    if (blockIdx.y >= b.nsorts) {
        // a Priority/Weighted tile; these rows come after every sampling
        // block in dispatch order, so their look-back waits only on tiles
        // dispatched before them
        if (blockIdx.x < b.part.tiles) part_body<kSmpTPB>(b.part, blockIdx.y - b.nsorts, blockIdx.x);
        return;
    }
    if (blockIdx.x >= b.nsb) return;
    const SsDesc &d = b.s[blockIdx.y];
    switch (d.kind) {
    case SortKind::Fifo: sample_body<SortKind::Fifo>(b, d, sk, sj); break;
    case SortKind::Budget: sample_body<SortKind::Budget>(b, d, sk, sj); break;
    default: sample_body<SortKind::Aging>(b, d, sk, sj); break;
    }
}

// The pairs of this thread's kScR positions of the tile (loads first, then
// the per-request key output).
template <SortKind K>
__device__ __forceinline__ void scatter_keys(const SsBatch &b, const SsDesc &d, uint32_t base, uint32_t cnt,
                                             uint64_t *k, uint32_t *jj, uint32_t *vv)
{
    const uint32_t n = b.n;
    const int w = (int)(threadIdx.x >> 6), lane = lane_id();
    double kv[kScR];
#pragma unroll
    for (int r = 0; r < kScR; r++) {
        const uint32_t idx = (uint32_t)w * (64u * kScR) + (uint32_t)r * 64u + (uint32_t)lane;
        jj[r] = base + idx;
        vv[r] = 0;
        kv[r] = idx < cnt ? primary_key<K>(b.in, n, base + idx, vv[r]) : 0.0;
    }
#pragma unroll
    for (int r = 0; r < kScR; r++) {
        const uint32_t idx = (uint32_t)w * (64u * kScR) + (uint32_t)r * 64u + (uint32_t)lane;
        k[r] = ordered_bits(kv[r]);
        if (d.key_out && idx < cnt) d.key_out[K == SortKind::Fifo ? base + idx : vv[r]] = kv[r];
    }
}

__global__ __launch_bounds__(kScTPB) void k_ss_scatter(SsBatch b)
{
    constexpr int kWaves = kScTPB / 64;
    constexpr uint32_t kWaveKeys = 64u * kScR;
    __shared__ uint64_t s_sk[kMaxBuckets];   // [1, 2^hgt): the search tree
    __shared__ uint32_t s_sj[kMaxBuckets];
    __shared__ uint32_t wcnt[kWaves][256];
    __shared__ uint32_t texcl[256];
    __shared__ uint32_t gbase[256];
    __shared__ uint32_t tmp4[4];
    __shared__ uint64_t lkey[kScTile];
    __shared__ uint32_t lj[kScTile];
    __shared__ uint8_t lb[kScTile];

    const SsDesc &d = b.s[blockIdx.y];
    const uint32_t t = threadIdx.x, n = b.n, nsp = b.nb - 1;
    const int w = (int)(t >> 6), lane = lane_id();
    const uint32_t tile = blockIdx.x, base = tile * kScTile;
    const uint32_t cnt = n - base < kScTile ? n - base : kScTile;
    const bool digit_thread = t < 256;

    uint64_t k[kScR];
    uint32_t jj[kScR], vv[kScR], bk[kScR], rk[kScR];
    switch (d.kind) {
    case SortKind::Fifo: scatter_keys<SortKind::Fifo>(b, d, base, cnt, k, jj, vv); break;
    case SortKind::Budget: scatter_keys<SortKind::Budget>(b, d, base, cnt, k, jj, vv); break;
    default: scatter_keys<SortKind::Aging>(b, d, base, cnt, k, jj, vv); break;
    }
    // splitters in breadth-first (Eytzinger) order of a complete search tree
    // of height hgt: node e (1-based) holds the splitter of in-order index
    // (2 p + 1) 2^(hgt - d - 1) - 1 (d = depth of e, p = e - 2^d); splitter i
    // is the sample of rank floor((i + 1) S / B), and in-order indices from
    // B - 1 on are padded with the largest pair. The first levels of every
    // search then read the same few LDS words in all lanes.
    uint32_t hgt = 0;
    while ((1u << hgt) < b.nb) hgt++;
    for (uint32_t e = t + 1; e < (1u << hgt); e += kScTPB) {
        const uint32_t dpt = 31u - (uint32_t)__clz((int)e), pp = e - (1u << dpt);
        const uint32_t i = (2u * pp + 1u) * (1u << (hgt - dpt - 1u)) - 1u;
        uint64_t kk = ~0ull;
        uint32_t jv = ~0u;
        if (i < nsp) {
            const uint32_t r = (i + 1) * b.ns / b.nb;   // < ns; (i + 1) ns < 2^19
            kk = d.smp_k[r];
            jv = d.smp_j[r];
        }
        s_sk[e] = kk;
        s_sj[e] = jv;
    }
    for (uint32_t i = t; i < kWaves * 256u; i += kScTPB) (&wcnt[0][0])[i] = 0;
    __syncthreads();   // splitters and counters ready
    // bucket = number of splitters <= (key, j): hgt steps down the tree
    // (the rounds advance together, so that their LDS reads overlap)
    uint32_t node[kScR];
#pragma unroll
    for (int r = 0; r < kScR; r++) node[r] = 1;
    for (uint32_t lvl = 0; lvl < hgt; lvl++) {
        uint64_t sk_[kScR];
        uint32_t sj_[kScR];
#pragma unroll
        for (int r = 0; r < kScR; r++) {
            sk_[r] = s_sk[node[r]];
            sj_[r] = s_sj[node[r]];
        }
#pragma unroll
        for (int r = 0; r < kScR; r++)
            node[r] = 2u * node[r] + (pair_less(k[r], jj[r], sk_[r], sj_[r]) ? 0u : 1u);
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
    uint32_t *st = d.status;
    if (digit_thread) st_relaxed(&st[(uint64_t)tile * 256u + t], (tile == 0 ? kPre : kAgg) | tc);
    const uint32_t tex = block_excl_scan_digits<kScTPB>(tc, tmp4);
    if (digit_thread) {
        texcl[t] = tex;
        uint32_t prefix = 0;
        if (tile > 0) {
            prefix = look_back(st, tile, t, &d.ctl->overflow);
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
            lkey[lp] = k[r];
            lj[lp] = vv[r];
            lb[lp] = (uint8_t)dg;
        }
    }
    __syncthreads();
    bool over = false;
    for (uint32_t s = t; s < cnt; s += kScTPB) {
        const uint32_t dg = lb[s];
        const uint32_t g = gbase[dg] + s - texcl[dg];
        if (g < kCap) {
            d.bkey[(uint64_t)dg * kCap + g] = lkey[s];
            d.bj[(uint64_t)dg * kCap + g] = lj[s];
        } else {
            over = true;
        }
    }
    if (over) atomicOr(&d.ctl->overflow, 1u);
}

// Output position pos of a sort holds val; the FIFO sort can also write the
// request's tier, budget and arrival at pos (the copies in FIFO order that
// the sorts after it read instead of gathering).
__device__ __forceinline__ void emit(const SsBatch &b, const SsDesc &d, uint32_t pos, uint32_t val)
{
    d.out[pos] = val;
    if (d.kind == SortKind::Fifo) {
        const uint32_t i = val < b.n ? val : 0u;
        if (b.side.ftier) b.side.ftier[pos] = b.in.tier[i];
        if (b.side.fbudget) b.side.fbudget[pos] = b.in.budget[i];
        if (b.side.farr) b.side.farr[pos] = b.in.arrival[i];
    }
}

// LDS scratch of the bucket sort (also used by the single-workgroup sort).
struct BkShared {
    uint32_t wcnt[2][kBkTPB / 64][256];   // per-wave digit counters, two passes' worth
    uint32_t texcl[256];
    uint32_t dcnt[256];
    uint32_t offs[256];
    uint32_t tmp4[4];
    uint64_t red[kBkTPB / 64];
    uint32_t redu[kBkTPB / 64];
    uint32_t wsum[kBkTPB / 64];
    uint32_t wmax[kBkTPB / 64];
    uint64_t kmin[kBkTPB / 64], kmax[kBkTPB / 64], kmin2[kBkTPB / 64];
    uint32_t bin[kBins + 1];              // bin histogram, then bin starts
    uint64_t lkey[kCap];
    uint32_t lj[kCap];
    uint16_t lslot[kCap];
};

// One stable LSD pass on byte p of the keys of m pairs held R_eff per thread
// (wave-major positions w * 64 R_eff + r * 64 + lane): returns each pair's
// place in the pass order through pos, leaves the digits' exclusive starts in
// sh.texcl and, for thread t < 256, digit t's count in tc. Counters buffer
// `cur` must be zero on entry; buffer cur ^ 1 is cleared for the next pass.
// Ends with a barrier; the caller's reads of pos-ordered data need another.
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

// The whole sequence sorted by one workgroup: LSD passes over global
// ping-pong buffers, in chunks of kCap pairs taken in order.
__device__ void serial_sort(const SsBatch &b, const SsDesc &d, BkShared &sh)
{
    const uint32_t n = b.n, t = threadIdx.x;
    const int w = (int)(t >> 6), lane = lane_id();
    for (uint32_t i = t; i < 2u * (kBkTPB / 64) * 256u; i += kBkTPB) (&sh.wcnt[0][0][0])[i] = 0;
    uint32_t cur = 0;
    for (uint32_t j = t; j < n; j += kBkTPB) {
        uint64_t k;
        uint32_t v;
        produce(b.in, d.kind, nullptr, n, j, k, v);
        d.fkey[0][j] = k;
        d.fj[0][j] = j;
    }
    __syncthreads();
    uint32_t src = 0;
    for (uint32_t p = 0; p < 8; p++) {
        // digit histogram; a pass whose digit is the same for all keys is skipped
        if (t < 256) sh.offs[t] = 0;
        __syncthreads();
        for (uint32_t j = t; j < n; j += kBkTPB)
            atomicAdd(&sh.offs[(uint32_t)(d.fkey[src][j] >> (8 * p)) & 255u], 1u);
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
            uint32_t jv[kBkR], pos[kBkR];
#pragma unroll
            for (int r = 0; r < kBkR; r++) {
                const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
                k[r] = 0;
                jv[r] = 0;
                if ((uint32_t)r < reff && idx < m) {
                    k[r] = d.fkey[src][c0 + idx];
                    jv[r] = d.fj[src][c0 + idx];
                }
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
                    d.fkey[src ^ 1u][g] = k[r];
                    d.fj[src ^ 1u][g] = jv[r];
                }
            }
            __syncthreads();
            if (t < 256) sh.offs[t] += tc;
            __syncthreads();
        }
        src ^= 1u;
    }
    for (uint32_t i = t; i < n; i += kBkTPB) emit(b, d, i, value_of(b.in, d.kind, n, d.fj[src][i]));
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
    for (uint32_t i = t; i < 2u * kWaves * 256u; i += kBkTPB) (&sh.wcnt[0][0][0])[i] = 0;
    const uint64_t *src_k = d.bkey + (uint64_t)bkt * kCap;
    const uint32_t *src_j = d.bj + (uint64_t)bkt * kCap;
    // the first kBkTPB slots are loaded before the size is known (a bucket
    // of at most kBkTPB pairs, the common case, needs no other load)
    const uint64_t k0 = src_k[t];
    const uint32_t j0 = src_j[t];
    // bucket sizes: the last tile's inclusive prefixes
    const uint32_t *last = d.status + (uint64_t)(b.tiles - 1) * 256u;
    const uint32_t c = t < b.nb ? (last[t] & kValMask) : 0u;
    uint32_t before = wave_sum(t < bkt ? c : 0u);
    if (lane == 0) sh.redu[w] = before;
    if (t == bkt) sh.offs[0] = c;
    __syncthreads();
    uint32_t off = 0;
#pragma unroll
    for (int q = 0; q < kWaves; q++) off += sh.redu[q];
    const uint32_t m = sh.offs[0];   // <= kCap: no region overflowed
    const uint32_t reff = (m + kBkTPB - 1) / kBkTPB;
    const uint32_t wk = 64u * reff;

    uint64_t k[kBkR];
    uint32_t jv[kBkR], pos[kBkR];
    uint64_t kmn = ~0ull, kmx = 0;
#pragma unroll
    for (int r = 0; r < kBkR; r++) {
        const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
        k[r] = 0;
        jv[r] = 0;
        if ((uint32_t)r < reff && idx < m) {
            if (reff == 1) {
                k[r] = k0;
                jv[r] = j0;
            } else {
                k[r] = src_k[idx];
                jv[r] = src_j[idx];
            }
            kmn = k[r] < kmn ? k[r] : kmn;
            kmx = k[r] > kmx ? k[r] : kmx;
        }
    }
    // key range of the bucket
#pragma unroll
    for (int sft = 32; sft >= 1; sft >>= 1) {
        const uint64_t a = shfl_xor_u64(kmn, sft), c2 = shfl_xor_u64(kmx, sft);
        kmn = a < kmn ? a : kmn;
        kmx = c2 > kmx ? c2 : kmx;
    }
    if (lane == 0) {
        sh.kmin[w] = kmn;
        sh.kmax[w] = kmx;
    }
    for (uint32_t i = t; i <= kBins; i += kBkTPB) sh.bin[i] = 0;
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kWaves; q++) {
        kmn = sh.kmin[q] < kmn ? sh.kmin[q] : kmn;
        kmx = sh.kmax[q] > kmx ? sh.kmax[q] : kmx;
    }
    if (kmn >= kmx) {
        // one key (or an empty bucket): position order is the order
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            if ((uint32_t)r < reff && idx < m && off + idx < n) emit(b, d, off + idx, jv[r]);
        }
        return;
    }
    // Pairs with the bucket's smallest key (the common heavy tie: aged
    // scores clamped to the floor) come first, in position order: their rank
    // is the number of such pairs at lower slots, from ballots. The others
    // go to bins, monotone in the key, over the range [x2, xmax] of the keys
    // above the minimum: for a finite range, kBins equal intervals
    // ((x - x2) * (kBins / (xmax - x2)), each step rounded, so monotone);
    // otherwise the kBinBits bits of key - key2 below its highest varying
    // bit. Their rank = pairs at the minimum + bin start + rank inside the
    // bin by (key, slot), the slot being the position order.
    uint32_t lowrank[kBkR], hirank[kBkR];
    uint32_t nlow;
    uint64_t kmn2 = ~0ull;   // smallest key above the minimum
    {
        uint32_t run = 0, runh = 0;
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            const bool valid = (uint32_t)r < reff && idx < m;
            const bool low = valid && k[r] == kmn;
            const uint64_t bl = __ballot(low), bh = __ballot(valid && !low);
            lowrank[r] = run + (uint32_t)__popcll(bl & lanemask_lt());
            hirank[r] = runh + (uint32_t)__popcll(bh & lanemask_lt());
            run += (uint32_t)__popcll(bl);
            runh += (uint32_t)__popcll(bh);
            if (valid && !low && k[r] < kmn2) kmn2 = k[r];
        }
#pragma unroll
        for (int sft = 32; sft >= 1; sft >>= 1) {
            const uint64_t a = shfl_xor_u64(kmn2, sft);
            kmn2 = a < kmn2 ? a : kmn2;
        }
        if (lane == 0) {
            sh.wsum[w] = run;
            sh.wmax[w] = runh;
            sh.kmin2[w] = kmn2;
        }
        __syncthreads();
        uint32_t before_w = 0, before_h = 0;
        nlow = 0;
#pragma unroll
        for (int q = 0; q < kWaves; q++) {
            before_w += q < w ? sh.wsum[q] : 0u;
            before_h += q < w ? sh.wmax[q] : 0u;
            nlow += sh.wsum[q];
            kmn2 = sh.kmin2[q] < kmn2 ? sh.kmin2[q] : kmn2;
        }
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            lowrank[r] += before_w;
            hirank[r] += before_h;
        }
        __syncthreads();   // sh.wsum, sh.wmax are reused by the bin scan
    }
    if (kmn2 >= kmx) {
        // two distinct keys: each in position order
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            if ((uint32_t)r < reff && idx < m) {
                const uint32_t rank = k[r] == kmn ? lowrank[r] : nlow + hirank[r];
                if (off + rank < n) emit(b, d, off + rank, jv[r]);
            }
        }
        return;
    }
    // bins over [kmn2, kmx] for the pairs above the minimum
    const int hb = 63 - __clzll((long long)(kmn2 ^ kmx));
    const uint32_t shift = hb >= (int)kBinBits ? (uint32_t)hb - (kBinBits - 1u) : 0u;
    const double xmn = from_ordered(kmn2), xmx = from_ordered(kmx);
    const double span = xmx - xmn;
    const bool linear = isfinite(span) && span > 0.0 && isfinite((double)kBins / span);
    const double scale = linear ? (double)kBins / span : 0.0;
    uint32_t dg[kBkR], bs[kBkR];
#pragma unroll
    for (int r = 0; r < kBkR; r++) {
        const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
        dg[r] = 0;
        bs[r] = 0;
        if ((uint32_t)r < reff && idx < m && k[r] != kmn) {
            if (linear) {
                const double f = (from_ordered(k[r]) - xmn) * scale;   // in [0, kBins]
                const uint32_t q = f < (double)kBins ? (uint32_t)f : kBins - 1u;
                dg[r] = q;
            } else {
                dg[r] = (uint32_t)((k[r] - kmn2) >> shift);   // < kBins
            }
            bs[r] = atomicAdd(&sh.bin[dg[r]], 1u);
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
    if (maxbin <= kBinMax) {
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            if ((uint32_t)r < reff && idx < m && k[r] != kmn) {
                const uint32_t q = sh.bin[dg[r]] + bs[r];
                sh.lkey[q] = k[r];
                sh.lslot[q] = (uint16_t)idx;
            }
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            if ((uint32_t)r < reff && idx < m) {
                uint32_t rank = lowrank[r];
                if (k[r] != kmn) {
                    const uint32_t s0 = sh.bin[dg[r]], s1 = sh.bin[dg[r] + 1];
                    rank = nlow + s0;
                    for (uint32_t u = s0; u < s1; u++) {
                        const uint64_t ku = sh.lkey[u];
                        rank += (ku < k[r] || (ku == k[r] && sh.lslot[u] < idx)) ? 1u : 0u;
                    }
                }
                if (off + rank < n) emit(b, d, off + rank, jv[r]);
            }
        }
        return;
    }
    // crowded bins (many equal or near-equal keys): stable LSD passes over
    // all the pairs, on the key bytes up to the highest bit that varies in
    // the bucket (minimum included)
    const int hba = 63 - __clzll((long long)(kmn ^ kmx));
    const uint64_t diff = hba == 63 ? ~0ull : ((1ull << (hba + 1)) - 1ull);
    uint32_t cur = 0;
    for (uint32_t p = 0; p < 8; p++) {
        if (((diff >> (8 * p)) & 255u) == 0) continue;   // uniform
        uint32_t tc;
        lds_rank(sh, cur, k, reff, m, p, pos, tc);
        cur ^= 1u;
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            if ((uint32_t)r < reff && idx < m) {
                sh.lkey[pos[r]] = k[r];
                sh.lj[pos[r]] = jv[r];
            }
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < kBkR; r++) {
            const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
            if ((uint32_t)r < reff && idx < m) {
                k[r] = sh.lkey[idx];
                jv[r] = sh.lj[idx];
            }
        }
    }
#pragma unroll
    for (int r = 0; r < kBkR; r++) {
        const uint32_t idx = (uint32_t)w * wk + (uint32_t)r * 64u + (uint32_t)lane;
        if ((uint32_t)r < reff && idx < m && off + idx < n) emit(b, d, off + idx, jv[r]);
    }
}

uint32_t n_buckets(uint64_t n)
{
    const uint64_t b = cdiv(n, kBucketAvg);
    return (uint32_t)(b < 1 ? 1 : (b > kMaxBuckets ? kMaxBuckets : b));
}

uint64_t region_bytes(uint64_t n)
{
    const uint64_t tiles = cdiv(n, kScTile);
    const uint64_t nb = n_buckets(n);
    return align_up(sizeof(SsCtl), 256) + align_up(kSamples * 8, 256) + align_up(kSamples * 4, 256) +
           align_up(tiles * 256 * 4, 256) + align_up(nb * kCap * 8, 256) + align_up(nb * kCap * 4, 256) +
           2 * align_up(n * 8, 256) + 2 * align_up(n * 4, 256);
}

void carve(uint8_t *p, uint64_t n, SsDesc &d)
{
    const uint64_t tiles = cdiv(n, kScTile);
    const uint64_t nb = n_buckets(n);
    auto take = [&](uint64_t bytes) {
        uint8_t *q = p;
        p += align_up(bytes, 256);
        return q;
    };
    d.ctl = reinterpret_cast<SsCtl *>(take(sizeof(SsCtl)));
    d.smp_k = reinterpret_cast<uint64_t *>(take(kSamples * 8));
    d.smp_j = reinterpret_cast<uint32_t *>(take(kSamples * 4));
    d.status = reinterpret_cast<uint32_t *>(take(tiles * 256 * 4));
    d.bkey = reinterpret_cast<uint64_t *>(take(nb * kCap * 8));
    d.bj = reinterpret_cast<uint32_t *>(take(nb * kCap * 4));
    for (int i = 0; i < 2; i++) d.fkey[i] = reinterpret_cast<uint64_t *>(take(n * 8));
    for (int i = 0; i < 2; i++) d.fj[i] = reinterpret_cast<uint32_t *>(take(n * 4));
}

}  // namespace

size_t ssort_ws_bytes(uint64_t n, uint32_t nsorts)
{
    return n <= kSsMaxN ? (size_t)nsorts * region_bytes(n) : 0;
}

uint32_t ssort_sample_blocks(uint64_t n)
{
    const uint64_t smax = n <= (1u << 17) ? kSamples / 2 : kSamples;
    const uint64_t ns = n < smax ? n : smax;
    return (uint32_t)cdiv(ns ? ns : 1, kSmpPerBlock);
}

hipError_t ssort_launch(const SortInput &in, const SortJob *jobs, uint32_t nsorts, bool serial,
                        void *ws, hipStream_t s, const SsSide *side, const PartBatch *part)
{
    if (in.n == 0 || nsorts == 0) return hipSuccess;
    if (nsorts > kMaxSorts || in.n > kSsMaxN) return hipErrorInvalidValue;
    SsBatch b;
    b.in = in;
    b.n = in.n;
    b.tiles = (uint32_t)cdiv(in.n, kScTile);
    b.nb = n_buckets(in.n);
    // 1024 samples (4 per bucket) up to 2^17 keys, 2048 above, where the
    // average bucket is a quarter of the region capacity
    const uint32_t smax = in.n <= (1u << 17) ? kSamples / 2 : kSamples;
    b.ns = in.n < smax ? in.n : smax;
    b.serial = serial ? 1u : 0u;
    b.side = side ? *side : SsSide{nullptr, 0u, nullptr, nullptr, nullptr, nullptr};
    b.nsorts = nsorts;
    b.nsb = ssort_sample_blocks(in.n);
    if (part) {
        b.part = *part;
    } else {
        memset(&b.part, 0, sizeof(b.part));
    }
    uint8_t *p = static_cast<uint8_t *>(ws);
    for (uint32_t i = 0; i < nsorts; i++) {
        SsDesc &d = b.s[i];
        if (jobs[i].kind != SortKind::Fifo && jobs[i].kind != SortKind::Budget &&
            jobs[i].kind != SortKind::Aging)
            return hipErrorInvalidValue;
        d.kind = jobs[i].kind;
        d.key_out = jobs[i].key_out;
        d.out = jobs[i].out;
        carve(p, in.n, d);
        p += region_bytes(in.n);
    }
    const uint32_t gx = b.part.njobs && b.part.tiles > b.nsb ? b.part.tiles : b.nsb;
    hipLaunchKernelGGL(k_ss_sample, dim3(gx, nsorts + b.part.njobs), dim3(kSmpTPB), 0, s, b);
    hipLaunchKernelGGL(k_ss_scatter, dim3(b.tiles, nsorts), dim3(kScTPB), 0, s, b);
    hipLaunchKernelGGL(k_ss_bucket, dim3(b.nb, nsorts), dim3(kBkTPB), 0, s, b);
    return hipGetLastError();
}

}  // namespace ds
