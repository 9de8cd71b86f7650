// Stable LSD radix sorts of (key, value) pairs, 8-bit digits, one kernel per
// digit pass, with decoupled look-back between tiles. Several independent
// sorts of the same length run in the same launches (grid.y = sort).
//
// Used for: the FIFO rank (key = arrival), SJF and Aging (key = budget or
// aged score over the FIFO sequence, so that ties keep FIFO order), the
// one-pass partitions of Priority (priority class) and Weighted (tier, then
// the round-robin position: a closed form for the blocked and stride
// interleavings, the period table built by k_sort_plan for the smooth one),
// and the group partition of the calibration scan.
//
// Launches of one batch of sorts:
//   k_sort_init  produces the pairs from the inputs, writes each block's digit
//                histograms of every pass (no atomics), clears the
//                look-back words of the passes
//   k_sort_plan  one block per (pass, sort): sums the block histograms into
//                exclusive digit offsets and marks a pass whose digit is the
//                same for every key (it is skipped)
//   k_sort_pass  one per digit pass: per tile of TPB*R keys, wave ranking by
//                ballots over the digit bits, per-wave LDS counters,
//                look-back over earlier tiles' per-digit counts (windows of
//                16 predecessors loaded at once, bounded wait), reorder
//                through LDS, coalesced runs of global writes. The buffer a
//                pass reads, and whether it is the last active pass, follow
//                from the active flags.
// Tile t of a pass is block t, and it waits only on tiles with a smaller
// index. Blocks of a dispatch are handed out in index order on each XCD, so
// the unfinished tile of smallest index has been started (every earlier
// block of its XCD has finished and freed its slot) and waits on nobody: the
// passes always make progress. The wait is bounded all the same; a wait that
// runs out is reported in the caller's status word (WaitCfg).
#include "common.h"
#include "kernels.h"
#include "keys.h"
#include "lookback.h"
#include "wrrplan.h"

namespace ds {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxPasses = 8;
constexpr uint32_t kInitBlocks = 256;     // block histograms per sort (at most)

struct SortCtl {
    uint32_t excl[kMaxPasses][256];
    uint32_t active[kMaxPasses];
    uint32_t error;
    uint32_t pad[15];
};

struct SortDesc {
    SortKind kind;
    uint32_t passes;
    double *key_out;
    uint32_t *out;
    SortCtl *ctl;
    uint32_t *bhist;       // [init blocks][passes][256]
    uint64_t *key[2];
    uint32_t *val[2];
    uint32_t *status;      // [passes][tiles][256]
    WrrPlan *plan;         // Tier, smooth round robin: the period table (built by k_sort_plan)
    uint32_t *tpos;        // its start-up positions (val[1]: a one-pass sort leaves it unused)
};

struct SortBatch {
    SortInput in;          // shared inputs and parameters
    uint32_t n;
    uint32_t tiles;
    uint32_t nsorts;
    uint32_t init_blocks;
    SortDesc s[kMaxSorts];
};

__host__ __device__ inline uint32_t n_passes(uint32_t key_bits)
{
    uint32_t p = (key_bits + 7) / 8;
    return p == 0 ? 1 : (p > kMaxPasses ? kMaxPasses : p);
}

constexpr int kInitPer = 4;        // keys per thread per step of the init kernel
constexpr int kPlanTPB = 1024;     // threads per plan block: four per digit

// TPB: 1024 threads for batches of one or two sorts, 512 for more, so that
// the init blocks of a batch (at most kInitBlocks per sort) are resident at
// once.
template <int TPB>
__global__ __launch_bounds__(TPB) void k_sort_init(SortBatch b, uint64_t status_words)
{
    __shared__ uint32_t h[kMaxPasses][256];
    const SortDesc &d = b.s[blockIdx.y];
    const uint32_t P = d.passes;
    const uint32_t n = b.n;
    // clear this sort's look-back words (used by the passes)
    {
        uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
        uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
        if (t == 0) d.ctl->error = 0;
        if (t == 0 && blockIdx.y == 0 && b.in.wait.clear && b.in.wait.status) *b.in.wait.status = 0;
        uint64_t words = (uint64_t)P * status_words;
        for (uint64_t i = t; i < words; i += stride) d.status[i] = 0;
    }
    for (uint32_t i = threadIdx.x; i < P * 256; i += blockDim.x) (&h[0][0])[i] = 0;
    __syncthreads();
    const uint32_t step = gridDim.x * blockDim.x * kInitPer;
    for (uint32_t j0 = blockIdx.x * blockDim.x * kInitPer; j0 < n; j0 += step) {
        uint64_t k[kInitPer];
        uint32_t v[kInitPer];
        bool ok[kInitPer];
#pragma unroll
        for (int r = 0; r < kInitPer; r++) {
            uint32_t j = j0 + (uint32_t)r * blockDim.x + threadIdx.x;
            ok[r] = j < n;
            k[r] = 0;
            v[r] = 0;
            if (ok[r]) produce(b.in, d.kind, d.key_out, n, j, k[r], v[r]);
        }
#pragma unroll
        for (int r = 0; r < kInitPer; r++) {
            uint32_t j = j0 + (uint32_t)r * blockDim.x + threadIdx.x;
            if (ok[r]) {
                d.key[0][j] = k[r];
                d.val[0][j] = v[r];
            }
            const uint64_t act = __ballot(ok[r]);
            for (uint32_t p = 0; p < P; p++) {
                uint32_t dg = (uint32_t)(k[r] >> (8 * p)) & 255u;
                // a digit shared by the whole wave (the common case for high
                // digits) is counted with one atomic
                uint32_t d0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)dg);
                if (__ballot(ok[r] && dg != d0) == 0) {
                    if (lane_id() == 0 && act) atomicAdd(&h[p][d0], (uint32_t)__popcll(act));
                } else if (ok[r]) {
                    atomicAdd(&h[p][dg], 1u);
                }
            }
        }
    }
    __syncthreads();
    uint32_t *bh = d.bhist + (uint64_t)blockIdx.x * P * 256u;
    for (uint32_t i = threadIdx.x; i < P * 256; i += blockDim.x) bh[i] = (&h[0][0])[i];
}

// One block per (pass, sort): digit totals from the block histograms,
// exclusive offsets, and whether the pass does anything. Four threads per
// digit each add up every fourth block histogram, 32 loads in flight at a
// time.
__global__ __launch_bounds__(kPlanTPB) void k_sort_plan(SortBatch b)
{
    constexpr uint32_t kParts = kPlanTPB / 256, kBatch = 32;
    __shared__ uint32_t part[kParts][256];
    __shared__ uint32_t tmp4[4];
    const SortDesc &d = b.s[blockIdx.y];
    const uint32_t p = blockIdx.x;
    if (p >= d.passes) return;
    const uint32_t t = threadIdx.x, dig = t & 255u, q = t >> 8;
    const uint32_t stride = d.passes * 256u;
    uint32_t c = 0;
    for (uint32_t i0 = 0; i0 * kParts < b.init_blocks; i0 += kBatch) {
        uint32_t x[kBatch];
#pragma unroll
        for (uint32_t k = 0; k < kBatch; k++) {
            const uint32_t blk = q + kParts * (i0 + k);
            x[k] = blk < b.init_blocks ? d.bhist[(uint64_t)blk * stride + p * 256u + dig] : 0u;
        }
#pragma unroll
        for (uint32_t k = 0; k < kBatch; k++) c += x[k];
    }
    part[q][dig] = c;
    __syncthreads();
    c = 0;
    if (t < 256) {
#pragma unroll
        for (uint32_t k = 0; k < kParts; k++) c += part[k][t];
    }
    const int full = __syncthreads_or(t < 256 && c == b.n ? 1 : 0);
    // exclusive scan of the 256 digit totals (waves 0..3)
    uint32_t incl = 0;
    if (t < 256) {
        incl = wave_incl_scan_dpp(c);
        if (lane_id() == 63) tmp4[t >> 6] = incl;
    }
    __syncthreads();
    if (t < 256) {
        uint32_t off = 0;
        for (uint32_t k = 0; k < (t >> 6); k++) off += tmp4[k];
        d.ctl->excl[p][t] = off + incl - c;
    }
    if (t == 0) d.ctl->active[p] = full ? 0u : 1u;
    if (d.kind == SortKind::Tier && b.in.wrr_mode == kWrrSmooth && t < 64) {
        // the smooth interleaving's period table (digit t = tier t)
        __shared__ uint16_t per[kWrrMaxWeightSum];
        const uint32_t nq = b.in.n_tiers < kWrrTiers ? b.in.n_tiers : kWrrTiers;
        const bool tl = t < nq;
        wrr_plan_build(tl ? c : 0u, tl ? b.in.weight[t] : 0u, per, d.plan, d.tpos);
    }
}

// Weighted round robin position of the k-th (FIFO) request of tier q:
// rounds before r = floor(k / w_q) dispatch sum_q' min(n_q', r w_q'); in
// round r the tiers before q dispatch min(w_q', max(0, n_q' - r w_q')).
__device__ __forceinline__ uint64_t wrr_pos(const SortInput &in, const uint32_t *tstart, uint32_t n,
                                            uint32_t q, uint64_t k, uint64_t &round)
{
    uint64_t wq = in.weight[q] ? in.weight[q] : 1;
    uint64_t r = k / wq;
    uint64_t pos = k - r * wq;
    for (uint32_t t = 0; t < in.n_tiers; t++) {
        // requests of tier t: start of the next tier's range minus its own
        uint64_t nt = (uint64_t)tstart[t + 1] - tstart[t], wt = in.weight[t];
        uint64_t full = r * wt;
        pos += nt < full ? nt : full;
        if (t < q) {
            uint64_t left = nt > full ? nt - full : 0;
            pos += left < wt ? left : wt;
        }
    }
    round = r;
    return pos;
}

// One digit pass over tiles of TPB * R keys (tile t = block t).
template <int TPB, int R>
__global__ __launch_bounds__(TPB) void k_sort_pass(SortBatch b, uint32_t p)
{
    constexpr uint32_t kTile = TPB * R;
    constexpr int kWaves = TPB / 64;
    constexpr uint32_t kWaveKeys = 64u * R;
    __shared__ uint32_t wcnt[kWaves][256];
    __shared__ uint32_t texcl[256];
    __shared__ uint32_t gbase[256];
    __shared__ uint32_t tmp4[4];
    __shared__ uint64_t lkey[kTile];
    __shared__ uint32_t lval[kTile];

    const SortDesc &d = b.s[blockIdx.y];
    if (p >= d.passes) return;
    SortCtl *ctl = d.ctl;
    const uint32_t n = b.n;
    const uint32_t t = threadIdx.x;
    const bool digit_thread = t < 256;
    // plan words: the pass reads the buffer written by the last active pass
    // before it, and writes the output if no later pass is active
    uint32_t act[kMaxPasses];
#pragma unroll
    for (uint32_t q = 0; q < kMaxPasses; q++) act[q] = q < d.passes ? ctl->active[q] : 0u;
    const uint32_t dexcl = digit_thread ? ctl->excl[p][t] : 0u;
    const uint32_t active = act[p];
    uint32_t before = 0, after = 0;
#pragma unroll
    for (uint32_t q = 0; q < kMaxPasses; q++) {
        if (q < p) before += act[q];
        if (q > p) after += act[q];
    }
    const uint32_t srcb = before & 1u;
    if (!active) {
        // a pass whose digit is constant is skipped; if no pass is active
        // the input order is the result (the last pass copies it out)
        if (p + 1 == d.passes && before == 0) {
            for (uint32_t j = blockIdx.x * blockDim.x + threadIdx.x; j < n; j += gridDim.x * blockDim.x) {
                uint32_t val = d.val[0][j];
                d.out[j] = val;
                if (d.kind == SortKind::Tier && d.key_out && val < n) {
                    // one non-empty tier: the k-th request is served in round k / w
                    uint32_t q = (uint32_t)d.key[0][j] & 15u;
                    uint32_t wq = b.in.weight[q] ? b.in.weight[q] : 1u;
                    d.key_out[val] = (double)(j / wq);
                }
            }
        }
        return;
    }
    const int w = (int)(t >> 6);
    const int lane = lane_id();
    for (uint32_t i = t; i < kWaves * 256u; i += TPB) (&wcnt[0][0])[i] = 0;
    const uint32_t tile = blockIdx.x;
    const uint32_t base = tile * kTile;
    const uint32_t cnt = n - base < kTile ? n - base : kTile;
    const uint32_t shift = 8 * p;
    const uint64_t *ik = d.key[srcb];
    const uint32_t *iv = d.val[srcb];
    const bool last = after == 0;

    uint64_t k[R];
    uint32_t v[R];
    uint32_t rk[R];
#pragma unroll
    for (int r = 0; r < R; r++) {
        uint32_t idx = (uint32_t)w * kWaveKeys + (uint32_t)r * 64u + (uint32_t)lane;
        bool ok = idx < cnt;
        k[r] = ok ? ik[base + idx] : 0ull;
        v[r] = ok ? iv[base + idx] : 0u;
    }
    __syncthreads();
    // stable rank within the wave, round by round (rounds are in index order)
#pragma unroll
    for (int r = 0; r < R; r++) {
        uint32_t idx = (uint32_t)w * kWaveKeys + (uint32_t)r * 64u + (uint32_t)lane;
        bool ok = idx < cnt;
        uint32_t dg = (uint32_t)(k[r] >> shift) & 255u;
        uint64_t peers = __ballot(ok);
#pragma unroll
        for (int bb = 0; bb < 8; bb++) {
            bool bit = (dg >> bb) & 1u;
            uint64_t m = __ballot(bit);
            peers &= bit ? m : ~m;
        }
        uint32_t below = (uint32_t)__popcll(peers & lanemask_lt());
        uint32_t old = ok ? wcnt[w][dg] : 0u;
        rk[r] = old + below;
        if (ok && below == 0) wcnt[w][dg] = old + (uint32_t)__popcll(peers);
        __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();
    // per digit (thread t = digit): tile count, per-wave exclusive offsets
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
    // publish this tile's count first, then scan and look back
    uint32_t *st = d.status + (uint64_t)p * b.tiles * 256u;
    if (digit_thread) st_relaxed(&st[(uint64_t)tile * 256u + t], (tile == 0 ? kPre : kAgg) | tc);
    const uint32_t tex = block_excl_scan_digits<TPB>(tc, tmp4);
    if (digit_thread) {
        texcl[t] = tex;
        uint32_t prefix = 0;
        if (tile > 0) {
            prefix = look_back(st, tile, t, b.in.wait.status ? b.in.wait.status : &ctl->error,
                               b.in.wait.no_wait ? 0u : kSpinLimit);
            st_relaxed(&st[(uint64_t)tile * 256u + t], kPre | (prefix + tc));
        }
        gbase[t] = dexcl + prefix;
    }
    __syncthreads();
    // reorder the tile through LDS by digit
#pragma unroll
    for (int r = 0; r < R; r++) {
        uint32_t idx = (uint32_t)w * kWaveKeys + (uint32_t)r * 64u + (uint32_t)lane;
        if (idx < cnt) {
            uint32_t dg = (uint32_t)(k[r] >> shift) & 255u;
            uint32_t lp = texcl[dg] + wcnt[w][dg] + rk[r];
            lkey[lp] = k[r];
            lval[lp] = v[r];
        }
    }
    __syncthreads();
    if (d.kind == SortKind::Tier) {
        // single pass: digit = tier; scatter to the weighted position
        const uint32_t *tstart = ctl->excl[0];
        WrrPlanHead &wh = *reinterpret_cast<WrrPlanHead *>(&wcnt[0][0]);   // the counters are done
        static_assert(sizeof(WrrPlanHead) <= sizeof(wcnt), "plan header fits the counters");
        const bool smooth = b.in.wrr_mode == kWrrSmooth;
        if (smooth) {
            __syncthreads();
            for (uint32_t i = t; i < sizeof(WrrPlanHead) / 4; i += TPB)
                reinterpret_cast<uint32_t *>(&wh)[i] = reinterpret_cast<const uint32_t *>(&d.plan->h)[i];
            __syncthreads();
        }
        for (uint32_t s = t; s < cnt; s += TPB) {
            uint32_t q = (uint32_t)lkey[s] & 255u;
            uint32_t g = gbase[q] + s - texcl[q];
            uint64_t kq = g - ctl->excl[0][q];
            uint64_t rnd;
            uint64_t pos;
            if (smooth) {
                uint32_t r32;
                pos = wrr_smooth_pos(wh, d.plan, d.tpos, b.in.weight[q & 15u], q & 15u, (uint32_t)kq, r32);
                rnd = r32;
            } else if (b.in.wrr_mode == kWrrStride) {
                const uint32_t qc = q & 15u, wq = b.in.weight[qc] ? b.in.weight[qc] : 1u;
                rnd = kq / wq;
                pos = wrr_stride_pos(qc, kq, b.in.weight, b.in.n_tiers < 16u ? b.in.n_tiers : 16u,
                                     [&](uint32_t u) { return tstart[u + 1] - tstart[u]; });
            } else {
                pos = wrr_pos(b.in, tstart, n, q, kq, rnd);
            }
            uint32_t val = lval[s];
            if (pos < n) d.out[pos] = val;   // always true when tiers are < n_tiers
            if (d.key_out && val < n) d.key_out[val] = (double)rnd;
        }
        return;
    }
    uint64_t *okey = d.key[srcb ^ 1u];
    uint32_t *ov = last ? d.out : d.val[srcb ^ 1u];
    for (uint32_t s = t; s < cnt; s += TPB) {
        uint64_t kk = lkey[s];
        uint32_t dg = (uint32_t)(kk >> shift) & 255u;
        uint32_t g = gbase[dg] + s - texcl[dg];
        ov[g] = lval[s];
        if (!last) okey[g] = kk;
    }
}

// Tile shapes: 2048 keys (512 threads x 4) up to 2^18 keys, 4096 keys (512
// threads x 8) above: larger tiles shorten the look-back, and at 2^20 keys
// 4096-key tiles still give every CU a tile of each sort (8192-key tiles
// left half of them idle).
constexpr uint32_t kSmallN = 1u << 18;
uint32_t tile_keys(uint64_t n) { return n <= kSmallN ? 512u * 4u : 512u * 8u; }

uint64_t region_bytes(uint64_t n)
{
    uint64_t tiles = cdiv(n, tile_keys(n));
    return align_up(sizeof(SortCtl), 256) + align_up((uint64_t)kInitBlocks * kMaxPasses * 256 * 4, 256) +
           2 * align_up(n * 8, 256) + 2 * align_up(n * 4, 256) +
           align_up((uint64_t)kMaxPasses * tiles * 256 * 4, 256) + align_up(sizeof(WrrPlan), 256);
}

void carve(uint8_t *p, uint64_t n, SortDesc &d)
{
    d.ctl = reinterpret_cast<SortCtl *>(p);
    p += align_up(sizeof(SortCtl), 256);
    d.bhist = reinterpret_cast<uint32_t *>(p);
    p += align_up((uint64_t)kInitBlocks * kMaxPasses * 256 * 4, 256);
    for (int i = 0; i < 2; i++) {
        d.key[i] = reinterpret_cast<uint64_t *>(p);
        p += align_up(n * 8, 256);
    }
    for (int i = 0; i < 2; i++) {
        d.val[i] = reinterpret_cast<uint32_t *>(p);
        p += align_up(n * 4, 256);
    }
    d.status = reinterpret_cast<uint32_t *>(p);
    p += align_up((uint64_t)kMaxPasses * cdiv(n, tile_keys(n)) * 256 * 4, 256);
    d.plan = reinterpret_cast<WrrPlan *>(p);
    d.tpos = d.val[1];
}

}  // namespace

size_t sort_ws_bytes(uint64_t n, uint32_t nsorts)
{
    return (size_t)nsorts * region_bytes(n);
}

hipError_t sort_launch(const SortInput &in, const SortJob *jobs, uint32_t nsorts, void *ws,
                       hipStream_t s)
{
    if (in.n == 0 || nsorts == 0) return hipSuccess;
    if (nsorts > kMaxSorts) return hipErrorInvalidValue;
    SortBatch b;
    b.in = in;
    b.n = in.n;
    const uint32_t tk = tile_keys(in.n);
    b.tiles = (uint32_t)cdiv(in.n, tk);
    b.nsorts = nsorts;
    uint32_t maxp = 0;
    uint8_t *p = static_cast<uint8_t *>(ws);
    for (uint32_t i = 0; i < nsorts; i++) {
        SortDesc &d = b.s[i];
        d.kind = jobs[i].kind;
        d.passes = n_passes(jobs[i].key_bits);
        d.key_out = jobs[i].key_out;
        d.out = jobs[i].out;
        carve(p, in.n, d);
        p += region_bytes(in.n);
        maxp = d.passes > maxp ? d.passes : maxp;
    }
    const uint64_t status_words = (uint64_t)b.tiles * 256u;
    const bool wide = nsorts <= 2;
    const uint32_t itpb = wide ? 1024u : 512u;
    uint64_t ibw = cdiv(in.n, (uint64_t)itpb * kInitPer);
    b.init_blocks = (uint32_t)(ibw < kInitBlocks ? (ibw ? ibw : 1) : kInitBlocks);
    if (wide)
        hipLaunchKernelGGL(k_sort_init<1024>, dim3(b.init_blocks, nsorts), dim3(1024), 0, s, b, status_words);
    else
        hipLaunchKernelGGL(k_sort_init<512>, dim3(b.init_blocks, nsorts), dim3(512), 0, s, b, status_words);
    hipLaunchKernelGGL(k_sort_plan, dim3(maxp, nsorts), dim3(kPlanTPB), 0, s, b);
    for (uint32_t pass = 0; pass < maxp; pass++) {
        if (in.n <= kSmallN)
            hipLaunchKernelGGL((k_sort_pass<512, 4>), dim3(b.tiles, nsorts), dim3(512), 0, s, b, pass);
        else
            hipLaunchKernelGGL((k_sort_pass<512, 8>), dim3(b.tiles, nsorts), dim3(512), 0, s, b, pass);
    }
    return hipGetLastError();
}

}  // namespace ds
