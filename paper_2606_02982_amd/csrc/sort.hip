// Stable LSD radix sort of (key, value) pairs, 8-bit digits, one kernel per
// digit pass with decoupled look-back between tiles.
//
// Used for: the FIFO rank (key = arrival), SJF and Aging (key = budget or
// aged score, sorting the FIFO sequence so that ties keep FIFO order), the
// tier partitions of Priority and Weighted (one pass), and the group
// partition of the calibration scan.
//
// Kernels of one sort:
//   k_sort_zero  clears the digit histograms, tile tickets and look-back words
//   k_sort_init  produces the pairs from the inputs, counts all passes' digits
//   k_sort_plan  exclusive digit offsets; marks passes whose digit is the same
//                for every key (they are skipped) and routes the buffers
//   k_sort_pass  per 4096-key tile: wave-level match ranking (ballots over the
//                digit bits), per-wave LDS counters, look-back over earlier
//                tiles' per-digit counts, reorder through LDS, coalesced runs
//                of global writes
// Tiles take tickets from an atomic counter, so a tile only ever waits on
// tiles that are already running.
#include "common.h"
#include "kernels.h"

namespace ds {
namespace {

constexpr int kThreads = 256;
constexpr int kPer = 16;
constexpr uint32_t kTile = kThreads * kPer;   // 4096 keys
constexpr int kMaxPasses = 8;
constexpr uint32_t kAgg = 1u << 30;
constexpr uint32_t kPre = 2u << 30;
constexpr uint32_t kValMask = (1u << 30) - 1u;

struct SortCtl {
    uint32_t hist[kMaxPasses][256];
    uint32_t excl[kMaxPasses][256];
    uint32_t ticket[kMaxPasses];
    uint32_t active[kMaxPasses];
    uint32_t src[kMaxPasses];
    int32_t last;
    uint32_t pad[7];
};

struct SortBufs {
    SortCtl *ctl;
    uint64_t *key[2];
    uint32_t *val[2];
    uint32_t *status;       // [passes][tiles][256]
    uint32_t passes;
    uint32_t tiles;
};

__host__ __device__ inline uint32_t n_passes(uint32_t key_bits)
{
    uint32_t p = (key_bits + 7) / 8;
    return p == 0 ? 1 : (p > kMaxPasses ? kMaxPasses : p);
}

__device__ __forceinline__ void produce(const SortInput &in, uint32_t j, uint64_t &k, uint32_t &v)
{
    switch (in.kind) {
    case SortKind::Fifo: {
        double a = in.arrival[j];
        k = ordered_bits(a);
        v = j;
        if (in.key_out) in.key_out[j] = a;
        break;
    }
    case SortKind::Budget: {
        uint32_t i = in.fifo[j];
        i = i < in.n ? i : 0;
        double b = in.budget[i];
        k = ordered_bits(b);
        v = i;
        if (in.key_out) in.key_out[i] = b;
        break;
    }
    case SortKind::Aging: {
        uint32_t i = in.fifo[j];
        i = i < in.n ? i : 0;
        uint32_t q = in.tier[i];
        q = q < 16 ? q : 15;
        double w = in.t_now - in.arrival[i];
        if (w < 0.0) w = 0.0;
        double d = in.aging_rate * w;
        double e = in.prio[q] - d;
        if (e < in.aging_floor) e = in.aging_floor;
        k = ordered_bits(e);
        v = i;
        if (in.key_out) in.key_out[i] = e;
        break;
    }
    case SortKind::Class: {
        uint32_t i = in.fifo[j];
        i = i < in.n ? i : 0;
        uint32_t q = in.tier[i];
        q = q < 16 ? q : 15;
        k = in.cls[q];
        v = i;
        if (in.key_out) in.key_out[i] = in.prio[q];
        break;
    }
    case SortKind::Tier: {
        uint32_t i = in.fifo[j];
        i = i < in.n ? i : 0;
        uint32_t q = in.tier[i];
        k = q < 16 ? q : 15;
        v = i;
        break;
    }
    default: {   // Group
        k = in.group[j];
        v = j;
        break;
    }
    }
}

__global__ void k_sort_zero(SortCtl *__restrict__ ctl, uint32_t *__restrict__ status, uint64_t words)
{
    uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    uint32_t *c = reinterpret_cast<uint32_t *>(ctl);
    for (uint64_t i = t; i < sizeof(SortCtl) / 4; i += stride) c[i] = 0;
    for (uint64_t i = t; i < words; i += stride) status[i] = 0;
}

__global__ __launch_bounds__(256) void k_sort_init(SortInput in, SortBufs sb)
{
    __shared__ uint32_t h[kMaxPasses][256];
    const uint32_t P = sb.passes;
    for (uint32_t i = threadIdx.x; i < P * 256; i += blockDim.x) (&h[0][0])[i] = 0;
    __syncthreads();
    for (uint32_t j = blockIdx.x * blockDim.x + threadIdx.x; j < in.n; j += gridDim.x * blockDim.x) {
        uint64_t k;
        uint32_t v;
        produce(in, j, k, v);
        sb.key[0][j] = k;
        sb.val[0][j] = v;
        for (uint32_t p = 0; p < P; p++) atomicAdd(&h[p][(k >> (8 * p)) & 255u], 1u);
    }
    __syncthreads();
    for (uint32_t i = threadIdx.x; i < P * 256; i += blockDim.x) {
        uint32_t c = (&h[0][0])[i];
        if (c) atomicAdd(&sb.ctl->hist[i / 256][i % 256], c);
    }
}

// Exclusive scan of one value per thread over a 256-thread block.
__device__ uint32_t block_excl_scan256(uint32_t x, uint32_t *tmp4)
{
    uint32_t incl = wave_incl_scan(x);
    int w = threadIdx.x >> 6;
    if (lane_id() == 63) tmp4[w] = incl;
    __syncthreads();
    uint32_t off = 0;
    for (int k = 0; k < w; k++) off += tmp4[k];
    __syncthreads();
    return off + incl - x;
}

__global__ __launch_bounds__(256) void k_sort_plan(SortBufs sb, uint32_t n)
{
    __shared__ uint32_t tmp4[4];
    __shared__ uint32_t act[kMaxPasses];
    const uint32_t d = threadIdx.x;
    for (uint32_t p = 0; p < sb.passes; p++) {
        uint32_t c = sb.ctl->hist[p][d];
        int full = __syncthreads_or(c == n ? 1 : 0);
        uint32_t e = block_excl_scan256(c, tmp4);
        sb.ctl->excl[p][d] = e;
        if (d == 0) act[p] = full ? 0u : 1u;
    }
    __syncthreads();
    if (d == 0) {
        uint32_t cur = 0;
        int32_t last = -1;
        for (uint32_t p = 0; p < sb.passes; p++) {
            sb.ctl->active[p] = act[p];
            sb.ctl->src[p] = cur;
            if (act[p]) { cur ^= 1u; last = (int32_t)p; }
        }
        sb.ctl->last = last;
    }
}

// Weighted round robin position of the k-th (FIFO) request of tier q:
// rounds before r = floor(k / w_q) dispatch sum_q' min(n_q', r w_q'); in
// round r the tiers before q dispatch min(w_q', max(0, n_q' - r w_q')).
__device__ __forceinline__ uint64_t wrr_pos(const SortInput &in, const uint32_t *cnt, uint32_t q,
                                            uint64_t k, uint64_t &round)
{
    uint64_t wq = in.weight[q] ? in.weight[q] : 1;
    uint64_t r = k / wq;
    uint64_t pos = k - r * wq;
    for (uint32_t t = 0; t < in.n_tiers; t++) {
        uint64_t nt = cnt[t], wt = in.weight[t];
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

__global__ __launch_bounds__(kThreads) void k_sort_pass(SortInput in, SortBufs sb, uint32_t p,
                                                        uint32_t *__restrict__ out)
{
    __shared__ uint32_t s_ticket;
    __shared__ uint32_t wcnt[4][256];
    __shared__ uint32_t texcl[256];
    __shared__ uint32_t gbase[256];
    __shared__ uint32_t tmp4[4];
    __shared__ uint64_t lkey[kTile];
    __shared__ uint32_t lval[kTile];

    const SortCtl *ctl = sb.ctl;
    const uint32_t n = in.n;
    if (!ctl->active[p]) {
        // a pass whose digit is constant is skipped; if no pass is active
        // the input order is the result (the last pass copies it out)
        if (p + 1 == sb.passes && ctl->last < 0) {
            for (uint32_t j = blockIdx.x * blockDim.x + threadIdx.x; j < n; j += gridDim.x * blockDim.x) {
                uint32_t val = sb.val[0][j];
                out[j] = val;
                if (in.kind == SortKind::Tier && in.key_out) {
                    // one non-empty tier: the k-th request is served in round k / w
                    uint32_t q = (uint32_t)sb.key[0][j] & 15u;
                    uint32_t wq = in.weight[q] ? in.weight[q] : 1u;
                    if (val < n) in.key_out[val] = (double)(j / wq);
                }
            }
        }
        return;
    }
    const uint32_t t = threadIdx.x;
    const int w = (int)(t >> 6);
    const int lane = lane_id();
    if (t == 0) s_ticket = atomicAdd(&sb.ctl->ticket[p], 1u);
    for (uint32_t i = t; i < 4 * 256; i += kThreads) (&wcnt[0][0])[i] = 0;
    __syncthreads();
    const uint32_t tile = s_ticket;
    const uint32_t base = tile * kTile;
    const uint32_t cnt = n - base < kTile ? n - base : kTile;
    const uint32_t shift = 8 * p;
    const uint32_t srcb = ctl->src[p];
    const uint64_t *ik = sb.key[srcb];
    const uint32_t *iv = sb.val[srcb];
    const bool last = (int32_t)p == ctl->last;

    uint64_t k[kPer];
    uint32_t v[kPer];
    uint32_t rk[kPer];
#pragma unroll
    for (int r = 0; r < kPer; r++) {
        uint32_t idx = (uint32_t)w * (kTile / 4) + (uint32_t)r * 64u + (uint32_t)lane;
        bool ok = idx < cnt;
        k[r] = ok ? ik[base + idx] : 0ull;
        v[r] = ok ? iv[base + idx] : 0u;
    }
    // stable rank within the wave, round by round (rounds are in index order)
#pragma unroll
    for (int r = 0; r < kPer; r++) {
        uint32_t idx = (uint32_t)w * (kTile / 4) + (uint32_t)r * 64u + (uint32_t)lane;
        bool ok = idx < cnt;
        uint32_t d = (uint32_t)(k[r] >> shift) & 255u;
        uint64_t peers = __ballot(ok);
#pragma unroll
        for (int b = 0; b < 8; b++) {
            bool bit = (d >> b) & 1u;
            uint64_t bb = __ballot(bit);
            peers &= bit ? bb : ~bb;
        }
        uint32_t below = (uint32_t)__popcll(peers & lanemask_lt());
        uint32_t old = ok ? wcnt[w][d] : 0u;
        rk[r] = old + below;
        if (ok && below == 0) wcnt[w][d] = old + (uint32_t)__popcll(peers);
        __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();
    // per digit (thread t = digit): tile count, per-wave exclusive offsets
    uint32_t c0 = wcnt[0][t], c1 = wcnt[1][t], c2 = wcnt[2][t], c3 = wcnt[3][t];
    uint32_t tc = c0 + c1 + c2 + c3;
    wcnt[0][t] = 0;
    wcnt[1][t] = c0;
    wcnt[2][t] = c0 + c1;
    wcnt[3][t] = c0 + c1 + c2;
    texcl[t] = block_excl_scan256(tc, tmp4);
    // decoupled look-back over earlier tiles for digit t
    uint32_t *st = sb.status + (uint64_t)p * sb.tiles * 256u;
    uint32_t prefix = 0;
    if (tile == 0) {
        st_relaxed(&st[t], kPre | tc);
    } else {
        st_relaxed(&st[(uint64_t)tile * 256u + t], kAgg | tc);
        int64_t j = (int64_t)tile - 1;
        while (true) {
            uint32_t x = ld_relaxed(&st[(uint64_t)j * 256u + t]);
            if ((x & ~kValMask) == 0) { __builtin_amdgcn_s_sleep(1); continue; }
            prefix += x & kValMask;
            if ((x & ~kValMask) == kPre) break;
            j--;
        }
        st_relaxed(&st[(uint64_t)tile * 256u + t], kPre | (prefix + tc));
    }
    gbase[t] = ctl->excl[p][t] + prefix;
    __syncthreads();
    // reorder the tile through LDS by digit
#pragma unroll
    for (int r = 0; r < kPer; r++) {
        uint32_t idx = (uint32_t)w * (kTile / 4) + (uint32_t)r * 64u + (uint32_t)lane;
        if (idx < cnt) {
            uint32_t d = (uint32_t)(k[r] >> shift) & 255u;
            uint32_t lp = texcl[d] + wcnt[w][d] + rk[r];
            lkey[lp] = k[r];
            lval[lp] = v[r];
        }
    }
    __syncthreads();
    if (in.kind == SortKind::Tier) {
        // single pass: digit = tier; scatter to the weighted position
        const uint32_t *tcount = ctl->hist[0];
        for (uint32_t s = t; s < cnt; s += kThreads) {
            uint32_t q = (uint32_t)lkey[s] & 255u;
            uint32_t g = gbase[q] + s - texcl[q];
            uint64_t kq = g - ctl->excl[0][q];
            uint64_t rnd;
            uint64_t pos = wrr_pos(in, tcount, q, kq, rnd);
            uint32_t val = lval[s];
            if (pos < n) out[pos] = val;   // always true when tiers are < n_tiers
            if (in.key_out && val < n) in.key_out[val] = (double)rnd;
        }
        return;
    }
    uint64_t *ok_ = sb.key[srcb ^ 1u];
    uint32_t *ov = last ? out : sb.val[srcb ^ 1u];
    for (uint32_t s = t; s < cnt; s += kThreads) {
        uint64_t kk = lkey[s];
        uint32_t d = (uint32_t)(kk >> shift) & 255u;
        uint32_t g = gbase[d] + s - texcl[d];
        ov[g] = lval[s];
        if (!last) ok_[g] = kk;
    }
}

void carve(void *ws, uint64_t n, uint32_t key_bits, SortBufs &b)
{
    uint8_t *p = static_cast<uint8_t *>(ws);
    b.ctl = reinterpret_cast<SortCtl *>(p);
    p += align_up(sizeof(SortCtl), 256);
    for (int i = 0; i < 2; i++) {
        b.key[i] = reinterpret_cast<uint64_t *>(p);
        p += align_up(n * 8, 256);
    }
    for (int i = 0; i < 2; i++) {
        b.val[i] = reinterpret_cast<uint32_t *>(p);
        p += align_up(n * 4, 256);
    }
    b.passes = n_passes(key_bits);
    b.tiles = (uint32_t)cdiv(n, kTile);
    b.status = reinterpret_cast<uint32_t *>(p);
}

}  // namespace

size_t sort_ws_bytes(uint64_t n, uint32_t key_bits)
{
    uint64_t tiles = cdiv(n, kTile);
    return align_up(sizeof(SortCtl), 256) + 2 * align_up(n * 8, 256) + 2 * align_up(n * 4, 256) +
           align_up((uint64_t)n_passes(key_bits) * tiles * 256 * 4, 256);
}

hipError_t sort_launch(const SortInput &in, uint32_t *out, void *ws, hipStream_t s)
{
    if (in.n == 0) return hipSuccess;
    SortBufs b;
    carve(ws, in.n, in.key_bits, b);
    uint64_t words = (uint64_t)b.passes * b.tiles * 256u;
    uint32_t zb = (uint32_t)(cdiv(words, 256) < 1024 ? cdiv(words, 256) : 1024);
    hipLaunchKernelGGL(k_sort_zero, dim3(zb ? zb : 1), dim3(256), 0, s, b.ctl, b.status, words);
    uint32_t ib = (uint32_t)(cdiv(in.n, 256 * 8) < 1024 ? cdiv(in.n, 256 * 8) : 1024);
    hipLaunchKernelGGL(k_sort_init, dim3(ib ? ib : 1), dim3(256), 0, s, in, b);
    hipLaunchKernelGGL(k_sort_plan, dim3(1), dim3(256), 0, s, b, in.n);
    for (uint32_t p = 0; p < b.passes; p++)
        hipLaunchKernelGGL(k_sort_pass, dim3(b.tiles), dim3(kThreads), 0, s, in, b, p, out);
    return hipGetLastError();
}

}  // namespace ds
