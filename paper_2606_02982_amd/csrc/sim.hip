// Dispatch ticks of the online loop: the scheduler dispatches pending
// requests in batches (Sec. "Experimental Configuration": batch size 32) and
// keeps refining its estimates from completed requests (Sec. "Calibration
// and Evaluation Phases"; Sec. "Runtime Calibration and Feedback
// Adaptation", Eq. (5) with the ratio of Eq. (6)).
//
// At tick k (time t_k) the pending set is every request with arrival <= t_k
// that has not been dispatched. It is ordered by the policy (ties in FIFO
// order) with the factors as they stand: SJF scores budgets (Eq. (1), (2))
// from the current factors, Aging ages to t_k, Weighted starts a fresh
// round-robin cycle over the pending tier queues (blocked or smooth). The first min(batch,
// pending) requests are dispatched, and their completions (observed length
// against the B-free admission estimate) update the factors in dispatch
// order before the next tick.
//
// The loop is sequential across ticks and each tick needs only the first
// `batch` requests of the order, so one workgroup runs every tick of a run
// in a single launch (several runs, e.g. the five policies, are blocks of
// the same launch, after one shared FIFO sort):
//   * the pending set is a list in FIFO order: arrivals join its end (they
//     come after every pending request in FIFO order) and the previous
//     tick's dispatches are compacted out in the same pass that computes
//     this tick's keys;
//   * FIFO, Priority and Weighted need no comparison sort: a request's place
//     in the order follows from its rank within its class or tier queue and
//     the queue lengths (the Weighted place is the closed form of the
//     round-robin cycle);
//   * SJF and Aging select the `batch` smallest (key, list position) pairs
//     by an MSD radix select over the 96-bit pair, moving to LDS once the
//     surviving bucket is small, and rank the selected few by counting;
//   * the EMA updates of a batch run per group in parallel, each group's
//     events in dispatch order, so the factors are bit-identical to a
//     sequential evaluation.
#include <string.h>

#include "common.h"
#include "kernels.h"
#include "wrrplan.h"

namespace ds {
namespace {

constexpr uint32_t kTPB = 1024;
constexpr uint32_t kNW = kTPB / 64;
constexpr uint32_t kCand = 4096;            // LDS candidates of the radix select
constexpr uint32_t kTomb = 0x80000000u;      // list entry dispatched at the last tick
constexpr uint32_t kMaxQ = 16;               // tiers / priority classes
enum : uint32_t { kFifo = 0, kPriority = 1, kWeighted = 2, kSjf = 3, kAging = 4 };

// Per-request constants of the keys: SJF {T_base, S_tenant, F_input, words},
// Aging {arrival, tier priority}.
struct alignas(16) Aux {
    double a, b, c, d;
};

struct SetupArgs {
    uint32_t n, policy, n_cat, n_tenants, n_tiers;
    const uint32_t *counts, *tenant;
    const uint8_t *category, *tier;
    const double *t_base, *s_tenant, *arrival;
    double f_ref;
    uint32_t cls[kMaxQ];
    double prio[kMaxQ];
    double *est_base;
    Aux *aux;
    uint8_t *val;
    uint32_t *seq;
    int32_t *tick_of;
    uint32_t *wait_status;   // or NULL: zeroed here, before the FIFO sort's waits
};

struct EngineArgs {
    uint32_t n, n_groups, policy, batch, n_ticks, n_q;
    const double *tick_t;
    const uint32_t *fifo;
    const double *arrival;
    const uint32_t *group, *observed;
    const double *est_base;
    const Aux *aux;
    const uint8_t *val;
    uint32_t weight[kMaxQ];
    uint32_t wrr_mode;         // Weighted: kWrrBlocked, kWrrSmooth or kWrrStride
    double alpha, aging_rate, aging_floor;
    double *state;
    uint32_t *list[2];
    uint64_t *key;
    uint32_t *seq;
    int32_t *tick_of;
    uint32_t *n_dispatched;
    // the queue engine (every policy but SJF): the FIFO positions tier by
    // tier (rpos, with each tier's first entry in rstart), and candidate
    // scratch of kMaxQ x batch entries
    const uint32_t *rpos, *rstart;
    uint64_t *cand_k;
    uint32_t *cand_j, *cand_i;
};

// Several runs share one launch: run r is block row r of the setup and block
// r of the engine.
struct SetupBatch {
    SetupArgs r[kSimMaxRuns];
};
struct EngineBatch {
    EngineArgs r[kSimMaxRuns];
};
static_assert(sizeof(SetupBatch) <= 4096 && sizeof(EngineBatch) <= 4096, "kernel arguments within 4 KB");

__global__ void k_sim_setup(SetupBatch sb)
{
    const SetupArgs &a = sb.r[blockIdx.y];
    if (a.wait_status && blockIdx.x == 0 && threadIdx.x == 0) *a.wait_status = 0;
    const double nan = __builtin_nan("");
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < a.n; i += gridDim.x * blockDim.x) {
        const uint32_t cat = a.category[i], ten = a.tenant[i];
        const double words = (double)a.counts[i];
        const double tb = cat < a.n_cat ? a.t_base[cat] : nan;
        const double s = ten < a.n_tenants ? a.s_tenant[ten] : nan;
        const double F = 1.0 + words / a.f_ref;
        // the B-free estimate of Eq. (2), in the order of Alg. 1
        double e0 = tb * s;
        e0 = e0 * F;
        a.est_base[i] = e0;
        // a tier outside the contract joins the last queue
        uint32_t q = a.tier[i];
        q = q < a.n_tiers ? q : a.n_tiers - 1;
        if (a.policy == kSjf) a.aux[i] = Aux{tb, s, F, words};
        if (a.policy == kAging) a.aux[i] = Aux{a.arrival[i], a.prio[q], 0.0, 0.0};
        if (a.policy == kPriority) a.val[i] = (uint8_t)a.cls[q];
        if (a.policy == kWeighted) a.val[i] = (uint8_t)q;
        a.seq[i] = 0xFFFFFFFFu;
        a.tick_of[i] = -1;
    }
}

__device__ __forceinline__ uint64_t shfl_xor64(uint64_t x, int m)
{
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)x, m, 64);
    const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(x >> 32), m, 64);
    return ((uint64_t)hi << 32) | lo;
}

// Exclusive prefix of x over the block; total receives the block sum.
__device__ __forceinline__ uint32_t block_scan(uint32_t x, uint32_t *s_w, uint32_t &total)
{
    const uint32_t inc = wave_incl_scan_dpp(x);
    const uint32_t w = threadIdx.x >> 6;
    if (lane_id() == 63) s_w[w] = inc;
    __syncthreads();
    uint32_t off = 0, tot = 0;
#pragma unroll
    for (uint32_t k = 0; k < kNW; k++) {
        const uint32_t v = s_w[k];
        off += k < w ? v : 0u;
        tot += v;
    }
    __syncthreads();
    total = tot;
    return off + inc - x;
}

// Place in the round-robin order of the r-th (FIFO) pending request of tier
// q, with cnt[t] pending requests in tier t: the rounds before round
// floor(r / w_q) serve min(cnt_t, rounds * w_t) of each tier, and in that
// round the tiers before q serve min(w_t, what they have left).
__device__ __forceinline__ uint64_t wrr_place(uint32_t q, uint32_t r, const uint32_t *cnt,
                                              const uint32_t *wt, uint32_t nq)
{
    const uint64_t wq = wt[q];
    const uint64_t rounds = r / wq;
    uint64_t pos = r - rounds * wq;
    for (uint32_t t = 0; t < nq; t++) {
        const uint64_t c = cnt[t], full = rounds * wt[t];
        pos += c < full ? c : full;
        if (t < q) {
            const uint64_t left = c > full ? c - full : 0;
            pos += left < wt[t] ? left : wt[t];
        }
    }
    return pos;
}

// Digit d of the pair (key, list position): d = 11..4 are the key's bytes,
// d = 3..0 the position's.
__device__ __forceinline__ uint32_t pair_digit(uint64_t K, uint32_t J, int d)
{
    return d >= 4 ? (uint32_t)(K >> (8 * (d - 4))) & 255u : (J >> (8 * d)) & 255u;
}

__device__ void engine_list(const EngineArgs &a)
{
    __shared__ uint32_t s_w[kNW];
    __shared__ uint32_t s_hist[256];
    __shared__ uint32_t s_vw[kNW][kMaxQ];
    __shared__ uint32_t s_cnt[kMaxQ];
    __shared__ uint32_t s_wt[kMaxQ];
    __shared__ uint32_t s_pick[4];
    __shared__ uint64_t s_kmin[kNW], s_kmax[kNW];
    __shared__ uint32_t s_selpos[kSimMaxBatch];
    __shared__ uint64_t s_selK[kSimMaxBatch];
    __shared__ uint32_t s_selJ[kSimMaxBatch];
    __shared__ uint32_t s_evg[kSimMaxBatch], s_evo[kSimMaxBatch];
    __shared__ double s_evx[kSimMaxBatch];
    // Priority/Weighted: list positions of the first `batch` pending requests
    // of each queue; SJF/Aging: the radix select's candidates
    __shared__ union {
        uint32_t first[kMaxQ][kSimMaxBatch];
        struct {
            uint64_t k[kCand];
            uint32_t j[kCand];
        } cand;
    } s_big;

    const uint32_t tid = threadIdx.x, lane = (uint32_t)lane_id(), w = tid >> 6;
    const uint32_t n = a.n, policy = a.policy, batch = a.batch, nq = a.n_q;
    const bool keyed = policy == kSjf || policy == kAging;
    const bool queued = policy == kPriority || policy == kWeighted;
    const double oma = 1.0 - a.alpha;
    const double nan = __builtin_nan("");
    if (tid < kMaxQ) s_wt[tid] = a.weight[tid];

    uint32_t cur = 0;     // list buffer holding the pending list
    uint32_t P = 0;       // its entries (pending + last tick's dispatches)
    uint32_t A = 0;       // FIFO positions appended so far
    uint32_t total = 0;   // requests dispatched so far
    __syncthreads();
    for (uint32_t k = 0; k < a.n_ticks; k++) {
        const double t = a.tick_t[k];
        uint32_t *L = a.list[cur];
        uint32_t *Ln = a.list[cur ^ 1u];

        // 1. arrivals up to t join the end of the list; arrival is
        //    non-decreasing in FIFO order, so they are a prefix of each chunk
        while (A < n) {
            const uint32_t j = A + tid;
            uint32_t id = 0;
            bool arrived = false;
            if (j < n) {
                id = a.fifo[j];
                id = id < n ? id : 0u;   // the FIFO order is a permutation of 0..n-1
                arrived = a.arrival[id] <= t;
            }
            const uint32_t c = (uint32_t)__syncthreads_count(arrived);
            if (arrived) L[P + tid] = id;
            P += c;
            A += c;
            if (c < kTPB) break;
        }

        // 2. drop the last tick's dispatches into the other buffer, and
        //    compute keys (SJF, Aging) or queue ranks (Priority, Weighted)
        if (tid < kMaxQ) s_cnt[tid] = 0;
        uint64_t kmin = ~0ull, kmax = 0;
        uint32_t Pn = 0;
        __syncthreads();
        for (uint32_t c0 = 0; c0 < P; c0 += kTPB) {
            const uint32_t j = c0 + tid;
            const uint32_t id = j < P ? L[j] : kTomb;
            const bool alive = !(id & kTomb);
            uint32_t tot;
            const uint32_t np = Pn + block_scan(alive ? 1u : 0u, s_w, tot);
            if (alive) {
                Ln[np] = id;
                if (keyed) {
                    const Aux x = a.aux[id];
                    double e;
                    if (policy == kSjf) {
                        // Eq. (2) in the order of Alg. 1, then Eq. (1)
                        const uint32_t g = a.group[id];
                        const double B = g < a.n_groups ? a.state[g] : nan;
                        e = x.a * B;
                        e = e * x.b;
                        e = e * x.c;
                        e = x.d + e;
                    } else {
                        double wt = t - x.a;
                        if (wt < 0.0) wt = 0.0;
                        const double d = a.aging_rate * wt;
                        e = x.b - d;
                        if (e < a.aging_floor) e = a.aging_floor;
                    }
                    const uint64_t kk = ordered_bits(e);
                    a.key[np] = kk;
                    kmin = kk < kmin ? kk : kmin;
                    kmax = kk > kmax ? kk : kmax;
                }
            }
            if (queued) {
                const uint32_t v = alive ? a.val[id] : 0xFFu;
                uint64_t mine = 0;
                for (uint32_t q = 0; q < nq; q++) {
                    const uint64_t b = __ballot(v == q);
                    if (lane == 0) s_vw[w][q] = (uint32_t)__popcll(b);
                    mine = v == q ? b : mine;
                }
                __syncthreads();
                if (v < nq) {
                    uint32_t r = s_cnt[v] + (uint32_t)__popcll(mine & lanemask_lt());
                    for (uint32_t u = 0; u < w; u++) r += s_vw[u][v];
                    if (r < batch) s_big.first[v][r] = np;
                }
                __syncthreads();
                if (tid < nq) {
                    uint32_t c = 0;
                    for (uint32_t u = 0; u < kNW; u++) c += s_vw[u][tid];
                    s_cnt[tid] += c;
                }
                __syncthreads();
            }
            Pn += tot;
        }
        __syncthreads();   // the new list and keys, written by other threads, are read below
        P = Pn;
        cur ^= 1u;
        L = Ln;
        const uint32_t m = P < batch ? P : batch;
        if (m == 0) continue;

        // 3. list positions of the first m requests of the order
        if (policy == kFifo) {
            if (tid < m) s_selpos[tid] = tid;
        } else if (policy == kWeighted && a.wrr_mode == kWrrSmooth) {
            // the first m dispatches of a fresh smooth cycle, one per step,
            // by one wave (lane q = tier q); a queue running empty leaves and
            // the others keep their credits
            if (w == 0) {
                const uint32_t len = lane < nq ? s_cnt[lane] : 0u;
                const uint32_t wq = lane < nq ? s_wt[lane] : 0u;
                uint32_t served = 0;
                int32_t credit = 0;
                uint32_t W = wave_sum(len ? wq : 0u);
                for (uint32_t pos = 0; pos < m; pos++) {
                    const int b = wrr_pick(credit, served < len, wq, W);
                    const bool mine = lane == (uint32_t)b;
                    if (mine) s_selpos[pos] = s_big.first[lane][served];   // served < m <= batch
                    served += mine ? 1u : 0u;
                    if (__ballot(mine && served == len) != 0ull) W = wave_sum(served < len ? wq : 0u);
                }
            }
        } else if (queued) {
            for (uint32_t p = tid; p < nq * batch; p += kTPB) {
                const uint32_t q = p / batch, r = p - q * batch;
                if (r >= s_cnt[q]) continue;
                uint64_t pos;
                if (policy == kPriority) {
                    pos = r;
                    for (uint32_t u = 0; u < q; u++) pos += s_cnt[u];
                } else if (a.wrr_mode == kWrrStride) {
                    pos = wrr_stride_pos(q, r, s_wt, nq, [&](uint32_t u) { return s_cnt[u]; });
                } else {
                    pos = wrr_place(q, r, s_cnt, s_wt, nq);
                }
                if (pos < m) s_selpos[pos] = s_big.first[q][r];
            }
        } else {
            uint32_t ns;   // selected pairs in s_selK/s_selJ
            if (P == m) {
                for (uint32_t j = tid; j < P; j += kTPB) {
                    s_selK[j] = a.key[j];
                    s_selJ[j] = j;
                }
                ns = P;
            } else {
                // common leading bytes of all keys need no pass
#pragma unroll
                for (int s = 32; s >= 1; s >>= 1) {
                    const uint64_t x = shfl_xor64(kmin, s), y = shfl_xor64(kmax, s);
                    kmin = x < kmin ? x : kmin;
                    kmax = y > kmax ? y : kmax;
                }
                if (lane == 0) {
                    s_kmin[w] = kmin;
                    s_kmax[w] = kmax;
                }
                __syncthreads();
                kmin = s_kmin[0];
                kmax = s_kmax[0];
                for (uint32_t u = 1; u < kNW; u++) {
                    kmin = s_kmin[u] < kmin ? s_kmin[u] : kmin;
                    kmax = s_kmax[u] > kmax ? s_kmax[u] : kmax;
                }
                uint64_t TK = 0, mK = 0;   // fixed bits of the threshold pair and their masks
                uint32_t TJ = 0, mJ = 0;
                int d;
                if (kmin != kmax) {
                    const int byte = (63 - __clzll((long long)(kmin ^ kmax))) >> 3;
                    mK = byte == 7 ? 0ull : ~0ull << (8 * (byte + 1));
                    TK = kmin & mK;
                    d = 4 + byte;
                } else {
                    TK = kmin;
                    mK = ~0ull;
                    const uint32_t x = P - 1;   // positions 0 .. P-1
                    const int byte = x ? (31 - __clz((int)x)) >> 3 : 0;
                    mJ = byte == 3 ? 0u : ~0u << (8 * (byte + 1));
                    d = byte;
                }
                uint32_t need = m;      // pairs still to select among those matching the prefix
                bool in_lds = false;
                uint32_t nc = 0;
                for (; d >= 0; d--) {
                    if (tid < 256) s_hist[tid] = 0;
                    __syncthreads();
                    if (in_lds) {
                        for (uint32_t i = tid; i < nc; i += kTPB) {
                            const uint64_t K = s_big.cand.k[i];
                            const uint32_t J = s_big.cand.j[i];
                            if ((K & mK) == TK && (J & mJ) == TJ)
                                atomicAdd(&s_hist[pair_digit(K, J, d)], 1u);
                        }
                    } else {
                        for (uint32_t j = tid; j < P; j += kTPB) {
                            const uint64_t K = a.key[j];
                            if ((K & mK) == TK && (j & mJ) == TJ)
                                atomicAdd(&s_hist[pair_digit(K, j, d)], 1u);
                        }
                    }
                    __syncthreads();
                    const uint32_t h = tid < 256 ? s_hist[tid] : 0u;
                    uint32_t tot;
                    const uint32_t ex = block_scan(h, s_w, tot);
                    if (tid < 256 && ex < need && need <= ex + h) {
                        s_pick[0] = tid;
                        s_pick[1] = ex;
                        s_pick[2] = h;
                    }
                    __syncthreads();
                    const uint32_t b = s_pick[0], cnt_b = s_pick[2];
                    need -= s_pick[1];
                    if (d >= 4) {
                        TK |= (uint64_t)b << (8 * (d - 4));
                        mK |= 0xFFull << (8 * (d - 4));
                    } else {
                        TJ |= b << (8 * d);
                        mJ |= 0xFFu << (8 * d);
                    }
                    if (cnt_b == need) {
                        // the whole bucket is selected: everything up to its largest pair
                        if (d >= 4) {
                            TK |= (1ull << (8 * (d - 4))) - 1ull;
                            TJ = 0xFFFFFFFFu;
                        } else {
                            TJ |= (1u << (8 * d)) - 1u;
                        }
                        break;
                    }
                    if (!in_lds && cnt_b <= kCand) {
                        if (tid == 0) s_pick[3] = 0;
                        __syncthreads();
                        for (uint32_t j = tid; j < P; j += kTPB) {
                            const uint64_t K = a.key[j];
                            if ((K & mK) == TK && (j & mJ) == TJ) {
                                const uint32_t slot = atomicAdd(&s_pick[3], 1u);
                                if (slot < kCand) {
                                    s_big.cand.k[slot] = K;
                                    s_big.cand.j[slot] = j;
                                }
                            }
                        }
                        __syncthreads();
                        nc = s_pick[3] < kCand ? s_pick[3] : kCand;
                        in_lds = true;
                    }
                    __syncthreads();
                }
                // the selected pairs: all pairs up to the threshold
                if (tid == 0) s_pick[3] = 0;
                __syncthreads();
                for (uint32_t j = tid; j < P; j += kTPB) {
                    const uint64_t K = a.key[j];
                    if (K < TK || (K == TK && j <= TJ)) {
                        const uint32_t slot = atomicAdd(&s_pick[3], 1u);
                        if (slot < kSimMaxBatch) {
                            s_selK[slot] = K;
                            s_selJ[slot] = j;
                        }
                    }
                }
                __syncthreads();
                ns = s_pick[3] < m ? s_pick[3] : m;
            }
            __syncthreads();
            // rank the selected pairs by counting
            if (tid < ns) {
                const uint64_t K = s_selK[tid];
                const uint32_t J = s_selJ[tid];
                uint32_t r = 0;
                for (uint32_t u = 0; u < ns; u++) {
                    const uint64_t K2 = s_selK[u];
                    r += (K2 < K || (K2 == K && s_selJ[u] < J)) ? 1u : 0u;
                }
                s_selpos[r] = J;
            }
        }
        __syncthreads();

        // 4. dispatch, and the completion events of the batch
        if (tid < m) {
            const uint32_t j = s_selpos[tid];
            uint32_t id = j < P ? L[j] : kTomb;
            if (id >= n) id = 0;   // unreachable: the m places are filled by pending requests
            if (total + tid < n) a.seq[total + tid] = id;
            a.tick_of[id] = (int32_t)k;
            if (j < P) L[j] = id | kTomb;
            s_evg[tid] = a.group[id];
            s_evx[tid] = a.est_base[id];
            s_evo[tid] = a.observed[id];
        }
        __syncthreads();

        // 5. Eq. (5) with the ratio of Eq. (6): each group's first event of
        //    the batch walks that group's events in dispatch order
        if (tid < m) {
            const uint32_t g = s_evg[tid];
            bool lead = g < a.n_groups;
            for (uint32_t r = 0; r < tid && lead; r++) lead = s_evg[r] != g;
            if (lead) {
                double c = a.state[g];
                for (uint32_t r = tid; r < m; r++) {
                    if (s_evg[r] != g) continue;
                    const double x = s_evx[r];
                    if (!(isfinite(x) && x > 0.0)) continue;
                    const double ratio = (double)s_evo[r] / x;
                    const double t1 = oma * c;
                    const double t2 = a.alpha * ratio;
                    c = t1 + t2;
                }
                a.state[g] = c;
            }
        }
        total += m;
        __syncthreads();
    }
    if (tid == 0) a.n_dispatched[0] = total;
}

// The loop for FIFO, Priority, Weighted and Aging with one queue per tier.
// Within a tier each of these orders is the FIFO order (Aging's score is
// monotone in the arrival for a fixed priority), so the pending requests of
// tier q are always the stretch [head_q, tail_q) of the tier's FIFO run:
// arrivals move tail_q, dispatches move head_q. The first m dispatches of a
// tick are among the first m pending requests of each tier; those
// candidates are ranked by the policy's key across tiers (a binary search
// in every other tier's candidates, which are in key order) or placed by
// the round-robin closed forms, so a tick costs O(tiers x batch) rather
// than a pass over the pending set. Results equal the list engine's.
__device__ void engine_queues(const EngineArgs &a)
{
    __shared__ uint32_t s_head[kMaxQ], s_tail[kMaxQ], s_cnt[kMaxQ], s_d[kMaxQ], s_wt[kMaxQ];
    __shared__ uint32_t s_sel[kSimMaxBatch];
    __shared__ uint32_t s_evg[kSimMaxBatch], s_evo[kSimMaxBatch];
    __shared__ double s_evx[kSimMaxBatch];
    const uint32_t tid = threadIdx.x, lane = (uint32_t)lane_id(), w = tid >> 6;
    const uint32_t n = a.n, policy = a.policy, batch = a.batch, nq = a.n_q;
    const double oma = 1.0 - a.alpha;
    if (tid < kMaxQ) {
        s_head[tid] = 0;
        s_tail[tid] = 0;
        s_wt[tid] = a.weight[tid];
    }
    uint32_t total = 0;
    __syncthreads();
    for (uint32_t k = 0; k < a.n_ticks; k++) {
        const double t = a.tick_t[k];
        // 1. arrivals: wave q moves tier q's tail over its requests with
        //    arrival <= t (a prefix of the rest of its FIFO run)
        if (w < nq) {
            const uint32_t r0 = a.rstart[w], len = a.rstart[w + 1] - r0;
            uint32_t tail = s_tail[w];
            for (;;) {
                const uint32_t idx = tail + lane;
                bool ok = false;
                if (idx < len) {
                    uint32_t id = a.fifo[a.rpos[r0 + idx]];
                    id = id < n ? id : 0u;
                    ok = a.arrival[id] <= t;
                }
                const uint64_t b = __ballot(ok);
                const uint32_t c = ~b ? (uint32_t)__ffsll((unsigned long long)~b) - 1u : 64u;
                tail += c;
                if (c < 64u) break;
            }
            if (lane == 0) s_tail[w] = tail;
        }
        if (tid < kMaxQ) s_d[tid] = 0;
        __syncthreads();
        if (tid < kMaxQ) s_cnt[tid] = tid < nq ? s_tail[tid] - s_head[tid] : 0u;
        __syncthreads();
        uint32_t P = 0;
        for (uint32_t q = 0; q < nq; q++) P += s_cnt[q];
        const uint32_t m = P < batch ? P : batch;
        if (m == 0) continue;   // uniform

        // 2. candidates: the first min(m, pending) requests of each tier
        const bool ranked = policy == kFifo || policy == kPriority || policy == kAging;
        for (uint32_t p = tid; p < nq * batch; p += kTPB) {
            const uint32_t q = p / batch, r = p - q * batch;
            const uint32_t cq = s_cnt[q] < m ? s_cnt[q] : m;
            if (r >= cq) continue;
            const uint32_t j = a.rpos[a.rstart[q] + s_head[q] + r];
            uint32_t id = a.fifo[j];
            id = id < n ? id : 0u;
            if (ranked) {
                uint64_t K;
                if (policy == kFifo) {
                    K = 0;
                } else if (policy == kPriority) {
                    K = a.val[id];
                } else {
                    const Aux x = a.aux[id];
                    double wt = t - x.a;
                    if (wt < 0.0) wt = 0.0;
                    const double d = a.aging_rate * wt;
                    double e = x.b - d;
                    if (e < a.aging_floor) e = a.aging_floor;
                    K = ordered_bits(e);
                }
                a.cand_k[p] = K;
                a.cand_j[p] = j;
            } else if (a.wrr_mode != kWrrSmooth) {
                const uint64_t pos = a.wrr_mode == kWrrStride
                                         ? wrr_stride_pos(q, r, s_wt, nq, [&](uint32_t u) { return s_cnt[u]; })
                                         : wrr_place(q, r, s_cnt, s_wt, nq);
                if (pos < m) {
                    s_sel[pos] = id;
                    atomicAdd(&s_d[q], 1u);
                }
            }
            a.cand_i[p] = id;
        }
        __syncthreads();
        if (ranked) {
            // rank of each candidate: its place in its tier plus, in every
            // other tier, the candidates with a smaller (key, FIFO position)
            for (uint32_t p = tid; p < nq * batch; p += kTPB) {
                const uint32_t q = p / batch, r = p - q * batch;
                const uint32_t cq = s_cnt[q] < m ? s_cnt[q] : m;
                if (r >= cq) continue;
                const uint64_t K = a.cand_k[p];
                const uint32_t J = a.cand_j[p];
                uint32_t rank = r;
                for (uint32_t u = 0; u < nq && rank < m; u++) {
                    if (u == q) continue;
                    const uint32_t cu = s_cnt[u] < m ? s_cnt[u] : m;
                    uint32_t lo = 0, hi = cu;
                    while (lo < hi) {
                        const uint32_t mid = (lo + hi) >> 1;
                        const uint64_t K2 = a.cand_k[u * batch + mid];
                        const uint32_t J2 = a.cand_j[u * batch + mid];
                        if (K2 < K || (K2 == K && J2 < J)) lo = mid + 1u;
                        else hi = mid;
                    }
                    rank += lo;
                }
                if (rank < m) {
                    s_sel[rank] = a.cand_i[p];
                    atomicAdd(&s_d[q], 1u);
                }
            }
        } else if (a.wrr_mode == kWrrSmooth && w == 0) {
            // the first m dispatches of a fresh smooth cycle (lane q = tier q);
            // a queue running empty leaves and the others keep their credits
            const uint32_t len = lane < nq ? s_cnt[lane] : 0u;
            const uint32_t wq = lane < nq ? s_wt[lane] : 0u;
            uint32_t served = 0;
            int32_t credit = 0;
            uint32_t W = wave_sum(len ? wq : 0u);
            for (uint32_t pos = 0; pos < m; pos++) {
                const int b = wrr_pick(credit, served < len, wq, W);
                const bool mine = lane == (uint32_t)b;
                if (mine) s_sel[pos] = a.cand_i[lane * batch + served];   // served < m
                served += mine ? 1u : 0u;
                if (__ballot(mine && served == len) != 0ull) W = wave_sum(served < len ? wq : 0u);
            }
            if (lane < kMaxQ) s_d[lane] = served;
        }
        __syncthreads();

        // 3. dispatch, and the completion events of the batch
        if (tid < m) {
            const uint32_t id = s_sel[tid];
            if (total + tid < n) a.seq[total + tid] = id;
            a.tick_of[id] = (int32_t)k;
            s_evg[tid] = a.group[id];
            s_evx[tid] = a.est_base[id];
            s_evo[tid] = a.observed[id];
        }
        __syncthreads();

        // 4. Eq. (5) with the ratio of Eq. (6), each group's events of the
        //    batch in dispatch order
        if (tid < m) {
            const uint32_t g = s_evg[tid];
            bool lead = g < a.n_groups;
            for (uint32_t r = 0; r < tid && lead; r++) lead = s_evg[r] != g;
            if (lead) {
                double c = a.state[g];
                for (uint32_t r = tid; r < m; r++) {
                    if (s_evg[r] != g) continue;
                    const double x = s_evx[r];
                    if (!(isfinite(x) && x > 0.0)) continue;
                    const double ratio = (double)s_evo[r] / x;
                    const double t1 = oma * c;
                    const double t2 = a.alpha * ratio;
                    c = t1 + t2;
                }
                a.state[g] = c;
            }
        }
        if (tid < nq) s_head[tid] += s_d[tid];
        total += m;
        __syncthreads();
    }
    if (tid == 0) a.n_dispatched[0] = total;
}

// One workgroup per run: the queue engine where the run has its tier runs,
// else (SJF) the list engine.
__global__ __launch_bounds__(kTPB) void k_sim_engine(EngineBatch eb)
{
    const EngineArgs &a = eb.r[blockIdx.x];
    if (a.rpos) engine_queues(a);
    else engine_list(a);
}

__global__ void k_sim_empty(uint32_t *__restrict__ n_dispatched, uint32_t n_runs)
{
    if (threadIdx.x < n_runs) n_dispatched[threadIdx.x] = 0;
}

__global__ void k_sim_validate(const SimArgs a, uint32_t *__restrict__ flag)
{
    uint32_t bad = 0;
    const uint32_t stride = gridDim.x * blockDim.x;
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < a.n; i += stride) {
        if (a.tier[i] >= a.n_tiers || isnan(a.arrival[i]) || a.category[i] >= a.n_cat ||
            a.tenant[i] >= a.n_tenants || a.group[i] >= a.n_groups)
            bad = 1;
    }
    for (uint32_t k = blockIdx.x * blockDim.x + threadIdx.x; k < a.n_ticks; k += stride) {
        if (isnan(a.tick_t[k])) bad = 1;
        if (k + 1 < a.n_ticks && !(a.tick_t[k] <= a.tick_t[k + 1])) bad = 1;
    }
    if (bad) atomicOr(flag, 1u);
}

uint32_t grid_for(uint64_t n)
{
    const uint64_t b = cdiv(n, 256);
    return (uint32_t)(b < 1 ? 1 : (b > 1024 ? 1024 : b));
}

}  // namespace

constexpr uint64_t kCandBytes = (uint64_t)kMaxQ * kSimMaxBatch * (8 + 4 + 4);

size_t sim_ws_bytes(uint64_t n, uint32_t n_runs)
{
    // shared: fifo, the tier runs (positions and starts), then the FIFO sort
    // and the partition (one after the other); per run: list x2, est_base,
    // key, aux, val, the queue engine's candidates
    const uint64_t per = 2 * align_up(n * 4, 256) + 2 * align_up(n * 8, 256) +
                         align_up(n * sizeof(Aux), 256) + align_up(n, 256) + kCandBytes;
    const uint64_t sort = sort_ws_bytes(n, 1), part = am_partition_ws_bytes(n);
    return 2 * align_up(n * 4, 256) + 256 + (uint64_t)(n_runs ? n_runs : 1) * per + (sort > part ? sort : part);
}

hipError_t sim_launch(const SimArgs *runs, uint32_t n_runs, void *ws, uint32_t *flag, hipStream_t s,
                      WaitCfg wait)
{
    if (n_runs < 1 || n_runs > kSimMaxRuns) return hipErrorInvalidValue;
    const SimArgs &a0 = runs[0];
    const uint32_t n = a0.n;
    if (flag) {
        // the shared inputs, against the smallest tier count of the runs
        SimArgs v = a0;
        for (uint32_t r = 1; r < n_runs; r++) v.n_tiers = runs[r].n_tiers < v.n_tiers ? runs[r].n_tiers : v.n_tiers;
        hipLaunchKernelGGL(k_sim_validate, dim3(grid_for(n > v.n_ticks ? n : v.n_ticks)), dim3(256),
                           0, s, v, flag);
        return hipGetLastError();
    }
    if (n == 0) {
        // the runs' counters are one array (n_dispatched of run r = runs[0].n_dispatched + r)
        hipLaunchKernelGGL(k_sim_empty, dim3(1), dim3(64), 0, s, a0.n_dispatched, n_runs);
        return hipGetLastError();
    }
    uint8_t *p = static_cast<uint8_t *>(ws);
    auto take = [&](uint64_t bytes) {
        uint8_t *q = p;
        p += align_up(bytes, 256);
        return q;
    };
    uint32_t *fifo = reinterpret_cast<uint32_t *>(take((uint64_t)n * 4));
    uint32_t *rpos = reinterpret_cast<uint32_t *>(take((uint64_t)n * 4));
    uint32_t *rstart = reinterpret_cast<uint32_t *>(take(256));
    // every policy but SJF runs on the tier queues (up to the partition's limit)
    bool any_queues = false;
    for (uint32_t r = 0; r < n_runs; r++) any_queues = any_queues || (runs[r].policy != kSjf && n <= kAmMaxN);
    SetupBatch sb;
    EngineBatch eb;
    memset(&sb, 0, sizeof(sb));
    memset(&eb, 0, sizeof(eb));
    for (uint32_t r = 0; r < n_runs; r++) {
        const SimArgs &a = runs[r];
        uint32_t *list0 = reinterpret_cast<uint32_t *>(take((uint64_t)n * 4));
        uint32_t *list1 = reinterpret_cast<uint32_t *>(take((uint64_t)n * 4));
        double *est_base = reinterpret_cast<double *>(take((uint64_t)n * 8));
        uint64_t *key = reinterpret_cast<uint64_t *>(take((uint64_t)n * 8));
        Aux *aux = reinterpret_cast<Aux *>(take((uint64_t)n * sizeof(Aux)));
        uint8_t *val = take(n);
        uint8_t *cand = take(kCandBytes);

        SetupArgs &su = sb.r[r];
        su.n = n;
        su.policy = a.policy;
        su.n_cat = a.n_cat;
        su.n_tenants = a.n_tenants;
        su.n_tiers = a.n_tiers;
        su.counts = a.counts;
        su.tenant = a.tenant;
        su.category = a.category;
        su.tier = a.tier;
        su.t_base = a.t_base;
        su.s_tenant = a.s_tenant;
        su.arrival = a.arrival;
        su.f_ref = a.f_ref;
        // priority classes: rank of each tier's priority among the distinct values
        for (uint32_t q = 0; q < kMaxQ; q++) {
            su.prio[q] = a.prio[q];
            uint32_t c = 0;
            if (q < a.n_tiers)
                for (uint32_t u = 0; u < a.n_tiers; u++) {
                    bool first = true;   // count each distinct smaller value once
                    for (uint32_t v = 0; v < u; v++) first = first && a.prio[v] != a.prio[u];
                    if (first && a.prio[u] < a.prio[q]) c++;
                }
            su.cls[q] = c;
        }
        su.est_base = est_base;
        su.aux = aux;
        su.val = val;
        su.seq = a.seq;
        su.tick_of = a.tick_of;
        su.wait_status = r == 0 && wait.clear ? wait.status : nullptr;

        EngineArgs &ea = eb.r[r];
        ea.n = n;
        ea.n_groups = a.n_groups;
        ea.policy = a.policy;
        ea.batch = a.batch;
        ea.n_ticks = a.n_ticks;
        ea.n_q = a.n_tiers;
        ea.tick_t = a.tick_t;
        ea.fifo = fifo;
        ea.arrival = a.arrival;
        ea.group = a.group;
        ea.observed = a.observed;
        ea.est_base = est_base;
        ea.aux = aux;
        ea.val = val;
        for (uint32_t q = 0; q < kMaxQ; q++) ea.weight[q] = q < a.n_tiers && a.weight[q] ? a.weight[q] : 1u;
        ea.wrr_mode = a.wrr_mode;
        ea.alpha = a.alpha;
        ea.aging_rate = a.aging_rate;
        ea.aging_floor = a.aging_floor;
        ea.state = a.state;
        ea.list[0] = list0;
        ea.list[1] = list1;
        ea.key = key;
        ea.seq = a.seq;
        ea.tick_of = a.tick_of;
        ea.n_dispatched = a.n_dispatched;
        if (a.policy != kSjf && n <= kAmMaxN) {
            ea.rpos = rpos;
            ea.rstart = rstart;
            ea.cand_k = reinterpret_cast<uint64_t *>(cand);
            ea.cand_j = reinterpret_cast<uint32_t *>(cand + (uint64_t)kMaxQ * kSimMaxBatch * 8);
            ea.cand_i = reinterpret_cast<uint32_t *>(cand + (uint64_t)kMaxQ * kSimMaxBatch * 12);
        }
    }
    void *sort_ws = p;
    hipLaunchKernelGGL(k_sim_setup, dim3(grid_for(n), n_runs), dim3(256), 0, s, sb);

    SortInput in = {};
    in.n = n;
    in.arrival = a0.arrival;
    in.wait = wait;
    in.wait.clear = false;
    SortJob job = {SortKind::Fifo, 64, nullptr, fifo};
    hipError_t e = sort_launch(in, &job, 1, sort_ws, s);
    if (e != hipSuccess) return e;
    if (any_queues) {
        // the FIFO sequence split by tier, each tier in FIFO order (the sort's
        // workspace is free again on the stream)
        SortInput pin = {};
        pin.n = n;
        pin.fifo = fifo;
        pin.tier = a0.tier;
        pin.arrival = a0.arrival;
        for (uint32_t q = 0; q < kMaxQ; q++) pin.cls[q] = q;
        e = am_partition(pin, rpos, rstart, sort_ws, s);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(k_sim_engine, dim3(n_runs), dim3(kTPB), 0, s, eb);
    return hipGetLastError();
}

}  // namespace ds
