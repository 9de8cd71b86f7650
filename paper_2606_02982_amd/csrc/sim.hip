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

#include <memory>
#include <new>

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
    const uint32_t *qid;       // request, arrival, group, observed length and
    const double *qarr;        // B-free estimate of each run entry
    const uint32_t *qgrp, *qobs;
    const double *qest;
    double prio[kMaxQ];        // each tier's priority (Priority and Aging keys)
    uint64_t *cand_k;
    uint32_t *cand_j, *cand_i;
    // the class engine (SJF): each class's head bound, the pending bitmap over
    // the class lists, rebuild keys
    uint32_t *cls_head;
    uint64_t *cls_elig, *cls_kk;
    uint32_t *cls_kj;
    double f_ref;
};

// Several runs share one launch: run r is block r of the engine. Their
// arguments go by value, kSimChunk runs per kernel argument block: the
// set-up runs chunk by chunk (block row = run of the chunk); an engine
// launch of at most kSimChunk runs takes them directly, a larger one from
// the workspace, where a small kernel per chunk has copied them (kernel
// arguments are captured by value, so the launch stays capturable).
constexpr uint32_t kSimChunk = 8;
struct SetupBatch {
    SetupArgs r[kSimChunk];
};
struct EngineBatch {
    EngineArgs r[kSimChunk];
};
static_assert(sizeof(SetupBatch) <= 4096, "kernel arguments within 4 KB");

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

// LDS of the list engine.
struct ListLds {
    uint32_t s_w[kNW];
    uint32_t s_hist[256];
    uint32_t s_vw[kNW][kMaxQ];
    uint32_t s_cnt[kMaxQ];
    uint32_t s_wt[kMaxQ];
    uint32_t s_pick[4];
    uint64_t s_kmin[kNW], s_kmax[kNW];
    uint32_t s_selpos[kSimMaxBatch];
    uint64_t s_selK[kSimMaxBatch];
    uint32_t s_selJ[kSimMaxBatch];
    uint32_t s_evg[kSimMaxBatch], s_evo[kSimMaxBatch];
    double s_evx[kSimMaxBatch];
    // Priority/Weighted: list positions of the first `batch` pending requests
    // of each queue; SJF/Aging: the radix select's candidates
    union {
        uint32_t first[kMaxQ][kSimMaxBatch];
        struct {
            uint64_t k[kCand];
            uint32_t j[kCand];
        } cand;
    } s_big;
};

// The list engine from tick k0 on. A0 > 0: another engine ran the ticks
// before k0 (FIFO positions below A0 have arrived, total0 requests have been
// dispatched and carry their tick in tick_of); the pending list is rebuilt
// from those.
__device__ void engine_list(const EngineArgs &a, ListLds &L, uint32_t k0 = 0, uint32_t A0 = 0,
                            uint32_t total0 = 0)
{
    auto &s_w = L.s_w;
    auto &s_hist = L.s_hist;
    auto &s_vw = L.s_vw;
    auto &s_cnt = L.s_cnt;
    auto &s_wt = L.s_wt;
    auto &s_pick = L.s_pick;
    auto &s_kmin = L.s_kmin;
    auto &s_kmax = L.s_kmax;
    auto &s_selpos = L.s_selpos;
    auto &s_selK = L.s_selK;
    auto &s_selJ = L.s_selJ;
    auto &s_evg = L.s_evg;
    auto &s_evo = L.s_evo;
    auto &s_evx = L.s_evx;
    auto &s_big = L.s_big;

    const uint32_t tid = threadIdx.x, lane = (uint32_t)lane_id(), w = tid >> 6;
    const uint32_t n = a.n, policy = a.policy, batch = a.batch, nq = a.n_q;
    const bool keyed = policy == kSjf || policy == kAging;
    const bool queued = policy == kPriority || policy == kWeighted;
    const double oma = 1.0 - a.alpha;
    const double nan = __builtin_nan("");
    if (tid < kMaxQ) s_wt[tid] = a.weight[tid];

    uint32_t cur = 0;          // list buffer holding the pending list
    uint32_t P = 0;            // its entries (pending + last tick's dispatches)
    uint32_t A = A0;           // FIFO positions appended so far
    uint32_t total = total0;   // requests dispatched so far
    // resumed: the arrived requests not yet dispatched, in FIFO order
    for (uint32_t c0 = 0; c0 < A0; c0 += kTPB) {
        const uint32_t j = c0 + tid;
        uint32_t id = 0;
        bool keep = false;
        if (j < A0) {
            id = a.fifo[j];
            id = id < n ? id : 0u;
            keep = a.tick_of[id] < 0;
        }
        uint32_t tot;
        const uint32_t off = block_scan(keep ? 1u : 0u, s_w, tot);
        if (keep) a.list[0][P + off] = id;
        P += tot;
    }
    __syncthreads();
    for (uint32_t k = k0; k < a.n_ticks; k++) {
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

// Lanes below m whose g equals this lane's, matched bit by bit with ballots
// over the bits a group below n_groups can have (a lane at or past m, or
// with g >= n_groups, is its own class of one: its result is not used).
__device__ __forceinline__ uint64_t same_group_lanes(uint32_t g, uint32_t m, uint32_t n_groups)
{
    const int bits = n_groups > 1 ? 32 - __clz((int)(n_groups - 1)) : 1;
    const uint64_t active = m >= 64 ? ~0ull : (1ull << m) - 1ull;
    uint64_t same = active;
    for (int b = 0; b < bits; b++) {
        const bool one = (g >> b) & 1u;
        const uint64_t mk = __ballot(one);
        same &= one ? mk : ~mk;
    }
    // lanes whose g has higher bits set match only lanes with the same g
    // above the compared bits; a lane below n_groups has none of those
    const bool high = bits < 32 && (g >> bits) != 0u;
    const uint64_t hk = __ballot(high);
    return high ? (same & hk & (1ull << (uint32_t)lane_id())) : (same & ~hk);
}

// Batches up to kQLdsBatch with up to kQLdsGroups groups keep the queue
// engine's candidates, their completion events and the factors in LDS;
// other runs use the workspace and the state array.
constexpr uint32_t kQLdsBatch = 128;
constexpr uint32_t kQLdsGroups = 4096;
constexpr uint32_t kNoGroup = 0xFFFFFFFFu;
constexpr uint32_t kQCand = kMaxQ * kQLdsBatch;

struct QueueLds {
    uint32_t s_head[kMaxQ], s_tail[kMaxQ], s_cnt[kMaxQ], s_d[kMaxQ], s_wt[kMaxQ], s_rstart[kMaxQ + 1];
    double sst[kQLdsGroups];         // the factors during the run
    uint32_t s_sel[kSimMaxBatch];    // candidate of each dispatch place
    uint32_t s_evg[kSimMaxBatch], s_evo[kSimMaxBatch];
    double s_evx[kSimMaxBatch];
    uint64_t ck[kQCand];             // candidates: key, FIFO position, request, and its
    uint32_t cj[kQCand], ci[kQCand], cg[kQCand], co[kQCand];   // event: group, observed
    double cx[kQCand];                                          // length, B-free estimate
};

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
//
// Every key follows from the tier and the arrival (Priority: the tier's
// priority; Aging: it aged to t), so a candidate needs only its run entry's
// request, arrival, group, observed length and B-free estimate, laid out in
// run order once (one round of loads). In LDS mode (kL) the candidates and
// the factors stay in LDS (the factors are written back at the end), the
// phases are separated by LDS-only barriers, and each batch's factor
// updates run on one wave (lane i: the i-th event).
template <bool kL>
__device__ void engine_queues(const EngineArgs &a, QueueLds &Q)
{
    auto &s_head = Q.s_head;
    auto &s_tail = Q.s_tail;
    auto &s_cnt = Q.s_cnt;
    auto &s_d = Q.s_d;
    auto &s_wt = Q.s_wt;
    auto &s_sel = Q.s_sel;
    auto &s_evg = Q.s_evg;
    auto &s_evo = Q.s_evo;
    auto &s_evx = Q.s_evx;
    uint64_t *ck = kL ? Q.ck : a.cand_k;
    uint32_t *cj = kL ? Q.cj : a.cand_j;
    uint32_t *ci = kL ? Q.ci : a.cand_i;
    auto sync = [] {
        if (kL) lds_sync();
        else __syncthreads();
    };
    const uint32_t tid = threadIdx.x, lane = (uint32_t)lane_id(), w = tid >> 6;
    const uint32_t n = a.n, policy = a.policy, batch = a.batch, nq = a.n_q;
    const double oma = 1.0 - a.alpha;
    if (tid < kMaxQ) {
        s_head[tid] = 0;
        s_tail[tid] = 0;
        s_wt[tid] = a.weight[tid];
    }
    if (tid <= kMaxQ) Q.s_rstart[tid] = a.rstart[tid];
    if (kL)
        for (uint32_t g = tid; g < a.n_groups; g += kTPB) Q.sst[g] = a.state[g];
    uint32_t total = 0;
    __syncthreads();
    for (uint32_t k = 0; k < a.n_ticks; k++) {
        const double t = a.tick_t[k];
        if (!kL) __syncthreads();   // the last tick's factor updates, for every wave
        // 1. arrivals: wave q moves tier q's tail over its requests with
        //    arrival <= t (a prefix of the rest of its FIFO run)
        if (w < nq) {
            const uint32_t r0 = Q.s_rstart[w], len = Q.s_rstart[w + 1] - r0;
            uint32_t tail = s_tail[w];
            for (;;) {
                const uint32_t idx = tail + lane;
                const bool ok = idx < len && a.qarr[r0 + idx] <= t;
                const uint64_t b = __ballot(ok);
                const uint32_t c = ~b ? (uint32_t)__ffsll((unsigned long long)~b) - 1u : 64u;
                tail += c;
                if (c < 64u) break;
            }
            if (lane == 0) s_tail[w] = tail;
        }
        if (tid < kMaxQ) s_d[tid] = 0;
        sync();
        if (tid < kMaxQ) s_cnt[tid] = tid < nq ? s_tail[tid] - s_head[tid] : 0u;
        sync();
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
            const uint32_t x = Q.s_rstart[q] + s_head[q] + r;
            const uint32_t j = a.rpos[x];
            uint32_t id = a.qid[x];
            id = id < n ? id : 0u;
            if (ranked) {
                uint64_t K = 0;
                if (policy == kPriority) {
                    K = ordered_bits(a.prio[q]);
                } else if (policy == kAging) {
                    double wt = t - a.qarr[x];
                    if (wt < 0.0) wt = 0.0;
                    const double d = a.aging_rate * wt;
                    double e = a.prio[q] - d;
                    if (e < a.aging_floor) e = a.aging_floor;
                    K = ordered_bits(e);
                }
                ck[p] = K;
                cj[p] = j;
            } else if (a.wrr_mode != kWrrSmooth) {
                const uint64_t pos = a.wrr_mode == kWrrStride
                                         ? wrr_stride_pos(q, r, s_wt, nq, [&](uint32_t u) { return s_cnt[u]; })
                                         : wrr_place(q, r, s_cnt, s_wt, nq);
                if (pos < m) {
                    s_sel[pos] = p;
                    atomicAdd(&s_d[q], 1u);
                }
            }
            ci[p] = id;
            if (kL) {
                Q.cg[p] = a.qgrp[x];
                Q.cx[p] = a.qest[x];
                Q.co[p] = a.qobs[x];
            }
        }
        sync();
        if (ranked) {
            // rank of each candidate: its place in its tier plus, in every
            // other tier, the candidates with a smaller (key, FIFO position)
            for (uint32_t p = tid; p < nq * batch; p += kTPB) {
                const uint32_t q = p / batch, r = p - q * batch;
                const uint32_t cq = s_cnt[q] < m ? s_cnt[q] : m;
                if (r >= cq) continue;
                const uint64_t K = ck[p];
                const uint32_t J = cj[p];
                uint32_t rank = r;
                for (uint32_t u = 0; u < nq && rank < m; u++) {
                    if (u == q) continue;
                    const uint32_t cu = s_cnt[u] < m ? s_cnt[u] : m;
                    uint32_t lo = 0, hi = cu;
                    while (lo < hi) {
                        const uint32_t mid = (lo + hi) >> 1;
                        const uint64_t K2 = ck[u * batch + mid];
                        const uint32_t J2 = cj[u * batch + mid];
                        if (K2 < K || (K2 == K && J2 < J)) lo = mid + 1;
                        else hi = mid;
                    }
                    rank += lo;
                }
                if (rank < m) {
                    s_sel[rank] = p;
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
                if (mine) s_sel[pos] = lane * batch + served;   // served < m
                served += mine ? 1u : 0u;
                if (__ballot(mine && served == len) != 0ull) W = wave_sum(served < len ? wq : 0u);
            }
            if (lane < kMaxQ) s_d[lane] = served;
        }
        sync();

        // 3. dispatch, and the completion events of the batch (in LDS mode
        //    from wave 1 on: the global stores stay in flight on waves other
        //    than the one that runs the factor updates next)
        const uint32_t d = kL ? tid - 64 : tid;
        if ((!kL || tid >= 64) && d < m) {
            const uint32_t p = s_sel[d], id = ci[p];
            if (total + d < n) a.seq[total + d] = id;
            a.tick_of[id] = (int32_t)k;
            if (kL) {
                s_evg[d] = Q.cg[p];
                s_evx[d] = Q.cx[p];
                s_evo[d] = Q.co[p];
            } else {
                s_evg[d] = a.group[id];
                s_evx[d] = a.est_base[id];
                s_evo[d] = a.observed[id];
            }
        }
        sync();

        // 4. Eq. (5) with the ratio of Eq. (6), each group's events of the
        //    batch in dispatch order
        auto step = [&](double c, uint32_t r) {
            const double x = s_evx[r];
            if (!(isfinite(x) && x > 0.0)) return c;
            const double ratio = (double)s_evo[r] / x;
            const double t1 = oma * c;
            const double t2 = a.alpha * ratio;
            return t1 + t2;
        };
        if (kL && m <= 64) {
            if (w == 0) {
                const uint32_t g = lane < m ? s_evg[lane] : kNoGroup;
                const uint64_t same = same_group_lanes(g, m, a.n_groups);
                if (lane < m && g < a.n_groups && (same & lanemask_lt()) == 0) {
                    double c = Q.sst[g];
                    for (uint64_t bits = same; bits; bits &= bits - 1ull)
                        c = step(c, (uint32_t)__ffsll((unsigned long long)bits) - 1u);
                    Q.sst[g] = c;
                }
            }
        } else if (tid < m) {
            const uint32_t g = s_evg[tid];
            bool lead = g < a.n_groups;
            for (uint32_t r = 0; r < tid && lead; r++) lead = s_evg[r] != g;
            if (lead) {
                double c = kL ? Q.sst[g] : a.state[g];
                for (uint32_t r = tid; r < m; r++)
                    if (s_evg[r] == g) c = step(c, r);
                if (kL) Q.sst[g] = c;
                else a.state[g] = c;
            }
        }
        if (tid < nq) s_head[tid] += s_d[tid];
        total += m;
        sync();
    }
    if (kL)
        for (uint32_t g = tid; g < a.n_groups; g += kTPB) a.state[g] = Q.sst[g];
    if (tid == 0) a.n_dispatched[0] = total;
}

// ---- SJF on class lists ---------------------------------------------------------
//
// A class is the set of requests that share category, tenant and group.
// Within a class T_base, S_tenant and the factor B are common, so the budget
// of Eq. (1) with the estimate of Eq. (2), words + ((T_base B) S_tenant) F,
// is a strictly increasing function of the word count while E = (T_base B)
// S_tenant is finite and non-negative and the class's budgets stay at or
// below 2^50: F = 1 + words / f_ref is non-decreasing for f_ref > 0, every
// rounding step is monotone, and below 2^50 the rounded sum still moves
// with each extra word. The class's part of the SJF order (budget, FIFO
// position) is then its (words, FIFO position) order whatever the factors
// do. So every class is sorted once, the pending requests are bits of a
// bitmap over the class lists, and a class's key is the (budget, FIFO
// position) of its first pending member, its head. A tick:
//   * arrivals set their bits and pull their class's head back;
//   * the classes touched since the last tick (arrivals, the last batch's
//     dispatches, every class of a group whose factor the batch moved) get
//     their keys recomputed;
//   * a pool in LDS, sorted by key, holds every class whose key is at most
//     tau, at most kPool of them; every other class's key is above tau (or
//     it has no pending member). A touched class at or below tau enters, one
//     above it leaves; past kPool entries tau drops to the last one kept.
//     Should fewer than m pool classes remain (tau finite), every key is
//     recomputed and the kPool smallest are chosen by a radix select;
//   * the first m = min(batch, pending) requests of the order are in the
//     windows of the m best classes of the pool: the class of rank r holds at
//     most m - r of them (the r better heads come before all its members) and
//     none after the m-th best head. The windows come from the bitmap, their
//     budgets from the current factors; the candidates are sorted and the
//     first m dispatched.
// Every key computation checks the conditions above; if one fails, the run
// goes on from that tick with the list engine, so the result is the same.

constexpr uint32_t kClsMaxBatch = 32;   // larger batches: the list engine
constexpr uint32_t kPool = 512;          // pool classes kept after a tick
constexpr uint32_t kHash = 2048;         // touched-class set (open addressing)
constexpr uint32_t kDirtyMax = 1024;     // touched classes per tick before a rebuild
constexpr uint32_t kWin = kClsMaxBatch * kClsMaxBatch;   // window slots
constexpr uint32_t kNone = 0xFFFFFFFFu;
constexpr double kBudgetTop = 0x1p50;
static_assert(kWin == kTPB && kDirtyMax == kTPB && kPool < kTPB, "a thread per slot, entry and pool class");

// The class structure of a launch's requests, shared by its SJF runs.
struct ClassShared {
    const uint32_t *ctl;             // [0]: classes C; [1]: non-zero if an input is out of range
    const uint32_t *clist;           // request ids by (class, words, FIFO position)
    const uint32_t *lw, *lf, *lobs;  // words, FIFO position, observed length of each list entry
    const uint32_t *pos_f, *cls_f;   // list position and class of each FIFO position
    const double *arr_f;             // arrival of each FIFO position
    const uint32_t *cstart;          // first list position of each class, then n
    const double *ctb, *cs;          // T_base and S_tenant of each class
    const uint32_t *cg;              // group of each class (non-decreasing)
    const uint32_t *gfirst, *gend;   // the classes of that group
};

// Class entries are (key, FIFO position of the head, list position of the
// head, class); keys are the budget bits.
struct ClassLds {
    uint64_t pk[2][kPool];           // the pool, sorted, in one half at a time
    uint32_t pj[2][kPool], ph[2][kPool], pc[2][kPool];
    uint32_t pdrop[kPool + 1];       // pool entries leaving before each index
    uint64_t ek[kDirtyMax];          // the tick's entering classes, unsorted
    uint32_t ej[kDirtyMax], eh[kDirtyMax], ec[kDirtyMax];
    union {
        struct {                     // the entering classes, sorted
            uint64_t k[kDirtyMax];
            uint32_t j[kDirtyMax], h[kDirtyMax], c[kDirtyMax];
        } e;
        struct {                     // window candidates
            uint64_t k[kWin];
            double t2[kWin];         // alpha x its Eq. (6) ratio, if usable
            uint32_t j[kWin], id[kWin], use[kWin], slot[kWin];
        } w;
    } u;
    uint32_t sel[kClsMaxBatch];      // the candidate of each dispatch place
    uint32_t wpos[kClsMaxBatch][kClsMaxBatch];   // window of rank r: list positions
    uint32_t wn[kClsMaxBatch], sc[kClsMaxBatch], sg[kClsMaxBatch], sgf[kClsMaxBatch], sge[kClsMaxBatch],
        last[kClsMaxBatch];
    double sB[kClsMaxBatch];         // the factor of each window's group
    uint32_t hash[kHash], dirty[kDirtyMax];
    uint32_t cnt[4];                 // touched classes, overflow, entering classes, candidates
    uint32_t fail;
    uint32_t hist[256], w[kNW], pick[4];
    uint32_t evg[kClsMaxBatch], evo[kClsMaxBatch], evr[kClsMaxBatch];   // evo: usable
    double evx[kClsMaxBatch];                                           // alpha x ratio
    uint32_t rg0[kClsMaxBatch], rlen[kClsMaxBatch];   // classes touched by the factor updates
};

struct Resume {
    uint32_t k, A, total;
};

__device__ __forceinline__ bool pair_lt(uint64_t k1, uint32_t j1, uint64_t k2, uint32_t j2)
{
    return k1 < k2 || (k1 == k2 && j1 < j2);
}

__device__ __forceinline__ uint64_t ld_relaxed64(const uint64_t *p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Ascending bitonic sort of N (a power of two, at most 2 kTPB) pairs with two
// payloads, in LDS, by the whole block.
__device__ void bitonic(uint64_t *k, uint32_t *j, uint32_t *v, uint32_t *u, uint32_t N)
{
    const uint32_t t = threadIdx.x;
    for (uint32_t size = 2; size <= N; size <<= 1) {
        for (uint32_t stride = size >> 1; stride > 0; stride >>= 1) {
            __syncthreads();
            if (t < (N >> 1)) {
                const uint32_t lo = ((t & ~(stride - 1)) << 1) | (t & (stride - 1)), hi = lo + stride;
                const uint64_t k1 = k[lo], k2 = k[hi];
                const uint32_t j1 = j[lo], j2 = j[hi];
                if (pair_lt(k2, j2, k1, j1) == ((lo & size) == 0)) {
                    k[lo] = k2;
                    k[hi] = k1;
                    j[lo] = j2;
                    j[hi] = j1;
                    const uint32_t v1 = v[lo], u1 = u[lo];
                    v[lo] = v[hi];
                    v[hi] = v1;
                    u[lo] = u[hi];
                    u[hi] = u1;
                }
            }
        }
    }
    __syncthreads();
}

// Adds class c to the touched set. Callers check the count before each
// insertion, so with at most kTPB threads inserting at once the table never
// fills; past kDirtyMax members the set overflows (the next tick rebuilds).
__device__ void mark_dirty(uint32_t c, ClassLds &S)
{
    if (*(volatile uint32_t *)&S.cnt[0] >= kDirtyMax) {
        S.cnt[1] = 1;
        return;
    }
    uint32_t h = (c * 0x9E3779B1u) >> 21;
    for (;;) {
        const uint32_t old = atomicCAS(&S.hash[h], kNone, c);
        if (old == kNone) {
            const uint32_t i = atomicAdd(&S.cnt[0], 1u);
            if (i < kDirtyMax) S.dirty[i] = c;
            else S.cnt[1] = 1;
            return;
        }
        if (old == c) return;
        h = (h + 1) & (kHash - 1);
    }
}

__device__ __forceinline__ bool is_dirty(uint32_t c, const ClassLds &S)
{
    uint32_t h = (c * 0x9E3779B1u) >> 21;
    for (;;) {
        const uint32_t x = S.hash[h];
        if (x == c) return true;
        if (x == kNone) return false;
        h = (h + 1) & (kHash - 1);
    }
}

// Key of class c: (budget bits, FIFO position) of its first pending member
// and that member's list position H, all ones if it has none; the class's
// head moves up to that member. ok turns false if the class breaks the
// conditions of its static order.
__device__ void class_key(const EngineArgs &a, const ClassShared &cs, uint32_t c, uint64_t &K, uint32_t &J,
                          uint32_t &H, bool &ok)
{
    const uint32_t b0 = cs.cstart[c], e = cs.cstart[c + 1];
    const double tb = cs.ctb[c], s = cs.cs[c];
    const double B = a.state[cs.cg[c]];
    const uint32_t h0 = ld_relaxed(&a.cls_head[c]);
    const double wmax = (double)cs.lw[e > b0 ? e - 1 : b0];
    uint32_t p = e;
    if (h0 < e) {
        uint32_t wi = h0 >> 6;
        uint64_t bits = ld_relaxed64(&a.cls_elig[wi]) & (~0ull << (h0 & 63u));
        for (;;) {
            if (bits) {
                p = wi * 64u + (uint32_t)__ffsll((unsigned long long)bits) - 1u;
                break;
            }
            wi++;
            if ((uint64_t)wi * 64u >= e) break;
            bits = ld_relaxed64(&a.cls_elig[wi]);
        }
        if (p > e) p = e;
        if (p != h0) st_relaxed(&a.cls_head[c], p);
    }
    double E = tb * B;
    E = E * s;
    double top = E * (1.0 + wmax / a.f_ref);
    top = wmax + top;
    if (!(E >= 0.0 && top <= kBudgetTop)) ok = false;
    H = p;
    if (p >= e) {
        K = ~0ull;
        J = kNone;
        return;
    }
    const double wd = (double)cs.lw[p];
    double b = E * (1.0 + wd / a.f_ref);
    b = wd + b;
    K = ordered_bits(b);
    J = cs.lf[p];
}

// (TK, TJ) with exactly `need` of the C pairs (kk, kj) at or below it, need
// at most the number of finite pairs: an MSD radix select over the 96-bit
// pair, a byte per pass, until the bucket of the need-th pair is exactly
// what remains to select.
__device__ void select_pairs(const uint64_t *kk, const uint32_t *kj, uint32_t C, uint32_t need, uint64_t &TK,
                             uint32_t &TJ, ClassLds &S)
{
    uint64_t mK = 0;
    uint32_t mJ = 0;
    TK = 0;
    TJ = 0;
    for (int d = 11; d >= 0; d--) {
        if (threadIdx.x < 256) S.hist[threadIdx.x] = 0;
        __syncthreads();
        for (uint32_t c = threadIdx.x; c < C; c += kTPB) {
            const uint64_t K = kk[c];
            const uint32_t J = kj[c];
            if ((K & mK) == TK && (J & mJ) == TJ) atomicAdd(&S.hist[pair_digit(K, J, d)], 1u);
        }
        __syncthreads();
        const uint32_t h = threadIdx.x < 256 ? S.hist[threadIdx.x] : 0u;
        uint32_t tot;
        const uint32_t ex = block_scan(h, S.w, tot);
        if (threadIdx.x < 256 && ex < need && need <= ex + h) {
            S.pick[0] = threadIdx.x;
            S.pick[1] = ex;
            S.pick[2] = h;
        }
        __syncthreads();
        const uint32_t b = S.pick[0], cb = S.pick[2];
        need -= S.pick[1];
        __syncthreads();
        if (d >= 4) {
            TK |= (uint64_t)b << (8 * (d - 4));
            mK |= 0xFFull << (8 * (d - 4));
        } else {
            TJ |= b << (8 * d);
            mJ |= 0xFFu << (8 * d);
        }
        if (cb == need) {
            // the whole bucket: up to its largest possible pair
            if (d >= 4) {
                TK |= (1ull << (8 * (d - 4))) - 1ull;
                TJ = kNone;
            } else {
                TJ |= (1u << (8 * d)) - 1u;
            }
            return;
        }
    }
}

// Entries of a sorted array (k, j) of length len below the pair (K, J).
__device__ __forceinline__ uint32_t count_below(const uint64_t *k, const uint32_t *j, uint32_t len, uint64_t K,
                                                uint32_t J)
{
    uint32_t lo = 0, hi = len;
    while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        if (pair_lt(k[mid], j[mid], K, J)) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

// block_scan with LDS barriers.
__device__ __forceinline__ uint32_t lds_scan(uint32_t x, uint32_t *s_w, uint32_t &total)
{
    const uint32_t inc = wave_incl_scan_dpp(x);
    const uint32_t w = threadIdx.x >> 6;
    if (lane_id() == 63) s_w[w] = inc;
    lds_sync();
    uint32_t off = 0, tot = 0;
#pragma unroll
    for (uint32_t k = 0; k < kNW; k++) {
        const uint32_t v = s_w[k];
        off += k < w ? v : 0u;
        tot += v;
    }
    lds_sync();
    total = tot;
    return off + inc - x;
}

// Pairs of (k, j)[0, len) below (K, J), counted by one wave (64 entries at a
// time, a ballot each); stops counting at `limit`.
__device__ __forceinline__ uint32_t rank_in(const uint64_t *k, const uint32_t *j, uint32_t len, uint64_t K,
                                            uint32_t J, uint32_t limit)
{
    uint32_t r = 0;
    for (uint32_t c0 = 0; c0 < len && r < limit; c0 += 64) {
        const uint32_t u = c0 + (uint32_t)lane_id();
        const bool below = u < len && pair_lt(k[u], j[u], K, J);
        r += (uint32_t)__popcll(__ballot(below));
    }
    return r;
}

// SJF ticks on the class lists. Returns where the list engine must take
// over (k = n_ticks: every tick done, n_dispatched written).
//
// Global memory between waves: the bitmap and the head bounds change by the
// arrivals' atomics, which come after a full barrier (the last tick's
// stores are done) and before another (the keys below see them); a key
// computation tightens its class's head bound with a plain store, done by
// the next tick's first barrier. A dispatch does not move head bounds (a
// bound below the first pending member stays valid); it touches the class.
__device__ Resume engine_class(const EngineArgs &a, const ClassShared &cs, ClassLds &S)
{
    const uint32_t tid = threadIdx.x, lane = (uint32_t)lane_id(), w = tid >> 6;
    const uint32_t n = a.n, batch = a.batch;
    const double oma = 1.0 - a.alpha;
    const uint32_t C = cs.ctl[0];
    if (cs.ctl[1] != 0 || C == 0) return Resume{0, 0, 0};
    for (uint32_t c = tid; c < C; c += kTPB) a.cls_head[c] = cs.cstart[c + 1];
    for (uint32_t i = tid; i < (n + 63u) / 64u; i += kTPB) a.cls_elig[i] = 0;
    for (uint32_t i = tid; i < kHash; i += kTPB) S.hash[i] = kNone;
    if (tid < 4) S.cnt[tid] = 0;
    if (tid == 0) S.fail = 0;
    bool ok = true;
    __syncthreads();
    for (uint32_t c = tid; c < C; c += kTPB) {
        uint64_t K;
        uint32_t J, H;
        class_key(a, cs, c, K, J, H, ok);   // every head is the class end: the checks alone
    }
    if (__syncthreads_or(!ok)) return Resume{0, 0, 0};

    uint32_t cur = 0, np = 0;                 // pool half and entries
    uint64_t tK = ~0ull;                      // tau (all ones: every class with a key is in the pool)
    uint32_t tJ = kNone;
    uint32_t A = 0, P = 0, total = 0;         // FIFO positions arrived, pending, dispatched
    for (uint32_t k = 0; k < a.n_ticks; k++) {
        const double t = a.tick_t[k];
        // 1. arrivals: a prefix of the rest of the FIFO order
        for (;;) {
            const uint32_t j = A + tid;
            bool arrived = false;
            uint32_t p = 0, cl = 0;
            if (j < n) {
                arrived = cs.arr_f[j] <= t;
                p = cs.pos_f[j];
                cl = cs.cls_f[j];
            }
            const uint32_t c = (uint32_t)__syncthreads_count(arrived);
            if (arrived) {
                atomicOr((unsigned long long *)&a.cls_elig[p >> 6], 1ull << (p & 63u));
                atomicMin(&a.cls_head[cl], p);
                mark_dirty(cl, S);
            }
            A += c;
            P += c;
            if (c < kTPB) break;
        }
        __syncthreads();
        const uint32_t m = P < batch ? P : batch;
        if (m == 0) continue;   // uniform; the touched set carries over

        // 2. keys of the touched classes; those at or below tau enter the
        //    pool, the pool's touched classes leave it
        bool rebuild = S.cnt[1] != 0;
        if (!rebuild) {
            if (tid < S.cnt[0]) {
                const uint32_t c = S.dirty[tid];
                uint64_t K;
                uint32_t J, H;
                class_key(a, cs, c, K, J, H, ok);
                if (K != ~0ull && !pair_lt(tK, tJ, K, J)) {
                    const uint32_t slot = atomicAdd(&S.cnt[2], 1u);
                    S.ek[slot] = K;
                    S.ej[slot] = J;
                    S.eh[slot] = H;
                    S.ec[slot] = c;
                }
            }
            const bool drop = tid < np && is_dirty(S.pc[cur][tid], S);
            uint32_t dropped;
            const uint32_t before = lds_scan(drop ? 1u : 0u, S.w, dropped);
            if (tid <= np) S.pdrop[tid] = before;
        }
        if (!ok) S.fail = 1;
        lds_sync();
        if (S.fail) return Resume{k, A, total};
        const uint32_t nin = S.cnt[2];
        // the touched set is consumed
        for (uint32_t i = tid; i < kHash; i += kTPB) S.hash[i] = kNone;
        if (!rebuild) {
            // the entering classes in order (ranked by counting), then merged
            // with the pool's remaining classes into the other half
            for (uint32_t i = w; i < nin; i += kNW) {
                const uint64_t K = S.ek[i];
                const uint32_t J = S.ej[i];
                const uint32_t r = rank_in(S.ek, S.ej, nin, K, J, ~0u);
                if (lane == 0) {
                    S.u.e.k[r] = K;
                    S.u.e.j[r] = J;
                    S.u.e.h[r] = S.eh[i];
                    S.u.e.c[r] = S.ec[i];
                }
            }
            lds_sync();
            const uint32_t nx = cur ^ 1u, stay = np - S.pdrop[np];
            if (tid < np && S.pdrop[tid + 1] == S.pdrop[tid]) {
                const uint64_t K = S.pk[cur][tid];
                const uint32_t J = S.pj[cur][tid];
                const uint32_t pos = tid - S.pdrop[tid] + count_below(S.u.e.k, S.u.e.j, nin, K, J);
                if (pos < kPool) {
                    S.pk[nx][pos] = K;
                    S.pj[nx][pos] = J;
                    S.ph[nx][pos] = S.ph[cur][tid];
                    S.pc[nx][pos] = S.pc[cur][tid];
                }
            }
            if (tid < nin) {
                const uint64_t K = S.u.e.k[tid];
                const uint32_t J = S.u.e.j[tid];
                const uint32_t lb = count_below(S.pk[cur], S.pj[cur], np, K, J);
                const uint32_t pos = tid + lb - S.pdrop[lb];
                if (pos < kPool) {
                    S.pk[nx][pos] = K;
                    S.pj[nx][pos] = J;
                    S.ph[nx][pos] = S.u.e.h[tid];
                    S.pc[nx][pos] = S.u.e.c[tid];
                }
            }
            lds_sync();
            cur = nx;
            np = stay + nin;
            if (np > kPool) {
                np = kPool;
                tK = S.pk[cur][kPool - 1];
                tJ = S.pj[cur][kPool - 1];
            }
            rebuild = np < m && tK != ~0ull;
        }
        if (tid < 4) S.cnt[tid] = 0;
        if (rebuild) {
            __syncthreads();
            uint32_t fin = 0;
            for (uint32_t c = tid; c < C; c += kTPB) {
                uint64_t K;
                uint32_t J, H;
                class_key(a, cs, c, K, J, H, ok);
                a.cls_kk[c] = K;
                a.cls_kj[c] = J;
                fin += K != ~0ull ? 1u : 0u;
            }
            if (__syncthreads_or(!ok)) return Resume{k, A, total};
            block_scan(fin, S.w, fin);
            uint64_t TK = ~0ull;
            uint32_t TJ = kNone;
            if (fin > kPool) select_pairs(a.cls_kk, a.cls_kj, C, kPool, TK, TJ, S);
            __syncthreads();
            for (uint32_t c = tid; c < C; c += kTPB) {
                const uint64_t K = a.cls_kk[c];
                const uint32_t J = a.cls_kj[c];
                if (K != ~0ull && !pair_lt(TK, TJ, K, J)) {
                    const uint32_t slot = atomicAdd(&S.cnt[2], 1u);   // below kPool
                    if (slot < kPool) {
                        S.pk[cur][slot] = K;
                        S.pj[cur][slot] = J;
                        S.ph[cur][slot] = ld_relaxed(&a.cls_head[c]);
                        S.pc[cur][slot] = c;
                    }
                }
            }
            __syncthreads();
            np = S.cnt[2] < kPool ? S.cnt[2] : kPool;
            uint32_t N = 1;
            while (N < np) N <<= 1;
            if (tid >= np && tid < N) {
                S.pk[cur][tid] = ~0ull;
                S.pj[cur][tid] = kNone;
            }
            bitonic(S.pk[cur], S.pj[cur], S.ph[cur], S.pc[cur], N);
            tK = TK;
            tJ = TJ;
            if (tid == 0) S.cnt[2] = 0;
        }

        // 3. the windows of the m best classes, two per wave (a half-wave
        //    each): their pending members from the bitmap, their keys and
        //    what a dispatch needs of them; none after the m-th best head is
        //    among the first m
        const uint32_t R = m < np ? m : np;
        lds_sync();
        {
            const uint32_t half = lane >> 5, hl = lane & 31u, r = w + kNW * half;
            const bool act = r < R;
            uint32_t h = 0, e = 0, want = 0;
            double E = 0.0, TS = 0.0;
            if (act) {
                const uint32_t c = S.pc[cur][r];
                h = S.ph[cur][r];
                e = cs.cstart[c + 1];
                want = m - r;
                if (hl == 0) {
                    const uint32_t g = cs.cg[c];
                    const double tb = cs.ctb[c], s = cs.cs[c], B = a.state[g];
                    S.sc[r] = c;
                    S.sg[r] = g;
                    S.sgf[r] = cs.gfirst[c];
                    S.sge[r] = cs.gend[c];
                    S.sB[r] = B;
                    S.last[r] = 0;
                    E = tb * B;
                    E = E * s;
                    TS = tb * s;
                }
            }
            E = __shfl(E, (int)(lane & 32u), 64);
            TS = __shfl(TS, (int)(lane & 32u), 64);
            uint32_t got = 0;
            for (uint64_t wb = h >> 6;; wb += 32) {
                const bool need = act && got < want && wb * 64u < e;
                if (!__any(need)) break;
                const uint64_t wi = wb + hl;
                uint64_t bits = 0;
                if (need && wi * 64u < e) {
                    bits = ld_relaxed64(&a.cls_elig[wi]);
                    if (wi == (h >> 6)) bits &= ~0ull << (h & 63u);
                    const uint64_t below = e - wi * 64u;
                    if (below < 64) bits &= (1ull << below) - 1ull;
                }
                const uint32_t cnt = (uint32_t)__popcll(bits);
                const uint32_t incl = wave_incl_scan_dpp(cnt);
                const uint32_t lo = readlane32(incl, 31), hi = readlane32(incl, 63);
                uint32_t rank = got + (half ? incl - lo : incl) - cnt;
                while (bits && rank < want) {
                    S.wpos[r][rank] = (uint32_t)(wi * 64u) + (uint32_t)__ffsll((unsigned long long)bits) - 1u;
                    bits &= bits - 1ull;
                    rank++;
                }
                const uint32_t tot = half ? hi - lo : lo;
                got = got + tot < want ? got + tot : want;
            }
            if (act && hl < got) {
                // written by lanes of this wave above (LDS is in order per wave)
                const uint32_t p = S.wpos[r][hl];
                const uint32_t words = cs.lw[p], J = cs.lf[p], id = cs.clist[p], obs = cs.lobs[p];
                const double wd = (double)words;
                const double F = 1.0 + wd / a.f_ref;
                double b = E * F;
                b = wd + b;
                const uint64_t K = ordered_bits(b);
                if (hl == 0 || R < m || !pair_lt(S.pk[cur][m - 1], S.pj[cur][m - 1], K, J)) {
                    // the completion's term of Eq. (5), ahead of the serial updates
                    const double x = TS * F;
                    const bool use = isfinite(x) && x > 0.0;
                    const uint32_t slot = atomicAdd(&S.cnt[3], 1u);
                    S.u.w.k[slot] = K;
                    S.u.w.j[slot] = J;
                    S.u.w.t2[slot] = use ? a.alpha * ((double)obs / x) : 0.0;
                    S.u.w.id[slot] = id;
                    S.u.w.use[slot] = use ? 1u : 0u;
                    S.u.w.slot[slot] = (r << 5) | hl;
                }
            }
        }
        lds_sync();
        const uint32_t nc = S.cnt[3];
        if (nc < m) return Resume{k, A, total};   // not reached: the windows hold the first m
        for (uint32_t i = w; i < nc; i += kNW) {
            const uint32_t r = rank_in(S.u.w.k, S.u.w.j, nc, S.u.w.k[i], S.u.w.j[i], m);
            if (lane == 0 && r < m) S.sel[r] = i;
        }
        lds_sync();

        // 4. dispatch, and the completion events of the batch (wave 1: the
        //    global stores stay in flight on a wave other than the one that
        //    runs the factor updates next)
        if (tid >= 64 && tid - 64 < m) {
            const uint32_t d = tid - 64;
            const uint32_t i = S.sel[d], v = S.u.w.slot[i], r = v >> 5;
            const uint32_t p = S.wpos[r][v & 31u], id = S.u.w.id[i];
            if (total + d < n) a.seq[total + d] = id;
            a.tick_of[id] = (int32_t)k;
            atomicAnd((unsigned long long *)&a.cls_elig[p >> 6], ~(1ull << (p & 63u)));
            S.last[r] = 1;
            S.evg[d] = S.sg[r];
            S.evr[d] = r;
            S.evx[d] = S.u.w.t2[i];
            S.evo[d] = S.u.w.use[i];
        }
        if (tid == 0) S.cnt[3] = 0;
        lds_sync();
        // the classes served get new heads (wave 2, beside wave 0's updates)
        if (tid >= 128 && tid - 128 < R && S.last[tid - 128]) mark_dirty(S.sc[tid - 128], S);
        // 5. Eq. (5) with the ratio of Eq. (6) on one wave (lane i: the
        //    batch's i-th event): each group's first event walks that
        //    group's events in dispatch order; a group whose factor moved
        //    touches its classes (ranges, spread over the block below)
        if (w == 0) {
            const uint32_t g = lane < m ? S.evg[lane] : kNone;
            const uint64_t same = same_group_lanes(g, m, a.n_groups);
            uint32_t len = 0, g0 = 0;
            if (lane < m && (same & lanemask_lt()) == 0) {
                const uint32_t r0 = S.evr[lane];
                double c = S.sB[r0];
                bool moved = false;
                for (uint64_t bits = same; bits; bits &= bits - 1ull) {
                    const uint32_t r = (uint32_t)__ffsll((unsigned long long)bits) - 1u;
                    if (!S.evo[r]) continue;
                    const double t1 = oma * c;
                    c = t1 + S.evx[r];
                    moved = true;
                }
                if (moved) {
                    a.state[g] = c;
                    g0 = S.sgf[r0];
                    len = S.sge[r0] - g0;
                    if (len > kDirtyMax) {
                        S.cnt[1] = 1;
                        len = 0;
                    }
                }
            }
            if (lane < kClsMaxBatch) {
                S.rg0[lane] = g0;
                S.rlen[lane] = len;
            }
        }
        lds_sync();
        {
            // range r = tid / 32, its classes i, i + 32, ... from i = tid % 32
            const uint32_t r = tid >> 5, len = r < m ? S.rlen[r] : 0u;
            for (uint32_t u = tid & 31u; u < len && !S.cnt[1]; u += 32) mark_dirty(S.rg0[r] + u, S);
        }
        P -= m;
        total += m;
        lds_sync();
    }
    if (tid == 0) a.n_dispatched[0] = total;
    return Resume{a.n_ticks, A, total};
}

// LDS of the three engines (a run uses one at a time).
union EngineLds {
    ListLds l;
    QueueLds q;
    ClassLds c;
};

// One workgroup per run: the queue engine where the run has its tier runs,
// the class engine for SJF where it applies (the list engine taking over if
// its conditions fail), else the list engine.
__device__ __forceinline__ void engine_run(const EngineArgs &a, const ClassShared &cs, EngineLds &lds)
{
    if (a.rpos) {
        if (a.batch <= kQLdsBatch && a.n_groups <= kQLdsGroups) engine_queues<true>(a, lds.q);
        else engine_queues<false>(a, lds.q);
    } else if (a.cls_head) {
        const Resume r = engine_class(a, cs, lds.c);
        __syncthreads();
        if (r.k < a.n_ticks) engine_list(a, lds.l, r.k, r.A, r.total);
    } else {
        engine_list(a, lds.l);
    }
}

static_assert(sizeof(EngineBatch) + sizeof(ClassShared) <= 4096, "kernel arguments within 4 KB");

__global__ __launch_bounds__(kTPB) void k_sim_engine(EngineBatch eb, ClassShared cs)
{
    __shared__ EngineLds lds;
    engine_run(eb.r[blockIdx.x], cs, lds);
}

__global__ __launch_bounds__(kTPB) void k_sim_engine_many(const EngineArgs *__restrict__ runs, ClassShared cs)
{
    __shared__ EngineLds lds;
    engine_run(runs[blockIdx.x], cs, lds);
}

// A chunk's engine arguments (count runs) into their slots of the
// workspace's array.
__global__ void k_sim_stage(EngineBatch eb, EngineArgs *__restrict__ dst, uint32_t count)
{
    if (threadIdx.x < count) dst[threadIdx.x] = eb.r[threadIdx.x];
}

// ---- class structure set-up (the class engine's) -------------------------------------

struct ClassBuild {
    uint32_t n, n_cat, n_tenants, n_groups;
    const uint32_t *fifo, *counts, *tenant, *group, *observed;
    const uint8_t *category;
    const double *arrival, *t_base, *s_tenant;
    uint32_t *ctl, *fpos, *clist, *lpos, *lw, *lf, *lobs, *pos_f, *cls_f, *cls_pos, *cstart, *cg, *gfirst,
        *gend, *bcnt;
    double *wkey, *ckey, *arr_f, *ctb, *cs;
};

// FIFO position of each request; the two keys of the class sort (words,
// then the class as one integer, both exact in a double); inputs out of range
// leave the class engine out (ctl[1]).
__global__ void k_cls_prep(const ClassBuild b)
{
    bool bad = false;
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < b.n; i += gridDim.x * blockDim.x) {
        const uint32_t id = b.fifo[i];
        if (id < b.n) b.fpos[id] = i;
        else bad = true;
        const uint32_t cat = b.category[i], ten = b.tenant[i], g = b.group[i];
        const bool ok = cat < b.n_cat && ten < b.n_tenants && g < b.n_groups;
        bad = bad || !ok;
        b.wkey[i] = (double)b.counts[i];
        b.ckey[i] = ok ? (double)(((uint64_t)g * b.n_cat + cat) * b.n_tenants + ten) : 0.0;
    }
    if (bad) atomicOr(&b.ctl[1], 1u);
}

// Class boundaries of the sorted list, counted per block of kTPB positions;
// each entry's words, FIFO position and observed length.
__global__ __launch_bounds__(kTPB) void k_cls_mark(const ClassBuild b)
{
    const uint32_t p = blockIdx.x * kTPB + threadIdx.x;
    bool first = false;
    if (p < b.n) {
        const uint32_t id = b.clist[p];
        b.lpos[id] = p;
        b.lw[p] = b.counts[id];
        b.lf[p] = b.fpos[id];
        b.lobs[p] = b.observed[id];
        first = p == 0 || b.ckey[id] != b.ckey[b.clist[p - 1]];
    }
    const uint32_t c = (uint32_t)__syncthreads_count(first);
    if (threadIdx.x == 0) b.bcnt[blockIdx.x] = c;
}

// Exclusive scan of the block counts (one block); ctl[0] = the classes.
__global__ __launch_bounds__(kTPB) void k_cls_scan(const ClassBuild b, uint32_t nb)
{
    __shared__ uint32_t s_w[kNW];
    uint32_t run = 0;
    for (uint32_t c0 = 0; c0 < nb; c0 += kTPB) {
        const uint32_t i = c0 + threadIdx.x;
        const uint32_t x = i < nb ? b.bcnt[i] : 0u;
        uint32_t tot;
        const uint32_t ex = block_scan(x, s_w, tot);
        if (i < nb) b.bcnt[i] = run + ex;
        run += tot;
    }
    if (threadIdx.x == 0) b.ctl[0] = run;
}

// Class of each list position; each class's first position and constants.
__global__ __launch_bounds__(kTPB) void k_cls_ids(const ClassBuild b)
{
    __shared__ uint32_t s_w[kNW];
    const uint32_t p = blockIdx.x * kTPB + threadIdx.x;
    bool first = false;
    uint32_t id = 0;
    if (p < b.n) {
        id = b.clist[p];
        first = p == 0 || b.ckey[id] != b.ckey[b.clist[p - 1]];
    }
    uint32_t tot;
    const uint32_t ex = block_scan(first ? 1u : 0u, s_w, tot);
    if (p < b.n) {
        const uint32_t c = b.bcnt[blockIdx.x] + ex + (first ? 1u : 0u) - 1u;
        b.cls_pos[p] = c;
        if (first) {
            const double nan = __builtin_nan("");
            const uint32_t cat = b.category[id], ten = b.tenant[id];
            b.cstart[c] = p;
            b.ctb[c] = cat < b.n_cat ? b.t_base[cat] : nan;
            b.cs[c] = ten < b.n_tenants ? b.s_tenant[ten] : nan;
            b.cg[c] = b.group[id];
        }
        if (p == b.n - 1) b.cstart[c + 1] = b.n;
    }
}

// Each class's group range; list position, class and arrival of each FIFO
// position.
__global__ void k_cls_fin(const ClassBuild b)
{
    const uint32_t C = b.ctl[0];
    const uint32_t stride = gridDim.x * blockDim.x;
    for (uint32_t c = blockIdx.x * blockDim.x + threadIdx.x; c < C; c += stride) {
        const uint32_t g = b.cg[c];
        uint32_t lo = 0, hi = c;
        while (lo < hi) {
            const uint32_t mid = (lo + hi) >> 1;
            if (b.cg[mid] < g) lo = mid + 1;
            else hi = mid;
        }
        b.gfirst[c] = lo;
        lo = c + 1;
        hi = C;
        while (lo < hi) {
            const uint32_t mid = (lo + hi) >> 1;
            if (b.cg[mid] <= g) lo = mid + 1;
            else hi = mid;
        }
        b.gend[c] = lo;
    }
    for (uint32_t j = blockIdx.x * blockDim.x + threadIdx.x; j < b.n; j += stride) {
        uint32_t id = b.fifo[j];
        id = id < b.n ? id : 0u;
        uint32_t p = b.lpos[id];
        p = p < b.n ? p : 0u;   // the class list is a permutation of 0..n-1
        b.pos_f[j] = p;
        b.cls_f[j] = b.cls_pos[p];
        b.arr_f[j] = b.arrival[id];
    }
}

// The tier runs' entries in run order: request, arrival, group and
// observed length (with `shared`); and, per run of a chunk on the queue
// engine (blockIdx.y), the B-free estimate.
struct QPrep {
    const uint32_t *rpos, *fifo, *group, *observed;
    const double *arrival;
    uint32_t n, shared;
    uint32_t *qid, *qgrp, *qobs;
    double *qarr;
    const double *est[kSimChunk];
    double *qest[kSimChunk];
};

__global__ void k_sim_qprep(const QPrep q)
{
    const double *est = q.est[blockIdx.y];
    double *qest = q.qest[blockIdx.y];
    for (uint32_t r = blockIdx.x * blockDim.x + threadIdx.x; r < q.n; r += gridDim.x * blockDim.x) {
        uint32_t j = q.rpos[r];
        j = j < q.n ? j : 0u;
        uint32_t id = q.fifo[j];
        id = id < q.n ? id : 0u;   // the FIFO order is a permutation of 0..n-1
        if (q.shared && blockIdx.y == 0) {
            q.qid[r] = id;
            q.qarr[r] = q.arrival[id];
            q.qgrp[r] = q.group[id];
            q.qobs[r] = q.observed[id];
        }
        if (qest) qest[r] = est[id];
    }
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

// The class structure: 14 arrays of n words (cstart has n + 1), 5 of n
// doubles, the block counts and the control words.
uint64_t cls_shared_bytes(uint64_t n)
{
    return 13 * align_up(n * 4, 256) + align_up((n + 1) * 4, 256) + 5 * align_up(n * 8, 256) +
           align_up((n / kTPB + 1) * 4, 256) + 256;
}

// Per SJF run on the class engine: heads, the pending bitmap, rebuild keys.
uint64_t cls_run_bytes(uint64_t n)
{
    return 2 * align_up(n * 4, 256) + align_up((n / 64 + 1) * 8, 256) + align_up(n * 8, 256);
}

size_t sim_ws_bytes(uint64_t n, uint32_t n_runs)
{
    // shared: fifo, the tier runs (positions, starts, and each entry's
    // request, group, observed length and arrival), the class structure, then
    // the FIFO sort, the class sorts and the partition (one after the other);
    // per run: list x2, est_base, key, aux, val, the queue engine's
    // candidates, the class engine's state
    const uint64_t per = 2 * align_up(n * 4, 256) + 2 * align_up(n * 8, 256) +
                         align_up(n * sizeof(Aux), 256) + align_up(n, 256) + kCandBytes + cls_run_bytes(n);
    const uint64_t sort = sort_ws_bytes(n, 1), part = am_partition_ws_bytes(n);
    return 5 * align_up(n * 4, 256) + align_up(n * 8, 256) + 256 + cls_shared_bytes(n) +
           align_up((uint64_t)(n_runs ? n_runs : 1) * sizeof(EngineArgs), 256) +
           (uint64_t)(n_runs ? n_runs : 1) * per + (sort > part ? sort : part);
}

// SJF runs the class engine when its batches fit the windows, F is
// non-decreasing in the words (f_ref > 0), the class key is exact in a
// double and the run's index ranges are those the shared class structure
// was built with (the first run's).
bool class_engine_applies(const SimArgs &a, const SimArgs &a0)
{
    const double classes = (double)a.n_groups * (double)a.n_cat * (double)a.n_tenants;
    return a.policy == kSjf && a.batch >= 1 && a.batch <= kClsMaxBatch && a.f_ref > 0.0 && classes < 0x1p52 &&
           a.n_groups == a0.n_groups && a.n_cat == a0.n_cat && a.n_tenants == a0.n_tenants;
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
        hipLaunchKernelGGL(k_sim_empty, dim3(1), dim3(kSimMaxRuns), 0, s, a0.n_dispatched, n_runs);
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
    QPrep qp = {};
    qp.n = n;
    qp.rpos = rpos;
    qp.fifo = fifo;
    qp.group = a0.group;
    qp.observed = a0.observed;
    qp.arrival = a0.arrival;
    qp.qid = reinterpret_cast<uint32_t *>(take((uint64_t)n * 4));
    qp.qgrp = reinterpret_cast<uint32_t *>(take((uint64_t)n * 4));
    qp.qobs = reinterpret_cast<uint32_t *>(take((uint64_t)n * 4));
    qp.qarr = reinterpret_cast<double *>(take((uint64_t)n * 8));
    // every policy but SJF runs on the tier queues (up to the partition's limit)
    bool any_queues = false, any_class = false;
    for (uint32_t r = 0; r < n_runs; r++) {
        any_queues = any_queues || (runs[r].policy != kSjf && n <= kAmMaxN);
        any_class = any_class || class_engine_applies(runs[r], a0);
    }
    auto take32 = [&](uint64_t count) { return reinterpret_cast<uint32_t *>(take(count * 4)); };
    auto take64 = [&](uint64_t count) { return reinterpret_cast<double *>(take(count * 8)); };
    ClassBuild cb = {};
    cb.n = n;
    cb.n_cat = a0.n_cat;
    cb.n_tenants = a0.n_tenants;
    cb.n_groups = a0.n_groups;
    cb.fifo = fifo;
    cb.counts = a0.counts;
    cb.tenant = a0.tenant;
    cb.group = a0.group;
    cb.observed = a0.observed;
    cb.category = a0.category;
    cb.arrival = a0.arrival;
    cb.t_base = a0.t_base;
    cb.s_tenant = a0.s_tenant;
    cb.ctl = reinterpret_cast<uint32_t *>(take(256));
    cb.fpos = take32(n);
    cb.clist = take32(n);
    cb.lpos = take32(n);
    cb.lw = take32(n);
    cb.lf = take32(n);
    cb.lobs = take32(n);
    cb.pos_f = take32(n);
    cb.cls_f = take32(n);
    cb.cls_pos = take32(n);
    cb.cstart = take32((uint64_t)n + 1);
    cb.cg = take32(n);
    cb.gfirst = take32(n);
    cb.gend = take32(n);
    uint32_t *seq_words = take32(n);   // the requests by (words, FIFO position)
    cb.bcnt = take32(n / kTPB + 1);
    cb.wkey = take64(n);
    cb.ckey = take64(n);
    cb.arr_f = take64(n);
    cb.ctb = take64(n);
    cb.cs = take64(n);
    const ClassShared cshared = {cb.ctl, cb.clist, cb.lw, cb.lf, cb.lobs, cb.pos_f, cb.cls_f, cb.arr_f,
                                 cb.cstart, cb.ctb, cb.cs, cb.cg, cb.gfirst, cb.gend};
    EngineArgs *staged = reinterpret_cast<EngineArgs *>(take((uint64_t)n_runs * sizeof(EngineArgs)));
    // the runs' arguments, built here and launched chunk by chunk below
    std::unique_ptr<SetupArgs[]> sv(new (std::nothrow) SetupArgs[n_runs]);
    std::unique_ptr<EngineArgs[]> ev(new (std::nothrow) EngineArgs[n_runs]);
    std::unique_ptr<const double *[]> qest_in(new (std::nothrow) const double *[n_runs]);
    std::unique_ptr<double *[]> qest_out(new (std::nothrow) double *[n_runs]);
    if (!sv || !ev || !qest_in || !qest_out) return hipErrorOutOfMemory;
    memset(sv.get(), 0, n_runs * sizeof(SetupArgs));
    memset(ev.get(), 0, n_runs * sizeof(EngineArgs));
    for (uint32_t r = 0; r < n_runs; r++) {
        qest_in[r] = nullptr;
        qest_out[r] = nullptr;
    }
    for (uint32_t r = 0; r < n_runs; r++) {
        const SimArgs &a = runs[r];
        uint32_t *list0 = reinterpret_cast<uint32_t *>(take((uint64_t)n * 4));
        uint32_t *list1 = reinterpret_cast<uint32_t *>(take((uint64_t)n * 4));
        double *est_base = reinterpret_cast<double *>(take((uint64_t)n * 8));
        uint64_t *key = reinterpret_cast<uint64_t *>(take((uint64_t)n * 8));
        Aux *aux = reinterpret_cast<Aux *>(take((uint64_t)n * sizeof(Aux)));
        uint8_t *val = take(n);
        uint8_t *cand = take(kCandBytes);
        uint32_t *cls_head = take32(n);
        uint32_t *cls_kj = take32(n);
        uint64_t *cls_elig = reinterpret_cast<uint64_t *>(take64(n / 64 + 1));
        uint64_t *cls_kk = reinterpret_cast<uint64_t *>(take64(n));

        SetupArgs &su = sv[r];
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

        EngineArgs &ea = ev[r];
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
        for (uint32_t q = 0; q < kMaxQ; q++) {
            ea.weight[q] = q < a.n_tiers && a.weight[q] ? a.weight[q] : 1u;
            ea.prio[q] = a.prio[q];
        }
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
            ea.qid = qp.qid;
            ea.qarr = qp.qarr;
            ea.qgrp = qp.qgrp;
            ea.qobs = qp.qobs;
            // the list engine's key buffer, unused on this engine
            ea.qest = reinterpret_cast<double *>(key);
            qest_in[r] = est_base;
            qest_out[r] = reinterpret_cast<double *>(key);
            ea.cand_k = reinterpret_cast<uint64_t *>(cand);
            ea.cand_j = reinterpret_cast<uint32_t *>(cand + (uint64_t)kMaxQ * kSimMaxBatch * 8);
            ea.cand_i = reinterpret_cast<uint32_t *>(cand + (uint64_t)kMaxQ * kSimMaxBatch * 12);
        }
        if (class_engine_applies(a, a0)) {
            ea.cls_head = cls_head;
            ea.cls_elig = cls_elig;
            ea.cls_kk = cls_kk;
            ea.cls_kj = cls_kj;
        }
        ea.f_ref = a.f_ref;
    }
    void *sort_ws = p;
    for (uint32_t r0 = 0; r0 < n_runs; r0 += kSimChunk) {
        const uint32_t cnt = n_runs - r0 < kSimChunk ? n_runs - r0 : kSimChunk;
        SetupBatch sb;
        memset(&sb, 0, sizeof(sb));
        for (uint32_t i = 0; i < cnt; i++) sb.r[i] = sv[r0 + i];
        hipLaunchKernelGGL(k_sim_setup, dim3(grid_for(n), cnt), dim3(256), 0, s, sb);
    }

    SortInput in = {};
    in.n = n;
    in.arrival = a0.arrival;
    in.wait = wait;
    in.wait.clear = false;
    SortJob job = {SortKind::Fifo, 64, nullptr, fifo};
    hipError_t e = sort_launch(in, &job, 1, sort_ws, s);
    if (e != hipSuccess) return e;
    if (any_class) {
        // the class lists: the FIFO sequence sorted stably by words, then by
        // class (the sort's workspace is free again on the stream)
        e = fill_u32(cb.ctl, 0u, 2, s);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(k_cls_prep, dim3(grid_for(n)), dim3(256), 0, s, cb);
        SortInput cin = {};
        cin.n = n;
        cin.wait = in.wait;
        cin.fifo = fifo;
        cin.budget = cb.wkey;
        SortJob cj = {SortKind::Budget, 64, nullptr, seq_words};
        e = sort_launch(cin, &cj, 1, sort_ws, s);
        if (e != hipSuccess) return e;
        cin.fifo = seq_words;
        cin.budget = cb.ckey;
        cj.out = cb.clist;
        e = sort_launch(cin, &cj, 1, sort_ws, s);
        if (e != hipSuccess) return e;
        const uint32_t nb = (uint32_t)cdiv(n, kTPB);
        hipLaunchKernelGGL(k_cls_mark, dim3(nb), dim3(kTPB), 0, s, cb);
        hipLaunchKernelGGL(k_cls_scan, dim3(1), dim3(kTPB), 0, s, cb, nb);
        hipLaunchKernelGGL(k_cls_ids, dim3(nb), dim3(kTPB), 0, s, cb);
        hipLaunchKernelGGL(k_cls_fin, dim3(grid_for(n)), dim3(256), 0, s, cb);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
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
        for (uint32_t r0 = 0; r0 < n_runs; r0 += kSimChunk) {
            const uint32_t cnt = n_runs - r0 < kSimChunk ? n_runs - r0 : kSimChunk;
            qp.shared = r0 == 0;
            for (uint32_t i = 0; i < kSimChunk; i++) {
                qp.est[i] = i < cnt ? qest_in[r0 + i] : nullptr;
                qp.qest[i] = i < cnt ? qest_out[r0 + i] : nullptr;
            }
            hipLaunchKernelGGL(k_sim_qprep, dim3(grid_for(n), cnt), dim3(256), 0, s, qp);
        }
    }
    if (n_runs <= kSimChunk) {
        EngineBatch eb;
        memset(&eb, 0, sizeof(eb));
        for (uint32_t r = 0; r < n_runs; r++) eb.r[r] = ev[r];
        hipLaunchKernelGGL(k_sim_engine, dim3(n_runs), dim3(kTPB), 0, s, eb, cshared);
    } else {
        for (uint32_t r0 = 0; r0 < n_runs; r0 += kSimChunk) {
            const uint32_t cnt = n_runs - r0 < kSimChunk ? n_runs - r0 : kSimChunk;
            EngineBatch eb;
            memset(&eb, 0, sizeof(eb));
            for (uint32_t i = 0; i < cnt; i++) eb.r[i] = ev[r0 + i];
            hipLaunchKernelGGL(k_sim_stage, dim3(1), dim3(64), 0, s, eb, staged + r0, cnt);
        }
        hipLaunchKernelGGL(k_sim_engine_many, dim3(n_runs), dim3(kTPB), 0, s, staged, cshared);
    }
    return hipGetLastError();
}

}  // namespace ds
