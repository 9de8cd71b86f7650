// Stage 4: dispatch orders (Sec. "Scheduling Engine").
//
// Every policy ends ties in FIFO order, so each one is a stable reordering
// of the FIFO sequence:
//   FIFO      order of (arrival, index)
//   Priority  stable partition of the FIFO sequence by priority class
//   Weighted  stable partition by tier, then each request goes straight to
//             its cyclic round-robin position (closed form of the round, or
//             of the smooth interleaving's period table)
//   SJF       stable sort of the FIFO sequence by budget
//   Aging     stable sort of the FIFO sequence by the aged score
// Up to kSsMaxN requests FIFO, SJF and Aging are sample sorts by the
// composite key (policy key, arrival, index), all in the same three
// launches, and the FIFO sort's last launch also places Priority and
// Weighted. Above that, the FIFO permutation is sorted first (unless the
// caller passes it in) and the other policies are LSD radix sorts of the
// FIFO sequence, batched in one set of launches.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace ds {
namespace {

__global__ void k_copy_fifo(const uint32_t *__restrict__ fifo, const double *__restrict__ arrival,
                            uint32_t n, uint32_t *__restrict__ perm, double *__restrict__ key,
                            uint32_t *__restrict__ wait_status)
{
    if (wait_status && blockIdx.x == 0 && threadIdx.x == 0) *wait_status = 0;
    for (uint32_t j = blockIdx.x * blockDim.x + threadIdx.x; j < n; j += gridDim.x * blockDim.x) {
        perm[j] = fifo[j];
        if (key) key[j] = arrival[j];
    }
}

__global__ void k_order_validate(OrderArgs a, uint32_t *__restrict__ flag)
{
    uint32_t bad = 0;
    const bool need_budget = (a.mask >> 3) & 1u;
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < a.n; i += gridDim.x * blockDim.x) {
        if (a.tier[i] >= a.n_tiers) bad = 1;
        if (isnan(a.arrival[i])) bad = 1;
        if (need_budget && isnan(a.budget[i])) bad = 1;
        if (a.fifo_in) {
            // strictly increasing in (arrival, index) and in range: a permutation
            uint32_t f = a.fifo_in[i];
            if (f >= a.n) {
                bad = 1;
            } else if (i + 1 < a.n) {
                uint32_t h = a.fifo_in[i + 1];
                if (h >= a.n) {
                    bad = 1;
                } else {
                    double x = a.arrival[f], y = a.arrival[h];
                    if (!(x < y || (x == y && f < h))) bad = 1;
                }
            }
        }
    }
    if (bad) atomicOr(flag, 1u);
}

}  // namespace

size_t order_ws_bytes(uint64_t n, uint32_t npolicies)
{
    // sample sorts: the FIFO sort and each policy's; radix sorts: the FIFO
    // permutation, then the policy sorts (sharing the sort workspace with the
    // FIFO sort, which runs before them on the stream)
    const uint32_t np = npolicies < 1 ? 1 : npolicies;
    const uint32_t nss = np + 1 > kSsMaxSorts ? kSsMaxSorts : np + 1;
    const uint32_t nrs = np > kMaxSorts ? kMaxSorts : np;
    const size_t sample = ssort_ws_bytes(n < kSsMaxN ? n : kSsMaxN, nss);
    const size_t rs = sort_ws_bytes(n, nrs);
    // (FIFO-ordered copies of arrival, budget and tier for the batch over the
    // FIFO sequence, and the Aging runs with their merge scratch)
    const size_t lb = lsort_ws_bytes(n, 1, 2);
    const size_t ls = lb ? 2 * align_up(n * 8, 256) + align_up(n, 256) + 2 * align_up(n * 8, 256) +
                               2 * align_up(n * 4, 256) + align_up(17 * 4, 256) + lsort_sample_bytes(n) + lb
                         : 0;
    const size_t radix = align_up(n * 4, 256) + (ls > rs ? ls : rs);
    // the larger of the two keeps the size non-decreasing in n
    return n <= kSsMaxN ? sample : (radix > sample ? radix : sample);
}

hipError_t order_launch(const OrderArgs &a, void *ws, uint32_t *flag, hipStream_t s, WaitCfg wait)
{
    const uint32_t n = a.n;
    if (flag) {
        uint64_t nb = cdiv(n, 256);
        uint32_t vb = (uint32_t)(nb < 1024 ? nb : 1024);
        if (vb) hipLaunchKernelGGL(k_order_validate, dim3(vb), dim3(256), 0, s, a, flag);
        return hipGetLastError();
    }
    if (n == 0 || a.mask == 0) return hipSuccess;

    SortInput in = {};
    in.n = n;
    in.arrival = a.arrival;
    in.budget = a.budget;
    in.tier = a.tier;
    in.n_tiers = a.n_tiers;
    for (int q = 0; q < 16; q++) {
        in.prio[q] = a.prio[q];
        in.weight[q] = a.weight[q];
    }
    in.wrr_mode = a.wrr_mode;
    in.aging_rate = a.aging_rate;
    in.t_now = a.t_now;
    in.aging_floor = a.aging_floor;
    in.wait = wait;
    uint32_t n_classes = 1;
    if (a.mask & ((1u << 1) | (1u << 4))) {
        // priority classes: rank of each tier's priority among the distinct values
        double vals[16];
        for (uint32_t q = 0; q < a.n_tiers; q++) vals[q] = a.prio[q];
        std::sort(vals, vals + a.n_tiers);
        uint32_t nd = (uint32_t)(std::unique(vals, vals + a.n_tiers) - vals);
        n_classes = nd;
        for (uint32_t q = 0; q < 16; q++) {
            uint32_t c = 0;
            if (q < a.n_tiers)
                while (c + 1 < nd && vals[c] < a.prio[q]) c++;
            in.cls[q] = c;
        }
    }
    const bool want_fifo = a.mask & 1u;
    if (want_fifo && a.fifo_in) {
        uint64_t nb = cdiv(n, 256);
        uint32_t blocks = (uint32_t)(nb < 4096 ? nb : 4096);
        hipLaunchKernelGGL(k_copy_fifo, dim3(blocks), dim3(256), 0, s, a.fifo_in, a.arrival, n, a.perm[0],
                           a.key[0], wait.clear ? wait.status : nullptr);
        in.wait.clear = false;
    }
    if (n <= kSsMaxN) {
        // one batch of sample sorts: FIFO (carrying Priority and Weighted),
        // SJF, Aging; a given fifo_in only saves the FIFO sort when neither
        // partition is wanted
        const bool parts = a.mask & 6u;
        SsPartitions pw = {{nullptr, nullptr}, {nullptr, nullptr}};
        for (int e = 0; e < 2; e++)
            if (a.mask & (2u << e)) {
                pw.perm[e] = a.perm[1 + e];
                pw.key[e] = a.key[1 + e];
            }
        SortJob all[kSsMaxSorts];
        uint32_t na = 0;
        const bool fifo_out = want_fifo && !a.fifo_in;
        if (fifo_out || parts)
            all[na++] = {SortKind::Fifo, 64, fifo_out ? a.key[0] : nullptr, fifo_out ? a.perm[0] : nullptr};
        if (a.mask & (1u << 3)) all[na++] = {SortKind::Budget, 64, a.key[3], a.perm[3]};
        if (a.mask & (1u << 4)) all[na++] = {SortKind::Aging, 64, a.key[4], a.perm[4]};
        if (na == 0) return hipGetLastError();
        return ssort_launch(in, all, na, a.serial_sort, ws, s, parts ? &pw : nullptr);
    }

    uint8_t *p = static_cast<uint8_t *>(ws);
    uint32_t *fifo_ws = reinterpret_cast<uint32_t *>(p);
    void *sort_ws = p + align_up((uint64_t)n * 4, 256);
    if (n <= kLsMaxN) {
        // the FIFO sort, then every other policy over the FIFO sequence in
        // one batch of sample sorts and partitions (lsort.hip)
        uint8_t *q = static_cast<uint8_t *>(sort_ws);
        LsCopies cp;
        cp.arr = reinterpret_cast<double *>(q);
        q += align_up((uint64_t)n * 8, 256);
        cp.bud = (a.mask & (1u << 3)) ? reinterpret_cast<double *>(q) : nullptr;
        q += align_up((uint64_t)n * 8, 256);
        cp.tier = q;
        q += align_up(n, 256);
        uint64_t *rk[2];
        uint32_t *rp[2];
        for (int e = 0; e < 2; e++) {
            rk[e] = reinterpret_cast<uint64_t *>(q);
            q += align_up((uint64_t)n * 8, 256);
        }
        for (int e = 0; e < 2; e++) {
            rp[e] = reinterpret_cast<uint32_t *>(q);
            q += align_up((uint64_t)n * 4, 256);
        }
        LsRuns runs = {rk[0], rp[0], reinterpret_cast<uint32_t *>(q)};
        q += align_up(17 * 4, 256);
        LsSample sjf = lsort_sample_at(n, q);
        q += lsort_sample_bytes(n);
        void *batch_ws = q;
        const bool more = a.mask & ~1u;   // policies over the FIFO sequence
        const uint32_t *fifo = a.fifo_in;
        bool sjf_drawn = false;
        if (!fifo) {
            // (SJF's splitters are drawn in the same launches)
            sjf_drawn = (a.mask & (1u << 3)) != 0;
            SortJob job = {SortKind::Fifo, 64, want_fifo ? a.key[0] : nullptr, want_fifo ? a.perm[0] : fifo_ws};
            hipError_t err = lsort_launch(in, &job, 1, batch_ws, s, nullptr, more ? &cp : nullptr, nullptr,
                                          sjf_drawn ? &sjf : nullptr);
            if (err != hipSuccess) return err;
            fifo = job.out;
            in.wait.clear = false;
        }
        sjf.draw = false;
        in.fifo = fifo;
        // SJF sorts; Priority partitions (and lays out the priority classes'
        // runs, which the Aging merge then combines); Weighted partitions
        const bool prio = a.mask & (1u << 1), aging = a.mask & (1u << 4);
        SortJob jobs[3];
        uint32_t nj = 0;
        if (a.mask & (1u << 3)) jobs[nj++] = {SortKind::Budget, 64, a.key[3], a.perm[3]};
        if (prio || aging)
            jobs[nj++] = {SortKind::Class, 8, prio ? a.key[1] : nullptr, prio ? a.perm[1] : nullptr};
        if (a.mask & (1u << 2)) jobs[nj++] = {SortKind::Tier, 8, a.key[2], a.perm[2]};
        if (nj == 0) return hipGetLastError();
        hipError_t err = lsort_launch(in, jobs, nj, batch_ws, s, a.fifo_in ? nullptr : &cp, nullptr,
                                      aging ? &runs : nullptr, sjf_drawn ? &sjf : nullptr);
        if (err != hipSuccess || !aging) return err;
        return am_merge_launch(in, n_classes, runs.cstart, rk, rp, a.perm[4], a.key[4], s);
    }

    // the policy sorts over the FIFO sequence; Aging as the merge of the
    // priority classes' runs of that sequence (agmerge.hip) where its
    // buffers fit the sort workspace, else as one more radix sort
    const bool aging_merge = (a.mask & (1u << 4)) && n <= kAmMaxN && am_ws_bytes(n) <= sort_ws_bytes(n, 1);
    SortJob jobs[kMaxSorts];
    uint32_t nj = 0;
    if (a.mask & (1u << 1)) jobs[nj++] = {SortKind::Class, 8, a.key[1], a.perm[1]};
    if (a.mask & (1u << 2)) jobs[nj++] = {SortKind::Tier, 8, a.key[2], a.perm[2]};
    if (a.mask & (1u << 3)) jobs[nj++] = {SortKind::Budget, 64, a.key[3], a.perm[3]};
    if ((a.mask & (1u << 4)) && !aging_merge) jobs[nj++] = {SortKind::Aging, 64, a.key[4], a.perm[4]};

    // radix sorts: the FIFO permutation first, then the policies over it
    const uint32_t *fifo = a.fifo_in;
    if (!fifo) {
        SortJob job = {SortKind::Fifo, 64, want_fifo ? a.key[0] : nullptr, want_fifo ? a.perm[0] : fifo_ws};
        hipError_t err = sort_launch(in, &job, 1, sort_ws, s);
        if (err != hipSuccess) return err;
        fifo = job.out;
        in.wait.clear = false;
    }
    in.fifo = fifo;
    if (nj > 0) {
        hipError_t err = sort_launch(in, jobs, nj, sort_ws, s);
        if (err != hipSuccess) return err;
        in.wait.clear = false;
    }
    // (after the sorts on the stream: the merge reuses their workspace)
    if (aging_merge)
        return am_launch(in, n_classes, a.perm[4], a.key[4], sort_ws, s,
                         in.wait.clear ? in.wait.status : nullptr);
    return hipGetLastError();
}

__global__ void k_fill_u32(uint32_t *__restrict__ p, uint32_t v, uint64_t n)
{
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

hipError_t fill_u32(uint32_t *p, uint32_t v, uint64_t n, hipStream_t s)
{
    uint64_t nb = cdiv(n, 256);
    uint32_t blocks = (uint32_t)(nb < 1024 ? nb : 1024);
    if (blocks) hipLaunchKernelGGL(k_fill_u32, dim3(blocks), dim3(256), 0, s, p, v, n);
    return hipGetLastError();
}

}  // namespace ds
