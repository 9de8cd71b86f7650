// Stage 4: dispatch orders (Sec. "Scheduling Engine").
//
// Every policy ends ties in FIFO order, so each one is a stable reordering
// of the FIFO sequence:
//   FIFO      radix sort of (arrival, index)
//   Priority  stable partition of the FIFO sequence by priority class
//   Weighted  stable partition by tier, then each request goes straight to
//             its cyclic round-robin position (closed form of the round)
//   SJF       stable radix sort of the FIFO sequence by budget
//   Aging     stable radix sort of the FIFO sequence by the aged score
// The FIFO sort runs first (unless the caller passes it in); the requested
// policy sorts then run together in one batch of launches. Up to kSsMaxN
// requests the 64-bit-key sorts (FIFO, SJF, Aging) are sample sorts of three
// launches, and the one-pass partitions (Priority, Weighted) a batch of their
// own.
#include <algorithm>

#include "common.h"
#include "kernels.h"
#include "partbody.h"

namespace ds {
namespace {

__global__ void k_copy_fifo(const uint32_t *__restrict__ fifo, const double *__restrict__ arrival,
                            uint32_t n, uint32_t *__restrict__ perm, double *__restrict__ key)
{
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

// Up to kSsMaxN requests: the look-back words of the two partitions, an
// error word, the tier counts of the slices of the batch, and the tiers,
// budgets and arrivals in FIFO order.
static size_t part_region_bytes(uint64_t n)
{
    return n <= kSsMaxN ? 2 * part_ws_bytes(n) + 256 + align_up((uint64_t)ssort_sample_blocks(n) * 64, 256) +
                              align_up(n, 256) + 2 * align_up(n * 8, 256)
                        : 0;
}

size_t order_ws_bytes(uint64_t n, uint32_t npolicies)
{
    uint32_t nsorts = npolicies < 1 ? 1 : (npolicies > kMaxSorts ? kMaxSorts : npolicies);
    // the FIFO sort and the policy sorts run one after another on the stream
    // and share the sort workspace
    const size_t radix = sort_ws_bytes(n, nsorts), sample = ssort_ws_bytes(n, nsorts);
    return align_up(n * 4, 256) + part_region_bytes(n) + (radix > sample ? radix : sample);
}

hipError_t order_launch(const OrderArgs &a, void *ws, uint32_t *flag, hipStream_t s)
{
    const uint32_t n = a.n;
    if (flag) {
        uint64_t nb = cdiv(n, 256);
        uint32_t vb = (uint32_t)(nb < 1024 ? nb : 1024);
        if (vb) hipLaunchKernelGGL(k_order_validate, dim3(vb), dim3(256), 0, s, a, flag);
        return hipGetLastError();
    }
    if (n == 0 || a.mask == 0) return hipSuccess;
    // workspace: FIFO permutation, partition look-back words, sort workspace
    uint8_t *p = static_cast<uint8_t *>(ws);
    uint32_t *fifo_ws = reinterpret_cast<uint32_t *>(p);
    uint8_t *part_ws = p + align_up((uint64_t)n * 4, 256);
    void *sort_ws = part_ws + part_region_bytes(n);

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
    in.aging_rate = a.aging_rate;
    in.t_now = a.t_now;
    in.aging_floor = a.aging_floor;

    const bool want_fifo = a.mask & 1u;
    const uint32_t *fifo = a.fifo_in;
    hipError_t err;
    const bool sample = n <= kSsMaxN;
    const bool parts = sample && (a.mask & 6u);   // Priority or Weighted by the one-pass partition
    // partition region: look-back words of two jobs, error word, tier counts
    uint32_t *pstatus = reinterpret_cast<uint32_t *>(part_ws);
    uint32_t *perror = reinterpret_cast<uint32_t *>(part_ws + 2 * part_ws_bytes(n));
    uint32_t *tier_part = reinterpret_cast<uint32_t *>(part_ws + 2 * part_ws_bytes(n) + 256);
    const uint32_t nparts = sample ? ssort_sample_blocks(n) : 0u;
    const uint32_t clear_words = (uint32_t)(2 * part_ws_bytes(n) / 4 + 1);
    uint8_t *fcopy = part_ws + 2 * part_ws_bytes(n) + 256 + align_up((uint64_t)nparts * 64, 256);
    uint8_t *ftier = fcopy;
    double *fbudget = reinterpret_cast<double *>(fcopy + align_up(n, 256));
    double *farr = reinterpret_cast<double *>(fcopy + align_up(n, 256) + align_up((uint64_t)n * 8, 256));
    if (!fifo) {
        SortJob job = {SortKind::Fifo, 64, want_fifo ? a.key[0] : nullptr,
                       want_fifo ? a.perm[0] : fifo_ws};
        // the policies after the FIFO sort read tiers, budgets and arrivals
        // in FIFO order, written by its last launch
        SsSide side = {nullptr, 0u, nullptr, nullptr, nullptr, nullptr};
        if (sample) {
            if (parts) {
                side.clear = pstatus;
                side.clear_words = clear_words;
                side.tier_part = tier_part;
            }
            if (a.mask & 0x16u) side.ftier = ftier;                       // Priority, Weighted, Aging
            if ((a.mask & (1u << 3)) && a.budget) side.fbudget = fbudget;  // SJF
            if (a.mask & (1u << 4)) side.farr = farr;                      // Aging
        }
        err = sample ? ssort_launch(in, &job, 1, a.serial_sort, sort_ws, s, &side)
                     : sort_launch(in, &job, 1, sort_ws, s);
        if (err != hipSuccess) return err;
        fifo = job.out;
        in.ftier = side.ftier;
        in.fbudget = side.fbudget;
        in.farr = side.farr;
    } else {
        if (want_fifo) {
            uint64_t nb = cdiv(n, 256);
            uint32_t blocks = (uint32_t)(nb < 4096 ? nb : 4096);
            hipLaunchKernelGGL(k_copy_fifo, dim3(blocks), dim3(256), 0, s, fifo, a.arrival, n,
                               a.perm[0], a.key[0]);
        }
        if (parts) {
            err = part_prepare(in, pstatus, clear_words, tier_part, nparts, s);
            if (err != hipSuccess) return err;
        }
    }
    in.fifo = fifo;

    SortJob jobs[kMaxSorts];
    uint32_t nj = 0;
    if (a.mask & (1u << 1)) {
        // priority classes: rank of each tier's priority among the distinct values
        double vals[16];
        for (uint32_t q = 0; q < a.n_tiers; q++) vals[q] = a.prio[q];
        std::sort(vals, vals + a.n_tiers);
        uint32_t nd = (uint32_t)(std::unique(vals, vals + a.n_tiers) - vals);
        for (uint32_t q = 0; q < 16; q++) {
            uint32_t c = 0;
            if (q < a.n_tiers)
                while (c + 1 < nd && vals[c] < a.prio[q]) c++;
            in.cls[q] = c;
        }
        jobs[nj++] = {SortKind::Class, 8, a.key[1], a.perm[1]};
    }
    if (a.mask & (1u << 2)) jobs[nj++] = {SortKind::Tier, 8, a.key[2], a.perm[2]};
    if (a.mask & (1u << 3)) jobs[nj++] = {SortKind::Budget, 64, a.key[3], a.perm[3]};
    if (a.mask & (1u << 4)) jobs[nj++] = {SortKind::Aging, 64, a.key[4], a.perm[4]};
    if (nj == 0) return hipGetLastError();
    if (!sample) return sort_launch(in, jobs, nj, sort_ws, s);
    SortJob part[kMaxSorts], keyed[kMaxSorts];
    uint32_t np = 0, nk = 0;
    for (uint32_t i = 0; i < nj; i++) {
        if (jobs[i].kind == SortKind::Budget || jobs[i].kind == SortKind::Aging)
            keyed[nk++] = jobs[i];
        else
            part[np++] = jobs[i];
    }
    if (nk) {
        // SJF/Aging sampling and the Priority/Weighted tiles share a launch
        const PartBatch pb = part_batch(in, part, np, pstatus, perror, tier_part, nparts);
        return ssort_launch(in, keyed, nk, a.serial_sort, sort_ws, s, nullptr, np ? &pb : nullptr);
    }
    if (np) return part_launch(in, part, np, pstatus, perror, tier_part, nparts, s);
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
