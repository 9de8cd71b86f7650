// Stage 4, Priority and Weighted orders of up to kSsMaxN requests: the
// launches of the one-pass partition whose tile body is in partbody.h.
#include "partbody.h"

namespace ds {
namespace {

constexpr int kPTPB = 512;

__global__ __launch_bounds__(kPTPB) void k_part(PartBatch b)
{
    part_body<kPTPB>(b, blockIdx.y, blockIdx.x);
}

__global__ __launch_bounds__(256) void k_part_prepare(const uint8_t *tier, uint32_t n, uint32_t *clear,
                                                     uint32_t clear_words, uint32_t *tier_part)
{
    __shared__ uint32_t s_w[4 * kTierCounts];
    for (uint32_t i = blockIdx.x * 256u + threadIdx.x; i < clear_words; i += gridDim.x * 256u) clear[i] = 0;
    tier_partial<256>(tier, n, blockIdx.x, gridDim.x, tier_part, s_w);
}

}  // namespace

size_t part_ws_bytes(uint64_t n)
{
    return align_up(cdiv(n, kPTile) * kQ * 4, 256);
}

PartBatch part_batch(const SortInput &in, const SortJob *jobs, uint32_t njobs, uint32_t *status,
                     uint32_t *error, const uint32_t *tier_part, uint32_t nparts)
{
    PartBatch b;
    b.in = in;
    b.n = in.n;
    b.tiles = (uint32_t)cdiv(in.n, kPTile);
    b.njobs = njobs;
    b.tier_part = tier_part;
    b.nparts = nparts;
    for (uint32_t i = 0; i < njobs && i < 2; i++) {
        b.job[i].kind = jobs[i].kind;
        b.job[i].key_out = jobs[i].key_out;
        b.job[i].out = jobs[i].out;
        b.job[i].status = status + (uint64_t)i * b.tiles * kQ;
        b.job[i].error = error;
    }
    return b;
}

hipError_t part_prepare(const SortInput &in, uint32_t *clear, uint32_t clear_words,
                        uint32_t *tier_part, uint32_t nparts, hipStream_t s)
{
    hipLaunchKernelGGL(k_part_prepare, dim3(nparts), dim3(256), 0, s, in.tier, in.n, clear, clear_words,
                       tier_part);
    return hipGetLastError();
}

hipError_t part_launch(const SortInput &in, const SortJob *jobs, uint32_t njobs, uint32_t *status,
                       uint32_t *error, const uint32_t *tier_part, uint32_t nparts, hipStream_t s)
{
    if (in.n == 0 || njobs == 0) return hipSuccess;
    if (njobs > 2 || in.n > kSsMaxN) return hipErrorInvalidValue;
    for (uint32_t i = 0; i < njobs; i++)
        if (jobs[i].kind != SortKind::Class && jobs[i].kind != SortKind::Tier) return hipErrorInvalidValue;
    const PartBatch b = part_batch(in, jobs, njobs, status, error, tier_part, nparts);
    hipLaunchKernelGGL(k_part, dim3(b.tiles, njobs), dim3(kPTPB), 0, s, b);
    return hipGetLastError();
}

}  // namespace ds
