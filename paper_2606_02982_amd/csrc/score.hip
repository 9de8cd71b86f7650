// Stage 3: calibrated output estimate, token budget and runtime class
// (Eq. (2), Eq. (1), Eq. (4); the per-request arithmetic is score_one).
// Elementwise.
#include "common.h"
#include "kernels.h"
#include "scoremath.h"

namespace ds {
namespace {

__global__ __launch_bounds__(256) void k_score(ScoreArgs a)
{
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < a.n; i += gridDim.x * blockDim.x)
        score_one(a, i, a.counts[i]);
}

__global__ void k_score_validate(ScoreArgs a, uint32_t *__restrict__ flag)
{
    uint32_t bad = 0;
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < a.n; i += gridDim.x * blockDim.x)
        if (a.category[i] >= a.n_cat || a.tenant[i] >= a.n_tenants ||
            (a.group ? a.group[i] : i) >= a.n_groups)
            bad = 1;
    if (bad) atomicOr(flag, 1u);
}

}  // namespace

hipError_t score_launch(uint32_t n, const uint32_t *counts, const uint8_t *category,
                        const uint32_t *tenant, const uint32_t *group, const double *t_base,
                        uint32_t n_cat, const double *s_tenant, uint32_t n_tenants,
                        const double *state, uint32_t n_groups, double f_ref, double short_max,
                        double medium_max, double *est_base, double *est, double *budget,
                        uint8_t *job_class, uint32_t *flag, hipStream_t s)
{
    ScoreArgs a = {n, counts, category, tenant, group, t_base, n_cat, s_tenant, n_tenants,
                   state, n_groups, f_ref, short_max, medium_max, est_base, est, budget,
                   job_class};
    uint64_t nb = cdiv(n, 256);
    uint32_t blocks = (uint32_t)(nb < 8192 ? nb : 8192);
    if (blocks == 0) return hipSuccess;
    if (flag) {
        uint32_t vb = blocks < 1024 ? blocks : 1024;
        hipLaunchKernelGGL(k_score_validate, dim3(vb), dim3(256), 0, s, a, flag);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(k_score, dim3(blocks), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace ds
