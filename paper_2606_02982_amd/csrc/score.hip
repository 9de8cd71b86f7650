// Stage 3: calibrated output estimate, token budget and runtime class.
//
// Eq. (2) in the order Alg. 1 gathers its factors (T_base, then B_runtime,
// then S_tenant, then F_input), Eq. (1) T_budget = T_input + estimate, and
// the class thresholds of Eq. (4). Elementwise; the library is built with
// -ffp-contract=off, so every product and sum is rounded separately.
#include "common.h"
#include "kernels.h"

namespace ds {
namespace {

struct ScoreArgs {
    uint32_t n;
    const uint32_t *counts;
    const uint8_t *category;
    const uint32_t *tenant;
    const uint32_t *group;
    const double *t_base;
    uint32_t n_cat;
    const double *s_tenant;
    uint32_t n_tenants;
    const double *state;
    uint32_t n_groups;
    double f_ref, short_max, medium_max;
    double *est_base, *est, *budget;
    uint8_t *job_class;
};

__global__ __launch_bounds__(256) void k_score(ScoreArgs a)
{
    const double nan = __builtin_nan("");
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < a.n; i += gridDim.x * blockDim.x) {
        const uint32_t cat = a.category[i], ten = a.tenant[i], g = a.group[i];
        const double words = (double)a.counts[i];
        const bool ok = cat < a.n_cat && ten < a.n_tenants && g < a.n_groups;
        const double tb = ok ? a.t_base[cat] : nan;
        const double s = ok ? a.s_tenant[ten] : nan;
        const double b = ok ? a.state[g] : nan;
        const double F = 1.0 + words / a.f_ref;
        double e = tb * b;
        e = e * s;
        e = e * F;
        if (a.est_base) {
            double e0 = tb * s;
            e0 = e0 * F;
            a.est_base[i] = e0;
        }
        a.est[i] = e;
        const double total = words + e;
        a.budget[i] = total;
        uint8_t c = 2;
        if (total <= a.short_max) c = 0;
        else if (total <= a.medium_max) c = 1;
        a.job_class[i] = c;
    }
}

__global__ void k_score_validate(ScoreArgs a, uint32_t *__restrict__ flag)
{
    uint32_t bad = 0;
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < a.n; i += gridDim.x * blockDim.x)
        if (a.category[i] >= a.n_cat || a.tenant[i] >= a.n_tenants || a.group[i] >= a.n_groups) bad = 1;
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
