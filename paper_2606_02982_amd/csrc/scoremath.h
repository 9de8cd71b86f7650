// Stage 3 for one request (internal to the library): the calibrated output
// estimate of Eq. (2), its factors gathered in the order of Alg. 1 (T_base,
// then B_runtime, then S_tenant, then F_input), the budget of Eq. (1)
// (T_input + estimate) and the class thresholds of Eq. (4). The library is
// built with -ffp-contract=off, so every product and sum is rounded
// separately. Used by the score kernel and by the fused characterize pass.
#pragma once

#include "common.h"
#include "kernels.h"

namespace ds {

__device__ __forceinline__ void score_one(const ScoreArgs &a, uint32_t i, uint32_t count)
{
    const double nan = __builtin_nan("");
    // no group array: state holds each request's own factor (as-of scoring)
    const uint32_t cat = a.category[i], ten = a.tenant[i], g = a.group ? a.group[i] : i;
    const double words = (double)count;
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

}  // namespace ds
