// Estimation error of budget estimates against observed output lengths
// (Sec. "Impact of Workload Characterization and Runtime Calibration":
// tab:four_mode_token_error and tab:error_reduction) and runtime-class
// counts per semantic category (Eq. (4); tab:workload_mapping).
//
// Error: for every event with a usable estimate x = est[e] * factor[e]
// (finite and > 0; no factor = 1), d = x - obs[e]; per group and over all
// events: count, sum |d|, sum d^2 and sum obs / x. Each block takes a
// contiguous range of events and accumulates per-group sums in LDS (1024
// groups per pass over its range) and the all-events sums in registers; it
// stores its partial sums, and a last kernel adds the blocks' partials in a
// fixed order and forms MAE = sum|d| / count, RMSE = sqrt(sum d^2 / count),
// mean bias = sum(obs / x) / count. No sum uses floating-point atomics: every
// order of addition is fixed by the data and the launch shape, so results
// are the same from run to run and agree with any sequential sum within the
// rounding of an n-term sum.
#include "common.h"
#include "kernels.h"

namespace ds {
namespace {

constexpr uint32_t kT = 256;
constexpr uint32_t kLdsGroups = 1024;   // groups summed in LDS per pass
constexpr uint32_t kMaxBlocks = 256;

constexpr uint32_t kU = 8;              // events per thread per step

__device__ __forceinline__ bool usable(double x) { return isfinite(x) && x > 0.0; }

// Estimates (times factors) and observed lengths of events b0 + u kT + t,
// u < kU; events at or past e1 get x = 0 (not usable).
__device__ __forceinline__ void load_events(const double *__restrict__ est,
                                            const double *__restrict__ factor,
                                            const uint32_t *__restrict__ obs, uint64_t b0,
                                            uint64_t e1, double (&x)[kU], double (&o)[kU])
{
    double f[kU];
#pragma unroll
    for (uint32_t u = 0; u < kU; u++) {
        const uint64_t e = b0 + u * kT + threadIdx.x;
        const bool in = e < e1;
        x[u] = in ? est[e] : 0.0;
        f[u] = in && factor ? factor[e] : 1.0;
        o[u] = in ? (double)obs[e] : 0.0;
    }
#pragma unroll
    for (uint32_t u = 0; u < kU; u++) x[u] = x[u] * f[u];
}

// partial layout: [block][4][G + 1] (count, sum |d|, sum d^2, sum obs/x);
// slot G holds the all-events sums
__global__ __launch_bounds__(kT) void k_err_accum(uint64_t n, const double *__restrict__ est,
                                                  const double *__restrict__ factor,
                                                  const uint32_t *__restrict__ obs,
                                                  const uint32_t *__restrict__ group, uint32_t G,
                                                  double *__restrict__ partial)
{
    __shared__ double lacc[4][kLdsGroups];
    __shared__ double wsum[4][kT / 64];
    const uint64_t slots = (uint64_t)G + 1;
    double *mine = partial + (uint64_t)blockIdx.x * 4 * slots;
    const uint64_t per = cdiv(n, gridDim.x);
    const uint64_t e0 = (uint64_t)blockIdx.x * per;
    const uint64_t e1 = e0 + per < n ? e0 + per : n;

    // all events: registers, then a block reduction; kU events per thread
    // per step, their loads issued together
    double c = 0.0, sa = 0.0, sq = 0.0, sr = 0.0;
    for (uint64_t b0 = e0; b0 < e1; b0 += kU * kT) {
        double x[kU], o[kU];
        load_events(est, factor, obs, b0, e1, x, o);
#pragma unroll
        for (uint32_t u = 0; u < kU; u++) {
            if (!usable(x[u])) continue;
            const double d = x[u] - o[u];
            c += 1.0;
            sa += fabs(d);
            sq += d * d;
            sr += o[u] / x[u];
        }
    }
    for (int off = 32; off >= 1; off >>= 1) {
        c += __shfl_xor(c, off, 64);
        sa += __shfl_xor(sa, off, 64);
        sq += __shfl_xor(sq, off, 64);
        sr += __shfl_xor(sr, off, 64);
    }
    if (lane_id() == 0) {
        const int w = threadIdx.x >> 6;
        wsum[0][w] = c;
        wsum[1][w] = sa;
        wsum[2][w] = sq;
        wsum[3][w] = sr;
    }
    __syncthreads();
    if (threadIdx.x < 4) {
        double s = 0.0;
        for (int k = 0; k < (int)(kT / 64); k++) s += wsum[threadIdx.x][k];
        mine[threadIdx.x * slots + G] = s;
    }
    if (!group) return;

    // groups, kLdsGroups at a time, in a fixed order: each step's events go
    // to LDS in event order; wave w owns the groups g = w (mod kWaves) of
    // the pass and walks the step's events round by round (64 at a time, in
    // order); the lanes of one group in a round are added up in lane order
    // by the lowest of them, which adds that to the group's sums. The result
    // does not depend on scheduling.
    constexpr uint32_t kWaves = kT / 64, kStep = kU * kT;
    __shared__ uint32_t sg[kStep];
    __shared__ double sv[3][kStep];
    const uint32_t lane = (uint32_t)lane_id(), w = threadIdx.x >> 6;
    for (uint32_t c0 = 0; c0 < G; c0 += kLdsGroups) {
        const uint32_t cn = G - c0 < kLdsGroups ? G - c0 : kLdsGroups;
        for (uint32_t i = threadIdx.x; i < cn; i += kT)
            lacc[0][i] = lacc[1][i] = lacc[2][i] = lacc[3][i] = 0.0;
        __syncthreads();
        for (uint64_t b0 = e0; b0 < e1; b0 += kStep) {
            double x[kU], o[kU];
            uint32_t g[kU];
#pragma unroll
            for (uint32_t u = 0; u < kU; u++) {
                const uint64_t e = b0 + u * kT + threadIdx.x;
                g[u] = e < e1 ? group[e] - c0 : 0xFFFFFFFFu;   // wraps below c0
            }
            load_events(est, factor, obs, b0, e1, x, o);
#pragma unroll
            for (uint32_t u = 0; u < kU; u++) {
                const uint32_t slot = u * kT + threadIdx.x;   // event order
                const bool ok = g[u] < cn && usable(x[u]);
                const double d = x[u] - o[u];
                sg[slot] = ok ? g[u] : 0xFFFFFFFFu;
                sv[0][slot] = ok ? fabs(d) : 0.0;
                sv[1][slot] = ok ? d * d : 0.0;
                sv[2][slot] = ok ? o[u] / x[u] : 0.0;
            }
            __syncthreads();
            for (uint32_t r = 0; r < kStep / 64; r++) {
                const uint32_t slot = r * 64 + lane;
                const uint32_t gv = sg[slot];
                const bool own = gv != 0xFFFFFFFFu && gv % kWaves == w;
                uint64_t peers = __ballot(own);
#pragma unroll
                for (int bb = 0; bb < 10; bb++) {   // group bits within the pass (kLdsGroups = 1024)
                    const bool bit = (gv >> bb) & 1u;
                    const uint64_t mk = __ballot(bit);
                    peers &= bit ? mk : ~mk;
                }
                if (own && (peers & lanemask_lt()) == 0) {
                    double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
                    for (uint64_t m = peers; m; m &= m - 1) {
                        const uint32_t q = r * 64 + (uint32_t)__builtin_ctzll(m);
                        s0 += 1.0;
                        s1 += sv[0][q];
                        s2 += sv[1][q];
                        s3 += sv[2][q];
                    }
                    lacc[0][gv] += s0;
                    lacc[1][gv] += s1;
                    lacc[2][gv] += s2;
                    lacc[3][gv] += s3;
                }
            }
            __syncthreads();
        }
        for (uint32_t i = threadIdx.x; i < cn; i += kT)
            for (int k = 0; k < 4; k++) mine[k * slots + c0 + i] = lacc[k][i];
        __syncthreads();
    }
}

// stats[4 g ..]: one wave per group slot adds the blocks' partials (lane l
// takes blocks l, l + 64, ..., then a fixed butterfly), then the means
__global__ __launch_bounds__(kT) void k_err_final(const double *__restrict__ partial,
                                                  uint32_t blocks, uint32_t G,
                                                  uint32_t with_groups, double *__restrict__ stats)
{
    const uint64_t slots = (uint64_t)G + 1;
    const uint64_t g = (uint64_t)blockIdx.x * (kT / 64) + (threadIdx.x >> 6);
    if (g >= slots) return;
    const uint32_t lane = (uint32_t)lane_id();
    double s[4] = {0.0, 0.0, 0.0, 0.0};
    if (g == G || with_groups)
        for (uint32_t b = lane; b < blocks; b += 64)
#pragma unroll
            for (int k = 0; k < 4; k++) s[k] += partial[((uint64_t)b * 4 + k) * slots + g];
#pragma unroll
    for (int k = 0; k < 4; k++)
        for (int off = 32; off >= 1; off >>= 1) s[k] += __shfl_xor(s[k], off, 64);
    if (lane != 0) return;
    stats[4 * g + 0] = s[0];
    if (s[0] > 0.0) {
        stats[4 * g + 1] = s[1] / s[0];
        const double m2 = s[2] / s[0];
        stats[4 * g + 2] = sqrt(m2);
        stats[4 * g + 3] = s[3] / s[0];
    } else {
        const double nan = __builtin_nan("");
        stats[4 * g + 1] = nan;
        stats[4 * g + 2] = nan;
        stats[4 * g + 3] = nan;
    }
}

__global__ void k_err_validate(uint64_t n, const uint32_t *__restrict__ group, uint32_t G,
                               uint32_t *__restrict__ flag)
{
    uint32_t bad = 0;
    for (uint64_t e = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (uint64_t)gridDim.x * blockDim.x)
        if (group[e] >= G) bad = 1;
    if (bad) atomicOr(flag, 1u);
}

// hist[c * 3 + k]: requests of category c in class k
__global__ __launch_bounds__(kT) void k_class_hist(uint32_t n, const uint8_t *__restrict__ category,
                                                   uint32_t n_cat, const uint8_t *__restrict__ cls,
                                                   uint32_t *__restrict__ hist)
{
    __shared__ uint32_t h[256 * 3];
    const uint32_t cells = n_cat * 3;
    for (uint32_t i = threadIdx.x; i < cells; i += kT) h[i] = 0;
    __syncthreads();
    for (uint32_t i = blockIdx.x * kT + threadIdx.x; i < n; i += gridDim.x * kT) {
        const uint32_t c = category[i], k = cls[i];
        if (c < n_cat && k < 3) atomicAdd(&h[c * 3 + k], 1u);
    }
    __syncthreads();
    for (uint32_t i = threadIdx.x; i < cells; i += kT)
        if (h[i]) atomicAdd(&hist[i], h[i]);
}

__global__ void k_hist_validate(uint32_t n, const uint8_t *__restrict__ category, uint32_t n_cat,
                                const uint8_t *__restrict__ cls, uint32_t *__restrict__ flag)
{
    uint32_t bad = 0;
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
        if (category[i] >= n_cat || cls[i] > 2) bad = 1;
    if (bad) atomicOr(flag, 1u);
}

uint32_t blocks_for(uint64_t n, uint32_t cap)
{
    uint64_t b = cdiv(n, kT);
    return (uint32_t)(b < 1 ? 1 : (b > cap ? cap : b));
}

}  // namespace

// Blocks of the error kernel: about 2048 events each, at most kMaxBlocks,
// and fewer when the partial sums of many groups would be large.
static uint32_t err_blocks(uint64_t n, uint32_t G)
{
    uint64_t b = cdiv(n ? n : 1, 2048);
    const uint64_t cap = (1ull << 22) / ((uint64_t)G + 1);   // <= 128 MB of partials
    if (b > kMaxBlocks) b = kMaxBlocks;
    if (b > cap) b = cap;
    return (uint32_t)(b < 1 ? 1 : b);
}

size_t err_ws_bytes(uint64_t n, uint32_t n_groups)
{
    return align_up((uint64_t)err_blocks(n, n_groups) * 4 * ((uint64_t)n_groups + 1) * 8, 256);
}

hipError_t err_launch(uint64_t n, const double *est, const double *factor, const uint32_t *obs,
                      const uint32_t *group, uint32_t G, double *stats, void *ws, uint32_t *flag,
                      hipStream_t s)
{
    if (flag) {
        if (group && n)
            hipLaunchKernelGGL(k_err_validate, dim3(blocks_for(n, 1024)), dim3(kT), 0, s, n, group,
                               G, flag);
        return hipGetLastError();
    }
    double *partial = static_cast<double *>(ws);
    const uint32_t blocks = err_blocks(n, G);
    hipLaunchKernelGGL(k_err_accum, dim3(blocks), dim3(kT), 0, s, n, est, factor, obs, group, G,
                       partial);
    hipLaunchKernelGGL(k_err_final, dim3((uint32_t)cdiv((uint64_t)G + 1, kT / 64)), dim3(kT), 0, s,
                       (const double *)partial, blocks, G, group ? 1u : 0u, stats);
    return hipGetLastError();
}

hipError_t hist_launch(uint32_t n, const uint8_t *category, uint32_t n_cat, const uint8_t *cls,
                       uint32_t *hist, uint32_t *flag, hipStream_t s)
{
    if (flag) {
        if (n)
            hipLaunchKernelGGL(k_hist_validate, dim3(blocks_for(n, 1024)), dim3(kT), 0, s, n,
                               category, n_cat, cls, flag);
        return hipGetLastError();
    }
    hipError_t e = fill_u32(hist, 0u, (uint64_t)n_cat * 3, s);
    if (e != hipSuccess) return e;
    if (n)
        hipLaunchKernelGGL(k_class_hist, dim3(blocks_for(n, 1024)), dim3(kT), 0, s, n, category,
                           n_cat, cls, hist);
    return hipGetLastError();
}

}  // namespace ds
