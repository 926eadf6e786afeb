// Evolution layer (Section 4.2) on one GPU: ensemble fusion, the
// evaluator's fitness and keep-best bookkeeping, the selector.  All are
// memory-bound passes over parameter vectors or reward rows; every
// reduction runs in a fixed order, so results are deterministic.
#include "device.hpp"
#include "internal.hpp"

namespace tpk {

namespace {

constexpr int EV_THREADS = 256;

int grid_over(int64_t n, int cap = 65535)
{
    const int64_t g = (n + EV_THREADS - 1) / EV_THREADS;
    return (int)(g < cap ? (g > 0 ? g : 1) : cap);
}

// fused[g][k][p] = mean over k of params[g][k][p]; grid-stride over (g, p)
__global__ __launch_bounds__(EV_THREADS) void fuse_kernel(float *__restrict__ params, int N, int K,
                                                         int64_t P)
{
    const int64_t total = (int64_t)N * P;
    for (int64_t i = blockIdx.x * (int64_t)EV_THREADS + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * EV_THREADS) {
        const int64_t g = i / P, p = i % P;
        float *base = params + (size_t)g * K * P + p;
        double s = 0.0;
        for (int k = 0; k < K; ++k) s += (double)base[(size_t)k * P];
        const float m = (float)(s / (double)K);
        for (int k = 0; k < K; ++k) base[(size_t)k * P] = m;
    }
}

// Per env: its discounted return (or NaN if any reward is NaN), written to
// ret[e]; consecutive threads read consecutive envs of each reward row.
__global__ __launch_bounds__(EV_THREADS) void env_return_kernel(const float *__restrict__ r, int L,
                                                               int E, double gamma,
                                                               double *__restrict__ ret)
{
    const int e = blockIdx.x * EV_THREADS + threadIdx.x;
    if (e >= E) return;
    double acc = 0.0, disc = 1.0;
    bool ok = true;
    // loads of a block of steps are issued together; the sum keeps step order
    constexpr int U = 16;
    int j = 0;
    for (; j + U <= L; j += U) {
        float x[U];
#pragma unroll
        for (int u = 0; u < U; ++u) x[u] = r[(size_t)(j + u) * E + e];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            ok &= !isnan(x[u]);
            acc += disc * (double)x[u];
            disc *= gamma;
        }
    }
    for (; j < L; ++j) {
        const float x = r[(size_t)j * E + e];
        ok &= !isnan(x);
        acc += disc * (double)x;
        disc *= gamma;
    }
    ret[e] = ok ? acc : __builtin_nan("");
}

// Per agent (one workgroup): the mean of its envs' returns, NaN ones left
// out, summed in env order by one lane.
__global__ __launch_bounds__(64) void agent_mean_kernel(const double *__restrict__ ret, int epa,
                                                       double *__restrict__ fit)
{
    if (threadIdx.x != 0) return;
    const int g = blockIdx.x;
    double s = 0.0;
    int cnt = 0;
    const double *p = ret + (size_t)g * epa;
    constexpr int U = 16;
    int e = 0;
    for (; e + U <= epa; e += U) {
        double x[U];
#pragma unroll
        for (int u = 0; u < U; ++u) x[u] = p[e + u];
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (!isnan(x[u])) {
                s += x[u];
                ++cnt;
            }
    }
    for (; e < epa; ++e) {
        const double x = p[e];
        if (!isnan(x)) {
            s += x;
            ++cnt;
        }
    }
    fit[g] = cnt ? s / (double)cnt : __builtin_nan("");
}

__device__ __forceinline__ bool beats(double f, double b)
{
    return !isnan(f) && (isnan(b) || f > b);
}

// Copy the parameters of improved agents (decided from the unchanged best).
__global__ __launch_bounds__(EV_THREADS) void keep_copy_kernel(const double *__restrict__ fit,
                                                              const double *__restrict__ best,
                                                              const float *__restrict__ params,
                                                              float *__restrict__ best_params,
                                                              int A, int64_t P)
{
    const int64_t total = (int64_t)A * P;
    for (int64_t i = blockIdx.x * (int64_t)EV_THREADS + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * EV_THREADS) {
        const int g = (int)(i / P);
        if (beats(fit[g], best[g])) best_params[i] = params[i];
    }
}

// Then the scalars (after the copies, on the same stream).
__global__ __launch_bounds__(EV_THREADS) void keep_update_kernel(const double *__restrict__ fit,
                                                                double *__restrict__ best,
                                                                int32_t *__restrict__ stall, int A)
{
    const int g = blockIdx.x * EV_THREADS + threadIdx.x;
    if (g >= A) return;
    if (beats(fit[g], best[g])) {
        best[g] = fit[g];
        stall[g] = 0;
    } else {
        stall[g] += 1;
    }
}

// rank[i] = number of agents ordered before i (fitness descending, NaN
// last, ties to the lower index)
__global__ __launch_bounds__(1024) void rank_kernel(const double *__restrict__ fit, int N,
                                                   int32_t *__restrict__ rank)
{
    const int i = threadIdx.x;
    if (i >= N) return;
    const double fi = fit[i];
    int r = 0;
    for (int j = 0; j < N; ++j) {
        const double fj = fit[j];
        bool before;
        if (isnan(fj)) before = isnan(fi) && j < i;
        else if (isnan(fi)) before = true;
        else before = fj > fi || (fj == fi && j < i);
        r += before;
    }
    rank[i] = r;
}

// Workgroup-row i (grid-stride over P): a non-survivor i takes the
// parameters of the survivor of rank (rank[i] - keep) mod keep.
__global__ __launch_bounds__(EV_THREADS) void select_copy_kernel(const int32_t *__restrict__ rank,
                                                                float *__restrict__ params, int N,
                                                                int64_t P, int keep)
{
    const int i = blockIdx.y;
    const int r = rank[i];
    if (r < keep) return;
    const int want = (r - keep) % keep;
    int src = 0;
    for (int j = 0; j < N; ++j)
        if (rank[j] == want) src = j;
    const float *s = params + (size_t)src * P;
    float *d = params + (size_t)i * P;
    for (int64_t p = blockIdx.x * (int64_t)EV_THREADS + threadIdx.x; p < P;
         p += (int64_t)gridDim.x * EV_THREADS)
        d[p] = s[p];
}

}  // namespace

hipError_t launch_ensemble_fuse(float *params, int N, int K, int64_t P, hipStream_t s)
{
    hipLaunchKernelGGL(fuse_kernel, dim3(grid_over((int64_t)N * P)), dim3(EV_THREADS), 0, s,
                       params, N, K, P);
    return hipGetLastError();
}

hipError_t launch_fitness(const float *r, int L, int E, int A, double gamma, double *fit,
                          double *env_return, hipStream_t s)
{
    hipLaunchKernelGGL(env_return_kernel, dim3((E + EV_THREADS - 1) / EV_THREADS),
                       dim3(EV_THREADS), 0, s, r, L, E, gamma, env_return);
    hipLaunchKernelGGL(agent_mean_kernel, dim3(A), dim3(64), 0, s, env_return, E / A, fit);
    return hipGetLastError();
}

hipError_t launch_keep_best(const double *fit, double *best, int32_t *stall, const float *params,
                            float *best_params, int A, int64_t P, hipStream_t s)
{
    hipLaunchKernelGGL(keep_copy_kernel, dim3(grid_over((int64_t)A * P)), dim3(EV_THREADS), 0, s,
                       fit, best, params, best_params, A, P);
    hipLaunchKernelGGL(keep_update_kernel, dim3((A + EV_THREADS - 1) / EV_THREADS),
                       dim3(EV_THREADS), 0, s, fit, best, stall, A);
    return hipGetLastError();
}

hipError_t launch_select(const double *fit, float *params, int N, int64_t P, int keep,
                         int32_t *rank, hipStream_t s)
{
    hipLaunchKernelGGL(rank_kernel, dim3(1), dim3(1024), 0, s, fit, N, rank);
    const int gx = grid_over(P, 1024);
    hipLaunchKernelGGL(select_copy_kernel, dim3(gx, N), dim3(EV_THREADS), 0, s, rank, params, N,
                       P, keep);
    return hipGetLastError();
}

}  // namespace tpk
