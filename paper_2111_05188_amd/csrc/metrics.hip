// Backtest metrics of total-asset series (Section 5.2, "Evaluation
// metrics"), time-parallel.  A workgroup of 1024 threads takes EB
// consecutive envs and splits each env's series V_1 .. V_T into TC = 1024/EB
// contiguous time chunks, one per thread; lanes with the same chunk read
// consecutive envs of a time row.  EB is chosen per launch: wide groups
// (whole cache lines of a row) when there are many envs, one env per
// workgroup with 1024 time lanes when a few envs have long series.
//
// Pass 1: per chunk, the sum of its returns r_t = V_t / V_{t-1} - 1 and its
// largest value; an LDS tree sums the returns per env (the mean) and an
// LDS scan gives each chunk the running peak of everything before it.
// Pass 2: per chunk, the squared deviations from the mean and the drawdown
// (peak_t - V_t) / peak_t with the running peak seeded from the scan, so
// every drawdown term is computed from the operands a serial walk uses and
// the maximum is exact; only the two sums are reassociated (a fixed tree,
// deterministic).
#include "device.hpp"
#include "internal.hpp"

namespace tpk {

namespace {

constexpr int MET_THREADS = 1024;

__global__ __launch_bounds__(MET_THREADS) void backtest_metrics_kernel(
    const double *__restrict__ v0, const double *__restrict__ v, int T, int E, double P,
    double rf, double *__restrict__ out, int eb_log2)
{
    __shared__ double s_a[MET_THREADS];
    __shared__ double s_b[MET_THREADS];
    const int EB = 1 << eb_log2, TC = MET_THREADS >> eb_log2;
    const int tid = threadIdx.x;
    const int eb = tid & (EB - 1), tc = tid >> eb_log2;
    const int e = blockIdx.x * EB + eb;
    const bool act = e < E;
    const int CL = (T + TC - 1) / TC;
    const int t0 = min(T, tc * CL), t1 = min(T, t0 + CL);
    const size_t ld = (size_t)E;
    const double *col = v + (act ? e : 0);

    const double first = act ? v0[e] : 1.0;
    const double start = (act && t0 > 0 && t0 < T) ? col[(size_t)(t0 - 1) * ld] : first;

    // pass 1: chunk return sum and chunk maximum
    double prev = start, sum = 0.0, cmax = -__builtin_inf();
    if (act) {
#pragma unroll 4
        for (int t = t0; t < t1; ++t) {
            const double cur = col[(size_t)t * ld];
            sum += cur / prev - 1.0;
            if (cur > cmax) cmax = cur;
            prev = cur;
        }
    }
    s_a[tid] = sum;
    s_b[tid] = cmax;
    __syncthreads();
    // inclusive max-scan over the chunks of each env (Hillis-Steele)
    for (int o = 1; o < TC; o <<= 1) {
        const double other = tc >= o ? s_b[tid - o * EB] : -__builtin_inf();
        __syncthreads();
        if (other > s_b[tid]) s_b[tid] = other;
        __syncthreads();
    }
    // tree sum of the chunk return sums
    for (int o = TC >> 1; o >= 1; o >>= 1) {
        if (tc < o) s_a[tid] += s_a[tid + o * EB];
        __syncthreads();
    }
    const double mean = s_a[eb] / (double)T;
    double peak = first;
    if (tc > 0 && s_b[tid - EB] > peak) peak = s_b[tid - EB];
    __syncthreads();

    // pass 2: squared deviations and drawdowns over the same chunk
    prev = start;
    double ss = 0.0, mdd = 0.0;
    if (act) {
#pragma unroll 4
        for (int t = t0; t < t1; ++t) {
            const double cur = col[(size_t)t * ld];
            const double d = (cur / prev - 1.0) - mean;
            ss += d * d;
            if (cur > peak) peak = cur;
            const double dd = (peak - cur) / peak;
            if (dd > mdd) mdd = dd;
            prev = cur;
        }
    }
    s_a[tid] = ss;
    s_b[tid] = mdd;
    __syncthreads();
    for (int o = TC >> 1; o >= 1; o >>= 1) {
        if (tc < o) {
            s_a[tid] += s_a[tid + o * EB];
            if (s_b[tid + o * EB] > s_b[tid]) s_b[tid] = s_b[tid + o * EB];
        }
        __syncthreads();
    }
    if (tc != 0 || !act) return;
    const double last = col[(size_t)(T - 1) * ld];
    const double sd = T > 1 ? sqrt(s_a[tid] / (double)(T - 1)) : 0.0;
    double *o = out + (size_t)e * 5;
    o[0] = last / first - 1.0;
    o[1] = pow(last / first, P / (double)T) - 1.0;
    o[2] = sd * sqrt(P);
    o[3] = sd > 0.0 ? (mean - rf / P) / sd * sqrt(P) : 0.0;
    o[4] = s_b[tid];
}

// log2 of the envs per workgroup: at least 256 workgroups while envs allow,
// whole 64-env rows when there are many envs, and no more time lanes than a
// quarter of the series length.
int metrics_eb_log2(int T, int E)
{
    int lg = 0;
    while (lg < 6 && ((int64_t)E >> (lg + 1)) >= 256) ++lg;
    const int lanes_max = T / 4 > 1 ? T / 4 : 1;
    while (lg < 6 && (MET_THREADS >> lg) > lanes_max) ++lg;
    return lg;
}

}  // namespace

hipError_t launch_backtest_metrics(const double *v0, const double *v, int T, int E,
                                   double periods_per_year, double risk_free, double *out,
                                   hipStream_t s)
{
    const int lg = metrics_eb_log2(T, E);
    const int eb = 1 << lg;
    hipLaunchKernelGGL(backtest_metrics_kernel, dim3((E + eb - 1) / eb), dim3(MET_THREADS), 0, s,
                       v0, v, T, E, periods_per_year, risk_free, out, lg);
    return hipGetLastError();
}

}  // namespace tpk
