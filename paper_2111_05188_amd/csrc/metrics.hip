// Backtest metrics of total-asset series (Section 5.2, "Evaluation
// metrics"): one thread per env walks its series V_0 .. V_T; consecutive
// threads read consecutive envs of a time row, so every pass over the
// time-major [T][E] array is coalesced.  Two passes (mean, then the sum of
// squared deviations) in fp64, the order a plain serial evaluation uses.
#include "device.hpp"
#include "internal.hpp"

namespace tpk {

namespace {

constexpr int MET_THREADS = 256;

__global__ __launch_bounds__(MET_THREADS) void backtest_metrics_kernel(
    const double *__restrict__ v0, const double *__restrict__ v, int T, int E, double P,
    double rf, double *__restrict__ out)
{
    const int e = blockIdx.x * MET_THREADS + threadIdx.x;
    if (e >= E) return;
    const size_t ld = (size_t)E;
    // pass 1: mean return, final value, drawdown against the running peak
    const double first = v0[e];
    double prev = first, sum = 0.0, peak = first, mdd = 0.0;
    for (int t = 0; t < T; ++t) {
        const double cur = v[t * ld + e];
        sum += cur / prev - 1.0;
        if (cur > peak) peak = cur;
        const double dd = (peak - cur) / peak;
        if (dd > mdd) mdd = dd;
        prev = cur;
    }
    const double last = prev;
    const double mean = sum / (double)T;
    // pass 2: sample variance of the returns
    double ss = 0.0;
    prev = first;
    for (int t = 0; t < T; ++t) {
        const double cur = v[t * ld + e];
        const double d = (cur / prev - 1.0) - mean;
        ss += d * d;
        prev = cur;
    }
    const double sd = T > 1 ? sqrt(ss / (double)(T - 1)) : 0.0;
    double *o = out + (size_t)e * 5;
    o[0] = last / first - 1.0;
    o[1] = pow(last / first, P / (double)T) - 1.0;
    o[2] = sd * sqrt(P);
    o[3] = sd > 0.0 ? (mean - rf / P) / sd * sqrt(P) : 0.0;
    o[4] = mdd;
}

}  // namespace

hipError_t launch_backtest_metrics(const double *v0, const double *v, int T, int E,
                                   double periods_per_year, double risk_free, double *out,
                                   hipStream_t s)
{
    hipLaunchKernelGGL(backtest_metrics_kernel, dim3((E + MET_THREADS - 1) / MET_THREADS),
                       dim3(MET_THREADS), 0, s, v0, v, T, E, periods_per_year, risk_free, out);
    return hipGetLastError();
}

}  // namespace tpk
