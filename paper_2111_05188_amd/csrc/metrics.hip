// Backtest metrics of total-asset series (Section 5.2, "Evaluation
// metrics").  Many envs: one launch, a workgroup per group of envs (see
// metrics_onepass_kernel).  Few envs with long series: split over time so
// that they still fill the GPU, as follows.
//
// Geometry: a workgroup of 256 threads takes EB consecutive envs (a power of
// two, at most 64: 16 or more envs make every row access whole 128-byte
// lines) and one segment of SL = TC x CL consecutive steps, TC = 256 / EB
// time lanes each walking a chunk of CL steps.  Segments are sized so that
// the grid has about 1024 workgroups.
//
// Three launches over a caller-provided workspace:
//   1. per segment: the sum of its returns r_t = V_t / V_{t-1} - 1, its
//      largest value, and each chunk's largest value;
//   2. per segment: every workgroup of an env group computes the envs' mean
//      return from the segment sums (lanes stride over the segments, then a
//      fixed LDS tree, so all workgroups agree) and the running peak before
//      its segment (earlier segments' maxima, then earlier chunks'); each
//      lane then walks its chunk once for the squared deviations and the
//      drawdowns (peak_t - V_t) / peak_t, seeded with that peak, so every
//      drawdown term has the operands of a serial walk and their maximum is
//      exact;
//   3. per env: the segments' squared deviations summed in segment order,
//      their largest drawdown, and the five metrics.
// Only the sums are reassociated (fixed order, deterministic).
#include <mutex>

#include "device.hpp"
#include "internal.hpp"

namespace tpk {

// Static device scratch for tp_backtest_metrics_noalloc (callers that cannot
// allocate).  Every shape the three-launch path takes needs at most
// 8 (4 s + s TC + E) bytes with s = nseg E <= 1024 EB and s TC <= 2^18, i.e.
// below 4.2 MiB; 4.5 MiB covers it.  Each GPU holds its own copy until the
// process ends.  In host code `scratch` names a host-side stand-in: its
// device address is taken once per device with hipGetSymbolAddress.
constexpr size_t METRICS_SCRATCH_BYTES = (size_t)9 << 19;   // 4.5 MiB
static __device__ __align__(256) double scratch[METRICS_SCRATCH_BYTES / sizeof(double)];

namespace {

constexpr int MT = 256;

struct MetGeo {
    int eb_log2, EB, TC, CL, SL, nseg, ngroups;
};

int pow2_ceil(int x)
{
    int p = 1;
    while (p < x) p <<= 1;
    return p;
}

MetGeo metrics_geometry(int T, int E)
{
    MetGeo g;
    g.EB = pow2_ceil(E < 64 ? E : 64);
    g.eb_log2 = 0;
    while ((1 << g.eb_log2) < g.EB) ++g.eb_log2;
    g.TC = MT / g.EB;
    g.ngroups = (E + g.EB - 1) / g.EB;
    int target = 1024 / g.ngroups;
    if (target < 1) target = 1;
    const int sl = (T + target - 1) / target;
    g.CL = (sl + g.TC - 1) / g.TC;
    if (g.CL < 1) g.CL = 1;
    g.SL = g.CL * g.TC;
    g.nseg = (T + g.SL - 1) / g.SL;
    return g;
}

// workspace arrays, each [nseg][E] doubles except cmax [nseg * TC][E] and
// mean [E]
struct MetWork {
    double *psum, *pmax, *pss, *pmdd, *cmax, *mean;
};

MetWork carve(void *work, const MetGeo &g, int E)
{
    double *w = (double *)work;
    const size_t se = (size_t)g.nseg * E;
    MetWork m;
    m.psum = w;
    m.pmax = w + se;
    m.pss = w + 2 * se;
    m.pmdd = w + 3 * se;
    m.cmax = w + 4 * se;
    m.mean = w + 4 * se + se * g.TC;
    return m;
}

struct Lane {
    int eb, tc, e, t0, t1;
    bool act;
};

__device__ __forceinline__ Lane lane_of(const MetGeo &g, int T, int E)
{
    Lane l;
    const int tid = threadIdx.x;
    l.eb = tid & (g.EB - 1);
    l.tc = tid >> g.eb_log2;
    l.e = blockIdx.y * g.EB + l.eb;
    l.act = l.e < E;
    const int s0 = blockIdx.x * g.SL;
    l.t0 = min(T, s0 + l.tc * g.CL);
    l.t1 = min(T, l.t0 + g.CL);
    return l;
}

__global__ __launch_bounds__(MT) void metrics_pass1_kernel(const double *__restrict__ v0,
                                                           const double *__restrict__ v, int T,
                                                           int E, MetGeo g, MetWork w)
{
    __shared__ double s_a[MT];
    __shared__ double s_b[MT];
    const Lane l = lane_of(g, T, E);
    const int tid = threadIdx.x;
    const size_t ld = (size_t)E;
    double sum = 0.0, cmax = -__builtin_inf();
    if (l.act && l.t0 < l.t1) {
        const double *col = v + l.e;
        double prev = l.t0 > 0 ? col[(size_t)(l.t0 - 1) * ld] : v0[l.e];
#pragma unroll 4
        for (int t = l.t0; t < l.t1; ++t) {
            const double cur = col[(size_t)t * ld];
            sum += cur / prev - 1.0;
            if (cur > cmax) cmax = cur;
            prev = cur;
        }
    }
    if (l.act) w.cmax[((size_t)blockIdx.x * g.TC + l.tc) * ld + l.e] = cmax;
    s_a[tid] = sum;
    s_b[tid] = cmax;
    __syncthreads();
    for (int o = g.TC >> 1; o >= 1; o >>= 1) {
        if (l.tc < o) {
            s_a[tid] += s_a[tid + o * g.EB];
            if (s_b[tid + o * g.EB] > s_b[tid]) s_b[tid] = s_b[tid + o * g.EB];
        }
        __syncthreads();
    }
    if (l.tc == 0 && l.act) {
        w.psum[(size_t)blockIdx.x * ld + l.e] = s_a[tid];
        w.pmax[(size_t)blockIdx.x * ld + l.e] = s_b[tid];
    }
}

__global__ __launch_bounds__(MT) void metrics_pass2_kernel(const double *__restrict__ v0,
                                                           const double *__restrict__ v, int T,
                                                           int E, MetGeo g, MetWork w)
{
    __shared__ double s_a[MT];
    __shared__ double s_b[MT];
    const Lane l = lane_of(g, T, E);
    const int tid = threadIdx.x;
    const size_t ld = (size_t)E;
    const int seg = blockIdx.x;
    // mean over all segments and peak over earlier ones, lanes striding
    double sum = 0.0, peak = -__builtin_inf();
    if (l.act) {
        for (int s = l.tc; s < g.nseg; s += g.TC) {
            sum += w.psum[(size_t)s * ld + l.e];
            if (s < seg) {
                const double m = w.pmax[(size_t)s * ld + l.e];
                if (m > peak) peak = m;
            }
        }
    }
    s_a[tid] = sum;
    s_b[tid] = peak;
    __syncthreads();
    for (int o = g.TC >> 1; o >= 1; o >>= 1) {
        if (l.tc < o) {
            s_a[tid] += s_a[tid + o * g.EB];
            if (s_b[tid + o * g.EB] > s_b[tid]) s_b[tid] = s_b[tid + o * g.EB];
        }
        __syncthreads();
    }
    const double mean = s_a[l.eb] / (double)T;
    const double first = l.act ? v0[l.e] : 1.0;
    double pk = first;
    if (s_b[l.eb] > pk) pk = s_b[l.eb];
    __syncthreads();
    // exclusive max-scan of this segment's chunk maxima (Hillis-Steele)
    s_b[tid] = l.act ? w.cmax[((size_t)seg * g.TC + l.tc) * ld + l.e] : -__builtin_inf();
    __syncthreads();
    for (int o = 1; o < g.TC; o <<= 1) {
        const double other = l.tc >= o ? s_b[tid - o * g.EB] : -__builtin_inf();
        __syncthreads();
        if (other > s_b[tid]) s_b[tid] = other;
        __syncthreads();
    }
    if (l.tc > 0 && s_b[tid - g.EB] > pk) pk = s_b[tid - g.EB];
    if (seg == 0 && l.tc == 0 && l.act) w.mean[l.e] = mean;
    // the chunk: squared deviations and drawdowns
    double ss = 0.0, mdd = 0.0;
    if (l.act && l.t0 < l.t1) {
        const double *col = v + l.e;
        double prev = l.t0 > 0 ? col[(size_t)(l.t0 - 1) * ld] : first;
#pragma unroll 4
        for (int t = l.t0; t < l.t1; ++t) {
            const double cur = col[(size_t)t * ld];
            const double d = (cur / prev - 1.0) - mean;
            ss += d * d;
            if (cur > pk) pk = cur;
            const double dd = (pk - cur) / pk;
            if (dd > mdd) mdd = dd;
            prev = cur;
        }
    }
    __syncthreads();
    s_a[tid] = ss;
    s_b[tid] = mdd;
    __syncthreads();
    for (int o = g.TC >> 1; o >= 1; o >>= 1) {
        if (l.tc < o) {
            s_a[tid] += s_a[tid + o * g.EB];
            if (s_b[tid + o * g.EB] > s_b[tid]) s_b[tid] = s_b[tid + o * g.EB];
        }
        __syncthreads();
    }
    if (l.tc == 0 && l.act) {
        w.pss[(size_t)seg * ld + l.e] = s_a[tid];
        w.pmdd[(size_t)seg * ld + l.e] = s_b[tid];
    }
}

// one workgroup per env group: lanes stride over the segments
__global__ __launch_bounds__(MT) void metrics_final_kernel(const double *__restrict__ v0,
                                                           const double *__restrict__ v, int T,
                                                           int E, double P, double rf, MetGeo g,
                                                           MetWork w, double *__restrict__ out)
{
    __shared__ double s_a[MT];
    __shared__ double s_b[MT];
    const int tid = threadIdx.x;
    const int eb = tid & (g.EB - 1), tc = tid >> g.eb_log2;
    const int e = blockIdx.x * g.EB + eb;
    const bool act = e < E;
    const size_t ld = (size_t)E;
    double ss = 0.0, mdd = 0.0;
    if (act) {
        for (int s = tc; s < g.nseg; s += g.TC) {
            ss += w.pss[(size_t)s * ld + e];
            const double m = w.pmdd[(size_t)s * ld + e];
            if (m > mdd) mdd = m;
        }
    }
    s_a[tid] = ss;
    s_b[tid] = mdd;
    __syncthreads();
    for (int o = g.TC >> 1; o >= 1; o >>= 1) {
        if (tc < o) {
            s_a[tid] += s_a[tid + o * g.EB];
            if (s_b[tid + o * g.EB] > s_b[tid]) s_b[tid] = s_b[tid + o * g.EB];
        }
        __syncthreads();
    }
    if (tc != 0 || !act) return;
    const double first = v0[e], last = v[(size_t)(T - 1) * ld + e];
    const double mean = w.mean[e];
    const double sd = T > 1 ? sqrt(s_a[tid] / (double)(T - 1)) : 0.0;
    double *o = out + (size_t)e * 5;
    o[0] = last / first - 1.0;
    o[1] = pow(last / first, P / (double)T) - 1.0;
    o[2] = sd * sqrt(P);
    o[3] = sd > 0.0 ? (mean - rf / P) / sd * sqrt(P) : 0.0;
    o[4] = s_b[tid];
}

// ---------------------------------------------------------------------------
// One launch, when the envs alone give the GPU enough workgroups: a
// workgroup of 1024 threads takes EB envs and splits each series into
// 1024 / EB contiguous chunks; pass 1 (chunk return sums and maxima), an LDS
// tree (the mean) and an LDS max-scan (the peak before each chunk), then
// pass 2 over the same chunks (squared deviations, exact drawdowns).
// ---------------------------------------------------------------------------
constexpr int MET_THREADS = 1024;

__global__ __launch_bounds__(MET_THREADS) void metrics_onepass_kernel(
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

size_t backtest_metrics_work_bytes(int T, int E)
{
    const MetGeo g = metrics_geometry(T, E);
    const size_t se = (size_t)g.nseg * E;
    return sizeof(double) * (4 * se + se * g.TC + (size_t)E);
}

static bool metrics_one_launch(int T, int E)
{
    const int lg = metrics_eb_log2(T, E);
    return ((E + (1 << lg) - 1) >> lg) >= 256;
}

size_t backtest_metrics_scratch_needed(int T, int E)
{
    return metrics_one_launch(T, E) ? 0 : backtest_metrics_work_bytes(T, E);
}

size_t backtest_metrics_scratch_capacity() { return METRICS_SCRATCH_BYTES; }

hipError_t backtest_metrics_scratch(void **ptr)
{
    constexpr int MAX_DEV = 64;
    static std::mutex mu;
    static void *addr[MAX_DEV] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= MAX_DEV) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> g(mu);
    if (!addr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    return hipSuccess;
}

hipError_t launch_backtest_metrics(const double *v0, const double *v, int T, int E,
                                   double periods_per_year, double risk_free, double *out,
                                   void *work, hipStream_t s)
{
    {
        const int lg = metrics_eb_log2(T, E);
        const int blocks = (E + (1 << lg) - 1) >> lg;
        if (blocks >= 256) {   // metrics_one_launch
            hipLaunchKernelGGL(metrics_onepass_kernel, dim3(blocks), dim3(MET_THREADS), 0, s, v0, v,
                               T, E, periods_per_year, risk_free, out, lg);
            return hipGetLastError();
        }
    }
    const MetGeo g = metrics_geometry(T, E);
    const MetWork w = carve(work, g, E);
    const dim3 grid(g.nseg, g.ngroups);
    hipLaunchKernelGGL(metrics_pass1_kernel, grid, dim3(MT), 0, s, v0, v, T, E, g, w);
    hipLaunchKernelGGL(metrics_pass2_kernel, grid, dim3(MT), 0, s, v0, v, T, E, g, w);
    hipLaunchKernelGGL(metrics_final_kernel, dim3(g.ngroups), dim3(MT), 0, s, v0, v, T, E,
                       periods_per_year, risk_free, g, w, out);
    return hipGetLastError();
}

}  // namespace tpk
