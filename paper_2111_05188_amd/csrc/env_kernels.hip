// Standalone env kernels: reset and one teacher-forced step.
// Each 64-lane wave owns two envs (one per 32-lane half, 4 stocks per lane);
// observation rows are assembled in LDS and written with 16-byte stores.
#include "device.hpp"
#include "env.hpp"
#include "internal.hpp"

namespace tpk {

constexpr int ENV_WPB = 4;              // waves per workgroup
// rounds of 16-byte indicator chunks a lane holds: n * n_ind <= 1024 gives
// at most 257 chunks of 4 (with the shifted first column), 9 rounds of 32
constexpr int ENV_IND_ROUNDS = 9;
constexpr int ENV_EPB = 2 * ENV_WPB;    // envs per workgroup

template <typename OT>
__device__ __forceinline__ int obs_ld_lds(const EnvConst &C)
{
    return (C.K_pad * (int)sizeof(OT) + 15) / 16 * 16 / (int)sizeof(OT);
}

// An env the call cannot start or step adds one to *n_invalid (lane 0 of
// its half; an integer count, so the total does not depend on the order).
__device__ __forceinline__ void count_invalid(int32_t *n_invalid, bool bad, int hl)
{
    if (n_invalid && bad && hl == 0) atomicAdd(n_invalid, 1);
}

__global__ void zero_i32_kernel(int32_t *p) { *p = 0; }

template <typename OT>
__global__ __launch_bounds__(ENV_WPB *WAVE) void env_reset_kernel(
    EnvConst C, double *cash, int32_t *shares, int64_t *t, const int64_t *t0,
    int E, OT *obs, int64_t ld_obs, int32_t *n_invalid)
{
    extern __shared__ __align__(16) uint8_t smem[];
    const int lane = threadIdx.x % WAVE, hl = lane % HALF;
    const int slot = threadIdx.x / HALF;               // env of this half in the block
    const int e = blockIdx.x * ENV_EPB + slot;
    OT *row = (OT *)smem + slot * obs_ld_lds<OT>(C);
    if (e < E) {
        const int n = C.n;
        const int64_t tt = t0[e];
        const bool ok = tt >= 0 && tt < C.T1 - 1;
        count_invalid(n_invalid, !ok, hl);
        for (int i = hl; i < n; i += HALF) shares[(size_t)e * n + i] = 0;
        if (hl == 0) {
            cash[e] = C.cash0;
            t[e] = ok ? tt : -1;
        }
        if (obs) {
            if (ok) {
                const float *prow = C.price + (size_t)tt * n;
                const float *irow = C.ind + (size_t)tt * C.nI;
                int h[SPL];
                float p[SPL], ind1[1];
#pragma unroll
                for (int c = 0; c < SPL; ++c) {
                    const int i = SPL * hl + c;
                    h[c] = 0;
                    p[c] = i < n ? prow[i] : 0.f;
                }
                ind1[0] = hl < C.nI ? irow[hl] : 0.f;
                write_obs_half<OT, 1>(row, C, C.cash0, h, p, ind1, irow, hl);
            } else {
                for (int k = hl; k < C.K_pad; k += HALF) row[k] = obs_cvt<OT>(0.0f);
            }
        }
    }
    __syncthreads();
    if (e < E && obs)
        copy16(obs + (size_t)e * ld_obs, row, (size_t)C.K_pad * sizeof(OT), hl, HALF);
}

template <typename OT>
__global__ __launch_bounds__(ENV_WPB *WAVE) void env_step_kernel(
    EnvConst C, double *cash, int32_t *shares, int64_t *t, const float *action,
    float *reward, int E, OT *obs, int64_t ld_obs, int32_t *n_invalid)
{
    extern __shared__ __align__(16) uint8_t smem[];
    const int lane = threadIdx.x % WAVE, hl = lane % HALF;
    const int slot = threadIdx.x / HALF;
    const int e = blockIdx.x * ENV_EPB + slot;
    OT *row = (OT *)smem + slot * obs_ld_lds<OT>(C);
    const int n = C.n;
    // every lane of the wave runs the half-wave step (idle halves trade
    // nothing); loads use valid addresses only
    const bool in = e < E;
    const int64_t tt = in ? t[e] : -1;
    const bool live = in && tt >= 0 && tt + 1 < C.T1;
    count_invalid(n_invalid, in && !live, hl);
    const int64_t trow = live ? tt : 0;
    const float *p0 = C.price + (size_t)trow * n;
    const float *p1 = p0 + (live ? n : 0);
    HalfEnv s;
    s.cash = live ? cash[e] : 0.0;
    float a[SPL], q[SPL];
    // a lane's 4 stocks are 16 contiguous bytes of the action, holdings and
    // price rows when n is a multiple of 4 and the arrays are 16-byte
    // aligned: one 16-byte access each instead of four
    const bool vec = n % SPL == 0 && ((uintptr_t)action | (uintptr_t)shares | (uintptr_t)C.price) % 16 == 0;
    if (vec) {
        typedef float f4 __attribute__((ext_vector_type(4)));
        typedef int i4 __attribute__((ext_vector_type(4)));
        const bool v = live && SPL * hl < n;
        const size_t o = (size_t)e * n + SPL * hl;
        const i4 hv = v ? *(const i4 *)(shares + o) : i4{0, 0, 0, 0};
        const f4 av = v ? *(const f4 *)(action + o) : f4{0.f, 0.f, 0.f, 0.f};
        const f4 pv = v ? *(const f4 *)(p0 + SPL * hl) : f4{0.f, 0.f, 0.f, 0.f};
        const f4 qv = v ? *(const f4 *)(p1 + SPL * hl) : f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < SPL; ++c) {
            s.h[c] = hv[c];
            a[c] = av[c];
            s.p[c] = pv[c];
            q[c] = qv[c];
        }
    } else {
#pragma unroll
        for (int c = 0; c < SPL; ++c) {
            const int i = SPL * hl + c;
            const bool v = live && i < n;
            s.h[c] = v ? shares[(size_t)e * n + i] : 0;
            s.p[c] = v ? p0[i] : 0.f;
            a[c] = v ? action[(size_t)e * n + i] : 0.f;
            q[c] = v ? p1[i] : 0.f;
        }
    }
    // bf16 rows of 4k stocks and 4k > 0 indicator values go out in aligned
    // stores (the aligned writer reads indicator chunks, so a market without
    // indicators takes the per-value writer); their indicator chunks are
    // loaded before the step's arithmetic
    const bool aligned_obs = sizeof(OT) == 2 && C.n % 4 == 0 && C.nI > 0 && C.nI % 4 == 0 &&
                             (uintptr_t)C.ind % 16 == 0;
    IndChunks<ENV_IND_ROUNDS> ind;
    if (sizeof(OT) == 2 && obs && aligned_obs)
        ind = load_ind_chunks<ENV_IND_ROUNDS>(C, C.ind + (size_t)(live ? tt + 1 : 0) * C.nI, hl);
    double none = 0.0;
    const float r = env_step_half(C, s, a, q, live, lane, none);
    if (live) {
        if (vec) {
            typedef int i4 __attribute__((ext_vector_type(4)));
            if (SPL * hl < n)
                *(i4 *)(shares + (size_t)e * n + SPL * hl) = i4{s.h[0], s.h[1], s.h[2], s.h[3]};
        } else {
#pragma unroll
            for (int c = 0; c < SPL; ++c) {
                const int i = SPL * hl + c;
                if (i < n) shares[(size_t)e * n + i] = s.h[c];
            }
        }
        if (hl == 0) {
            cash[e] = s.cash;
            t[e] = tt + 1;
            reward[e] = r;
        }
        if (obs && !aligned_obs) {
            const float *irow = C.ind + (size_t)(tt + 1) * C.nI;
            float ind1[1];
            ind1[0] = hl < C.nI ? irow[hl] : 0.f;
            write_obs_half<OT, 1>(row, C, s.cash, s.h, q, ind1, irow, hl);
        }
    } else if (in) {
        if (hl == 0) reward[e] = __builtin_nanf("");
        if (obs)
            for (int k = hl; k < C.K_pad; k += HALF) row[k] = obs_cvt<OT>(__builtin_nanf(""));
    }
    if constexpr (sizeof(OT) == 2) {
        if (obs && aligned_obs)   // every lane (shuffles); only live halves store
            write_obs_half_aligned<ENV_IND_ROUNDS>(row, C, s.cash, s.h, q, ind, lane, hl, live);
    }
    __syncthreads();
    if (in && obs)
        copy16(obs + (size_t)e * ld_obs, row, (size_t)C.K_pad * sizeof(OT), hl, HALF);
}

static size_t row_lds(const EnvConst &c, int esz)
{
    return (size_t)ENV_EPB * (((size_t)c.K_pad * esz + 15) / 16 * 16);
}

bool env_rows_fit(const EnvConst &c, int obs_bf16) { return row_lds(c, obs_bf16 ? 2 : 4) <= LDS_LIMIT; }

hipError_t launch_zero_i32(int32_t *p, hipStream_t s)
{
    hipLaunchKernelGGL(zero_i32_kernel, dim3(1), dim3(1), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_env_reset(const EnvConst &c, double *cash, int32_t *shares,
                            int64_t *t, const int64_t *t0, int E, void *obs,
                            int64_t ld_obs, int obs_bf16, int32_t *n_invalid,
                            hipStream_t s)
{
    if (!env_rows_fit(c, obs_bf16)) return hipErrorInvalidConfiguration;
    if (n_invalid) {
        const hipError_t e = launch_zero_i32(n_invalid, s);
        if (e != hipSuccess) return e;
    }
    const dim3 grid((E + ENV_EPB - 1) / ENV_EPB), block(ENV_WPB * WAVE);
    if (obs_bf16)
        hipLaunchKernelGGL(env_reset_kernel<__bf16>, grid, block, row_lds(c, 2), s, c,
                           cash, shares, t, t0, E, (__bf16 *)obs, ld_obs, n_invalid);
    else
        hipLaunchKernelGGL(env_reset_kernel<float>, grid, block, row_lds(c, 4), s, c,
                           cash, shares, t, t0, E, (float *)obs, ld_obs, n_invalid);
    return hipGetLastError();
}

hipError_t launch_env_step(const EnvConst &c, double *cash, int32_t *shares,
                           int64_t *t, const float *action, float *reward,
                           int E, void *obs, int64_t ld_obs, int obs_bf16,
                           int32_t *n_invalid, hipStream_t s)
{
    if (!env_rows_fit(c, obs_bf16)) return hipErrorInvalidConfiguration;
    if (n_invalid) {
        const hipError_t e = launch_zero_i32(n_invalid, s);
        if (e != hipSuccess) return e;
    }
    const dim3 grid((E + ENV_EPB - 1) / ENV_EPB), block(ENV_WPB * WAVE);
    if (obs_bf16)
        hipLaunchKernelGGL(env_step_kernel<__bf16>, grid, block, row_lds(c, 2), s, c,
                           cash, shares, t, action, reward, E, (__bf16 *)obs, ld_obs,
                           n_invalid);
    else
        hipLaunchKernelGGL(env_step_kernel<float>, grid, block, row_lds(c, 4), s, c,
                           cash, shares, t, action, reward, E, (float *)obs, ld_obs,
                           n_invalid);
    return hipGetLastError();
}

}  // namespace tpk
