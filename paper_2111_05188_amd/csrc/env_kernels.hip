// Standalone env kernels: reset and one teacher-forced step.
// One 64-lane wave per env; the observation row is assembled in LDS and
// written to HBM with 16-byte stores.
#include "device.hpp"
#include "env.hpp"
#include "internal.hpp"

namespace tpk {

constexpr int ENV_WPB = 4;  // envs (waves) per workgroup

template <typename OT>
__global__ __launch_bounds__(ENV_WPB *WAVE) void env_reset_kernel(
    EnvConst C, double *cash, int32_t *shares, int64_t *t, const int64_t *t0,
    int E, OT *obs, int64_t ld_obs)
{
    extern __shared__ __align__(16) uint8_t smem[];
    const int wave = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
    const int e = blockIdx.x * ENV_WPB + wave;
    const int ldr = (C.K_pad * (int)sizeof(OT) + 15) / 16 * 16 / (int)sizeof(OT);
    OT *row = (OT *)smem + wave * ldr;
    if (e < E) {
        const int n = C.n;
        const int64_t tt = t0[e];
        const bool ok = tt >= 0 && tt < C.T1 - 1;
        for (int i = lane; i < n; i += WAVE) shares[(size_t)e * n + i] = 0;
        if (lane == 0) {
            cash[e] = C.cash0;
            t[e] = ok ? tt : -1;
        }
        if (obs) {
            if (ok) {
                write_obs_row<OT>(row, C, C.cash0, 0, 0, C.price + (size_t)tt * n,
                                  C.ind + (size_t)tt * C.nI, lane);
            } else {
                for (int k = lane; k < C.K_pad; k += WAVE) row[k] = obs_cvt<OT>(0.0f);
            }
        }
    }
    __syncthreads();
    if (e < E && obs)
        copy16(obs + (size_t)e * ld_obs, row, (size_t)C.K_pad * sizeof(OT), lane, WAVE);
}

template <typename OT>
__global__ __launch_bounds__(ENV_WPB *WAVE) void env_step_kernel(
    EnvConst C, double *cash, int32_t *shares, int64_t *t, const float *action,
    float *reward, int E, OT *obs, int64_t ld_obs)
{
    extern __shared__ __align__(16) uint8_t smem[];
    const int wave = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
    const int e = blockIdx.x * ENV_WPB + wave;
    const int ldr = (C.K_pad * (int)sizeof(OT) + 15) / 16 * 16 / (int)sizeof(OT);
    OT *row = (OT *)smem + wave * ldr;
    if (e < E) {
        const int n = C.n;
        const int i0 = 2 * lane, i1 = i0 + 1;
        const int64_t tt = t[e];
        if (tt >= 0 && tt + 1 < C.T1) {
            const float *p = C.price + (size_t)tt * n;
            const float *p1 = p + n;
            const float *ar = action + (size_t)e * n;
            int32_t *hr = shares + (size_t)e * n;
            LaneEnv s{cash[e], 0, 0, 0.f, 0.f};
            float a0 = 0.f, a1 = 0.f, q0 = 0.f, q1 = 0.f;
            if (i0 < n) { s.h0 = hr[i0]; s.p0 = p[i0]; a0 = ar[i0]; q0 = p1[i0]; }
            if (i1 < n) { s.h1 = hr[i1]; s.p1 = p[i1]; a1 = ar[i1]; q1 = p1[i1]; }
            const float r = env_step_wave(C, s, a0, a1, q0, q1, lane);
            if (i0 < n) hr[i0] = s.h0;
            if (i1 < n) hr[i1] = s.h1;
            if (lane == 0) {
                cash[e] = s.cash;
                t[e] = tt + 1;
                reward[e] = r;
            }
            if (obs)
                write_obs_row<OT>(row, C, s.cash, s.h0, s.h1, p1,
                                  C.ind + (size_t)(tt + 1) * C.nI, lane);
        } else {
            if (lane == 0) reward[e] = __builtin_nanf("");
            if (obs)
                for (int k = lane; k < C.K_pad; k += WAVE) row[k] = obs_cvt<OT>(__builtin_nanf(""));
        }
    }
    __syncthreads();
    if (e < E && obs)
        copy16(obs + (size_t)e * ld_obs, row, (size_t)C.K_pad * sizeof(OT), lane, WAVE);
}

static size_t row_lds(const EnvConst &c, int esz)
{
    return (size_t)ENV_WPB * (((size_t)c.K_pad * esz + 15) / 16 * 16);
}

hipError_t launch_env_reset(const EnvConst &c, double *cash, int32_t *shares,
                            int64_t *t, const int64_t *t0, int E, void *obs,
                            int64_t ld_obs, int obs_bf16, hipStream_t s)
{
    const dim3 grid((E + ENV_WPB - 1) / ENV_WPB), block(ENV_WPB * WAVE);
    if (obs_bf16)
        hipLaunchKernelGGL(env_reset_kernel<__bf16>, grid, block, row_lds(c, 2), s, c,
                           cash, shares, t, t0, E, (__bf16 *)obs, ld_obs);
    else
        hipLaunchKernelGGL(env_reset_kernel<float>, grid, block, row_lds(c, 4), s, c,
                           cash, shares, t, t0, E, (float *)obs, ld_obs);
    return hipGetLastError();
}

hipError_t launch_env_step(const EnvConst &c, double *cash, int32_t *shares,
                           int64_t *t, const float *action, float *reward,
                           int E, void *obs, int64_t ld_obs, int obs_bf16,
                           hipStream_t s)
{
    const dim3 grid((E + ENV_WPB - 1) / ENV_WPB), block(ENV_WPB * WAVE);
    if (obs_bf16)
        hipLaunchKernelGGL(env_step_kernel<__bf16>, grid, block, row_lds(c, 2), s, c,
                           cash, shares, t, action, reward, E, (__bf16 *)obs, ld_obs);
    else
        hipLaunchKernelGGL(env_step_kernel<float>, grid, block, row_lds(c, 4), s, c,
                           cash, shares, t, action, reward, E, (float *)obs, ld_obs);
    return hipGetLastError();
}

}  // namespace tpk
