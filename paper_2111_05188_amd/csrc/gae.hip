// GAE / reward-to-go over a time-major rollout [L][E].
//
// The recurrence A_j = delta_j + c_j A_{j+1} (c_j = gamma lambda (1 - d_j))
// is sequential in time but a composition of affine maps, so it splits into
// time chunks: with zero carry-in, chunk [lo, hi) yields a local value A_loc
// at lo and the product P of its c_j, and the true value at lo is
// A_loc + P * A_hi.  A workgroup takes 64 envs (one per lane, coalesced rows)
// and NCH time chunks (one wave each): pass 1 computes (A_loc, P) per chunk,
// the carries are combined through LDS, pass 2 re-runs each chunk from its
// true carry and writes A and ret.  Chunks of up to 28 steps keep their
// inputs in registers between the passes (each input is read once); longer
// ones read them again.  fp64 arithmetic, fp32 I/O.
#include "device.hpp"
#include "internal.hpp"

namespace tpk {

constexpr int GAE_NCH = 16;
constexpr int GAE_CACHE = 28;   // chunks up to this long keep their inputs in registers

template <bool CACHE>
__global__ __launch_bounds__(GAE_NCH *WAVE) void gae_kernel(
    const float *__restrict__ r, const float *__restrict__ v,
    const uint8_t *__restrict__ d, int L, int E, double g, double gl,
    float *__restrict__ adv, float *__restrict__ ret)
{
    __shared__ double sA[GAE_NCH][WAVE], sP[GAE_NCH][WAVE];
    const int c = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
    const int e = blockIdx.x * WAVE + lane;
    const int cl = (L + GAE_NCH - 1) / GAE_NCH;
    const int lo = min(L, c * cl), hi = min(L, lo + cl);
    const bool ok = e < E;
    const size_t sE = (size_t)E;

    double A = 0.0, P = 1.0;
    // the chunk's inputs, step hi-1-k in slot k (CACHE: pass 2 reads them back)
    float cr[CACHE ? GAE_CACHE : 1], cv[CACHE ? GAE_CACHE : 1];
    uint32_t cd = 0;   // bit k: done at step hi-1-k
    if (ok && hi > lo) {
        double vn = (double)v[(size_t)hi * sE + e];
        if constexpr (CACHE) {
#pragma unroll
            for (int k = 0; k < GAE_CACHE; ++k) {
                const int j = hi - 1 - k;
                if (j >= lo) {
                    const size_t i = (size_t)j * sE + e;
                    cr[k] = r[i];
                    cv[k] = v[i];
                    cd |= (uint32_t)(d[i] != 0) << k;
                }
            }
#pragma unroll
            for (int k = 0; k < GAE_CACHE; ++k) {
                if (hi - 1 - k >= lo) {
                    const double nd = (cd >> k) & 1u ? 0.0 : 1.0;
                    const double vj = (double)cv[k];
                    const double delta = (double)cr[k] + g * nd * vn - vj;
                    const double cj = gl * nd;
                    A = delta + cj * A;
                    P *= cj;
                    vn = vj;
                }
            }
        } else {
#pragma unroll 4
            for (int j = hi - 1; j >= lo; --j) {
                const size_t i = (size_t)j * sE + e;
                const double nd = d[i] ? 0.0 : 1.0;
                const double vj = (double)v[i];
                const double delta = (double)r[i] + g * nd * vn - vj;
                const double cj = gl * nd;
                A = delta + cj * A;
                P *= cj;
                vn = vj;
            }
        }
    }
    sA[c][lane] = A;
    sP[c][lane] = P;
    __syncthreads();
    double carry = 0.0;
    for (int cc = GAE_NCH - 1; cc > c; --cc) carry = sA[cc][lane] + sP[cc][lane] * carry;

    if (ok && hi > lo) {
        A = carry;
        double vn = (double)v[(size_t)hi * sE + e];
        if constexpr (CACHE) {
#pragma unroll
            for (int k = 0; k < GAE_CACHE; ++k) {
                const int j = hi - 1 - k;
                if (j >= lo) {
                    const size_t i = (size_t)j * sE + e;
                    const double nd = (cd >> k) & 1u ? 0.0 : 1.0;
                    const double vj = (double)cv[k];
                    const double delta = (double)cr[k] + g * nd * vn - vj;
                    A = delta + gl * nd * A;
                    adv[i] = (float)A;
                    ret[i] = (float)(A + vj);
                    vn = vj;
                }
            }
        } else {
#pragma unroll 4
            for (int j = hi - 1; j >= lo; --j) {
                const size_t i = (size_t)j * sE + e;
                const double nd = d[i] ? 0.0 : 1.0;
                const double vj = (double)v[i];
                const double delta = (double)r[i] + g * nd * vn - vj;
                A = delta + gl * nd * A;
                adv[i] = (float)A;
                ret[i] = (float)(A + vj);
                vn = vj;
            }
        }
    }
}

hipError_t launch_gae(const float *r, const float *v, const uint8_t *d, int L,
                      int E, double g, double gl, float *adv, float *ret,
                      hipStream_t s)
{
    const int cl = (L + GAE_NCH - 1) / GAE_NCH;
    if (cl <= GAE_CACHE)
        hipLaunchKernelGGL(gae_kernel<true>, dim3((E + WAVE - 1) / WAVE), dim3(GAE_NCH * WAVE), 0,
                           s, r, v, d, L, E, g, gl, adv, ret);
    else
        hipLaunchKernelGGL(gae_kernel<false>, dim3((E + WAVE - 1) / WAVE), dim3(GAE_NCH * WAVE), 0,
                           s, r, v, d, L, E, g, gl, adv, ret);
    return hipGetLastError();
}

}  // namespace tpk
