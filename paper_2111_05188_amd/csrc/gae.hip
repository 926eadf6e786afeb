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
// ones read them again.  fp64 arithmetic, fp32 I/O.  This kernel serves
// rollouts longer than gae_wide_kernel (below) takes.
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

// Rollouts of up to GW_LMAX steps: a workgroup takes GW_E envs and GW_NCH
// chunks of at most GW_CL steps, one thread per (env, chunk), so that even
// a few thousand envs fill every CU.  Lane l of wave w holds env l % GW_E
// of chunk w * GW_K + l / GW_E; each wave reads GW_K row pieces of GW_E
// consecutive envs per step (64 or 128 bytes).  The chunk maps x -> A + P x (x: the
// value carried in from the chunk after) are composed within a wave by
// shuffles, across waves through LDS; every input is read once and kept in
// registers between the two passes.
constexpr int GW_W = 16;                 // waves per workgroup
constexpr int GW_LMAX = 512;             // longest rollout

template <int GW_E>   // envs per workgroup (16 or 32)
__global__ __launch_bounds__(GW_W *WAVE) void gae_wide_kernel(
    const float *__restrict__ r, const float *__restrict__ v,
    const uint8_t *__restrict__ d, int L, int E, int nblk, double g, double gl,
    float *__restrict__ adv, float *__restrict__ ret)
{
    constexpr int GW_K = WAVE / GW_E;                  // chunks per wave
    constexpr int GW_NCH = GW_K * GW_W;                // chunks per workgroup
    constexpr int GW_CL = GW_LMAX / GW_NCH;            // longest chunk
    __shared__ double sA[GW_W][GW_E], sP[GW_W][GW_E];
    // XCD-aware order: consecutive env groups (which share 128-byte lines)
    // go to one XCD's L2
    const int logical = (blockIdx.x % 8) * (gridDim.x / 8) + blockIdx.x / 8;
    if (logical >= nblk) return;   // whole workgroup: no barrier is skipped by part of it
    const int w = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
    const int le = lane % GW_E, k = lane / GW_E;
    const int e = logical * GW_E + le;
    const int c = w * GW_K + k;
    const int cl = (L + GW_NCH - 1) / GW_NCH;
    const int lo = min(L, c * cl), hi = min(L, lo + cl);
    const bool ok = e < E && hi > lo;
    const size_t sE = (size_t)E;

    // pass 1: the chunk's inputs (step hi-1-i in slot i) and its map
    float cr[GW_CL], cv[GW_CL];
    uint32_t cd = 0;
    double vend = 0.0;
    if (ok) {
        vend = (double)v[(size_t)hi * sE + e];
#pragma unroll
        for (int i = 0; i < GW_CL; ++i) {
            const int j = hi - 1 - i;
            if (j >= lo) {
                const size_t x = (size_t)j * sE + e;
                cr[i] = r[x];
                cv[i] = v[x];
                cd |= (uint32_t)(d[x] != 0) << i;
            }
        }
    }
    double A = 0.0, P = 1.0;
    if (ok) {
        double vn = vend;
#pragma unroll
        for (int i = 0; i < GW_CL; ++i) {
            if (hi - 1 - i >= lo) {
                const double nd = (cd >> i) & 1u ? 0.0 : 1.0;
                const double vj = (double)cv[i];
                const double delta = (double)cr[i] + g * nd * vn - vj;
                const double cj = gl * nd;
                A = delta + cj * A;
                P *= cj;
                vn = vj;
            }
        }
    }

    // suffix composition over the wave's GW_K chunks of this env: after
    // it, (A, P) maps the value entering chunk GW_K-1's end to chunk k's
    // start through chunks k .. GW_K-1 (chunks past the rollout are the
    // identity)
#pragma unroll
    for (int sh = 1; sh < GW_K; sh *= 2) {
        const double An = __shfl_down(A, sh * GW_E), Pn = __shfl_down(P, sh * GW_E);
        if (k + sh < GW_K) {
            A = A + P * An;
            P = P * Pn;
        }
    }
    if (k == 0) {
        sA[w][le] = A;
        sP[w][le] = P;
    }
    __syncthreads();
    // value entering this wave's last chunk: the later waves' maps applied
    // to 0, last wave first
    double carry = 0.0;
    for (int ww = GW_W - 1; ww > w; --ww) carry = sA[ww][le] + sP[ww][le] * carry;
    // value entering this chunk: the suffix map of chunk k + 1 applied to it
    {
        const double An = __shfl_down(A, GW_E), Pn = __shfl_down(P, GW_E);
        if (k + 1 < GW_K) carry = An + Pn * carry;
    }

    // pass 2: the chunk again from its true carry
    if (ok) {
        A = carry;
        double vn = vend;
#pragma unroll
        for (int i = 0; i < GW_CL; ++i) {
            const int j = hi - 1 - i;
            if (j >= lo) {
                const size_t x = (size_t)j * sE + e;
                const double nd = (cd >> i) & 1u ? 0.0 : 1.0;
                const double vj = (double)cv[i];
                const double delta = (double)cr[i] + g * nd * vn - vj;
                A = delta + gl * nd * A;
                adv[x] = (float)A;
                ret[x] = (float)(A + vj);
                vn = vj;
            }
        }
    }
}

// Many envs (E a multiple of 4, 16-byte aligned rows): the same two passes
// with four envs per lane, so every access is one 16-byte load or store of
// r, v, adv, ret (4-byte for done) and a wave instruction moves whole
// 256-byte row pieces.  A workgroup takes GV_E = 64 envs (16 lanes per row
// piece) and GV_W * 4 = 32 chunks of at most GV_CL steps; chunk maps
// compose by shuffles within a wave (4 chunks) and through LDS across the
// 8 waves.
constexpr int GV_W = 8;
constexpr int GV_E = 64;
constexpr int GV_RL = GV_E / 4;               // lanes per row piece
constexpr int GV_K = WAVE / GV_RL;            // chunks per wave
constexpr int GV_NCH = GV_K * GV_W;           // chunks per workgroup
constexpr int GV_LMAX = 416;                  // longest rollout
constexpr int GV_CL = GV_LMAX / GV_NCH;       // longest chunk (13 steps)

typedef float f4g __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(GV_W *WAVE) void gae_vec_kernel(
    const float *__restrict__ r, const float *__restrict__ v,
    const uint8_t *__restrict__ d, int L, int E, int nblk, double g, double gl,
    float *__restrict__ adv, float *__restrict__ ret)
{
    __shared__ double sA[GV_W][GV_E], sP[GV_W][GV_E];
    const int logical = (blockIdx.x % 8) * (gridDim.x / 8) + blockIdx.x / 8;
    if (logical >= nblk) return;   // whole workgroup
    const int w = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
    const int lr = lane % GV_RL, k = lane / GV_RL;
    const int e0 = logical * GV_E + 4 * lr;     // this lane's first env (E % 4 == 0)
    const int c = w * GV_K + k;
    const int cl = (L + GV_NCH - 1) / GV_NCH;
    const int lo = min(L, c * cl), hi = min(L, lo + cl);
    const bool ok = e0 < E && hi > lo;
    const size_t sE = (size_t)E;

    f4g cr[GV_CL], cv[GV_CL];
    uint32_t cd[GV_CL];   // done bytes of the 4 envs at step hi-1-i
    f4g vend = {0.f, 0.f, 0.f, 0.f};
    if (ok) {
        vend = __builtin_nontemporal_load((const f4g *)(v + (size_t)hi * sE + e0));
#pragma unroll
        for (int i = 0; i < GV_CL; ++i) {
            const int j = hi - 1 - i;
            if (j >= lo) {
                const size_t x = (size_t)j * sE + e0;
                cr[i] = __builtin_nontemporal_load((const f4g *)(r + x));
                cv[i] = __builtin_nontemporal_load((const f4g *)(v + x));
                cd[i] = __builtin_nontemporal_load((const uint32_t *)(d + x));
            }
        }
    }
    double A[4] = {0.0, 0.0, 0.0, 0.0}, P[4] = {1.0, 1.0, 1.0, 1.0};
    if (ok) {
        double vn[4] = {(double)vend[0], (double)vend[1], (double)vend[2], (double)vend[3]};
#pragma unroll
        for (int i = 0; i < GV_CL; ++i) {
            if (hi - 1 - i >= lo) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const double nd = (cd[i] >> (8 * q)) & 0xFFu ? 0.0 : 1.0;
                    const double vj = (double)cv[i][q];
                    const double delta = (double)cr[i][q] + g * nd * vn[q] - vj;
                    const double cj = gl * nd;
                    A[q] = delta + cj * A[q];
                    P[q] *= cj;
                    vn[q] = vj;
                }
            }
        }
    }
    // suffix composition over the wave's GV_K chunks of each env
#pragma unroll
    for (int sh = 1; sh < GV_K; sh *= 2) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const double An = __shfl_down(A[q], sh * GV_RL), Pn = __shfl_down(P[q], sh * GV_RL);
            if (k + sh < GV_K) {
                A[q] = A[q] + P[q] * An;
                P[q] = P[q] * Pn;
            }
        }
    }
    if (k == 0) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            sA[w][4 * lr + q] = A[q];
            sP[w][4 * lr + q] = P[q];
        }
    }
    __syncthreads();
    double carry[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        double cq = 0.0;
        for (int ww = GV_W - 1; ww > w; --ww) cq = sA[ww][4 * lr + q] + sP[ww][4 * lr + q] * cq;
        const double An = __shfl_down(A[q], GV_RL), Pn = __shfl_down(P[q], GV_RL);
        carry[q] = k + 1 < GV_K ? An + Pn * cq : cq;
    }

    // pass 2 from the true carries
    if (ok) {
        double vn[4] = {(double)vend[0], (double)vend[1], (double)vend[2], (double)vend[3]};
#pragma unroll
        for (int q = 0; q < 4; ++q) A[q] = carry[q];
#pragma unroll
        for (int i = 0; i < GV_CL; ++i) {
            const int j = hi - 1 - i;
            if (j >= lo) {
                f4g a4, r4;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const double nd = (cd[i] >> (8 * q)) & 0xFFu ? 0.0 : 1.0;
                    const double vj = (double)cv[i][q];
                    const double delta = (double)cr[i][q] + g * nd * vn[q] - vj;
                    A[q] = delta + gl * nd * A[q];
                    a4[q] = (float)A[q];
                    r4[q] = (float)(A[q] + vj);
                    vn[q] = vj;
                }
                const size_t x = (size_t)j * sE + e0;
                __builtin_nontemporal_store(a4, (f4g *)(adv + x));
                __builtin_nontemporal_store(r4, (f4g *)(ret + x));
            }
        }
    }
}

hipError_t launch_gae(const float *r, const float *v, const uint8_t *d, int L,
                      int E, double g, double gl, float *adv, float *ret,
                      hipStream_t s)
{
    // rollouts up to GW_LMAX steps: 16-env workgroups below 16,384 envs
    // (so that every CU gets one), whole-line 32-env ones from there on
    const bool vec_ok = E % 4 == 0 && (uintptr_t)r % 16 == 0 && (uintptr_t)v % 16 == 0 &&
                        (uintptr_t)d % 4 == 0 && (uintptr_t)adv % 16 == 0 &&
                        (uintptr_t)ret % 16 == 0;
    if (L <= GV_LMAX && E >= 16384 && vec_ok) {
        const int nblk = (E + GV_E - 1) / GV_E;
        hipLaunchKernelGGL(gae_vec_kernel, dim3((nblk + 7) / 8 * 8), dim3(GV_W * WAVE), 0, s, r, v,
                           d, L, E, nblk, g, gl, adv, ret);
        return hipGetLastError();
    }
    if (L <= GW_LMAX) {
        if (E >= 16384) {
            const int nblk = (E + 31) / 32;
            hipLaunchKernelGGL(gae_wide_kernel<32>, dim3((nblk + 7) / 8 * 8), dim3(GW_W * WAVE), 0, s,
                               r, v, d, L, E, nblk, g, gl, adv, ret);
        } else {
            const int nblk = (E + 15) / 16;
            hipLaunchKernelGGL(gae_wide_kernel<16>, dim3((nblk + 7) / 8 * 8), dim3(GW_W * WAVE), 0, s,
                               r, v, d, L, E, nblk, g, gl, adv, ret);
        }
        return hipGetLastError();
    }
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
