// The stock-trading env step on one wavefront (paper Section 3, eqs. (2)-(4)).
//
// One 64-lane wavefront owns one env.  Lane l holds stocks 2l and 2l+1
// (n <= 128), so stock order equals (lane, slot) order and lane-order prefix
// sums are prefix sums in stock index order.
//
//   k_i  = trunc(clip(a_i, -1, 1) * hmax)   (fp32 product, NaN -> 0)
//   sells: s_i = min(-k_i, h_i) at p_t, credit S*(1 - fee)
//   buys : ascending stock index, each the largest q_i <= k_i with
//          (1 + fee) * (G + p_i q_i) <= b_s, G = value bought so far
//   b'   = b_s - (1 + fee) G;  V = b + p_t^T h;  V' = b' + p_{t+1}^T h'
//   r    = reward_scale * (V' - V)
//
// Every p*q with q <= 128 and p in [2^-2, 2^13) is a multiple of 2^-25 below
// 2^20, so S, G and every partial sum of them are exact in fp64 in any order:
// the wave-level sums and scans below give the same bits as a serial loop.
// The buy test fma(f_b, X, -b_s) <= 0 rounds once, so its sign is the sign
// of the exact f_b*X - b_s.  Balances therefore agree bit for bit with a
// serial implementation, and so do share counts.
#pragma once

#include "device.hpp"
#include "internal.hpp"

namespace tpk {

__device__ __forceinline__ int shares_from_action(float a, int hmax)
{
    const float u = isnan(a) ? 0.0f : fminf(fmaxf(a, -1.0f), 1.0f);
    return (int)truncf(u * (float)hmax);
}

// Per-env state held by the owning wave: lane l keeps stocks 2l, 2l+1.
struct LaneEnv {
    double cash;   // balance (same on every lane)
    int h0, h1;    // holdings (0 for stocks >= n)
    float p0, p1;  // prices at the current row (0 for stocks >= n)
};

// One transition.  a0/a1: raw actions of this lane's stocks; q0/q1: their
// prices at the next row.  Returns the reward (same on every lane).  Must be
// called by all 64 lanes.
__device__ __forceinline__ float env_step_wave(const EnvConst &C, LaneEnv &s,
                                               float a0, float a1, float q0,
                                               float q1, int lane)
{
    const int n = C.n;
    const bool v0 = 2 * lane < n, v1 = 2 * lane + 1 < n;
    const int k0 = v0 ? shares_from_action(a0, C.hmax) : 0;
    const int k1 = v1 ? shares_from_action(a1, C.hmax) : 0;
    const double pa = (double)s.p0, pb = (double)s.p1;

    // total asset before the step (fp64; products h*p are exact)
    const double V = s.cash + wave_sum((double)s.h0 * pa + (double)s.h1 * pb);

    // sells
    const int sa = k0 < 0 ? min(-k0, s.h0) : 0;
    const int sb = k1 < 0 ? min(-k1, s.h1) : 0;
    int h0 = s.h0 - sa, h1 = s.h1 - sb;
    const double S = wave_sum(pa * (double)sa + pb * (double)sb);  // exact
    const double b_s = fma(S, C.f_s, s.cash);
    const double fb = C.f_b;

    // buys: resolve the greedy in ascending stock order in rounds.  A round
    // first drops every pending stock that cannot pay for one share at the
    // current G (G only grows, so it never will), then finds the first
    // pending stock whose full order no longer fits: every pending stock
    // before it is bought in full, it gets its largest affordable q, and the
    // next round continues after it.
    const double c0 = k0 > 0 ? pa * (double)k0 : 0.0;
    const double c1 = k1 > 0 ? pb * (double)k1 : 0.0;
    bool pend0 = k0 > 0, pend1 = k1 > 0;
    int q0n = 0, q1n = 0;
    double G = 0.0;
    for (bool first = true;; first = false) {
        if (!first) {
            if (pend0 && fma(fb, G + pa, -b_s) > 0.0) pend0 = false;
            if (pend1 && fma(fb, G + pb, -b_s) > 0.0) pend1 = false;
        }
        if (__ballot(pend0 || pend1) == 0) break;
        const double cc0 = pend0 ? c0 : 0.0, cc1 = pend1 ? c1 : 0.0;
        const double tot = cc0 + cc1;
        const double incl = wave_inclusive_scan(tot);
        const double base = G + (incl - tot);  // exact
        const double P0 = base + cc0, P1 = P0 + cc1;
        const bool bad0 = pend0 && fma(fb, P0, -b_s) > 0.0;
        const bool bad1 = pend1 && fma(fb, P1, -b_s) > 0.0;
        const uint64_t m = __ballot(bad0 || bad1);
        if (m == 0) {
            if (pend0) q0n = k0;
            if (pend1) q1n = k1;
            G = lane_value(base + tot, WAVE - 1);
            break;
        }
        const int fl = __ffsll((unsigned long long)m) - 1;
        const bool f_is_1 = lane_value(bad0 ? 0 : 1, fl) != 0;
        // stocks before the first misfit are bought in full
        if (lane < fl) {
            if (pend0) q0n = k0;
            if (pend1) q1n = k1;
            pend0 = pend1 = false;
        } else if (lane == fl && f_is_1 && pend0) {
            q0n = k0;
            pend0 = false;
        }
        const double Gf = lane_value(f_is_1 ? P1 - cc1 : P0 - cc0, fl);
        const double pf = lane_value(f_is_1 ? pb : pa, fl);
        const int kf = lane_value(f_is_1 ? k1 : k0, fl);
        // largest q in [0, kf-1] with f_b (Gf + pf q) <= b_s: estimate, then
        // step to the exact boundary with the sign-exact test
        const double rem = fma(-fb, Gf, b_s);
        double est = floor(rem / (pf * fb));
        est = fmin(fmax(est, 0.0), (double)(kf - 1));
        int q = (int)est;
        while (q < kf - 1 && fma(fb, Gf + pf * (double)(q + 1), -b_s) <= 0.0) ++q;
        while (q > 0 && fma(fb, Gf + pf * (double)q, -b_s) > 0.0) --q;
        G = Gf + pf * (double)q;
        if (lane == fl) {
            if (f_is_1) {
                q1n = q;
                pend1 = false;
            } else {
                q0n = q;
                pend0 = false;
            }
        }
    }
    h0 += q0n;
    h1 += q1n;
    double nb = fma(-fb, G, b_s);
    if (nb < 0.0) nb = 0.0;

    const double V1 = nb + wave_sum((double)h0 * (double)q0 + (double)h1 * (double)q1);
    s.cash = nb;
    s.h0 = h0;
    s.h1 = h1;
    s.p0 = q0;
    s.p1 = q1;
    return (float)(C.reward_scale * (V1 - V));
}

template <typename T> __device__ __forceinline__ T obs_cvt(float x);
template <> __device__ __forceinline__ float obs_cvt<float>(float x) { return x; }
template <> __device__ __forceinline__ __bf16 obs_cvt<__bf16>(float x) { return to_bf16(x); }

// Observation row [b*cs, p*ps (n), h*ss (n), ind (nI), 0 ... K_pad) written
// to `row` (LDS or global).  prow: the n prices of the observed row; irow:
// its nI indicators.  All 64 lanes call it.
template <typename T>
__device__ __forceinline__ void write_obs_row(T *row, const EnvConst &C,
                                              double cash, int h0, int h1,
                                              const float *prow,
                                              const float *irow, int lane)
{
    const int n = C.n, nI = C.nI, S = 1 + 2 * n + nI;
    const int i0 = 2 * lane, i1 = i0 + 1;
    if (lane == 0) row[0] = obs_cvt<T>((float)(cash * (double)C.cash_scale));
    if (i0 < n) {
        row[1 + i0] = obs_cvt<T>(prow[i0] * C.price_scale);
        row[1 + n + i0] = obs_cvt<T>((float)h0 * C.share_scale);
    }
    if (i1 < n) {
        row[1 + i1] = obs_cvt<T>(prow[i1] * C.price_scale);
        row[1 + n + i1] = obs_cvt<T>((float)h1 * C.share_scale);
    }
    for (int k = lane; k < nI; k += WAVE) row[1 + 2 * n + k] = obs_cvt<T>(irow[k]);
    for (int k = S + lane; k < C.K_pad; k += WAVE) row[k] = obs_cvt<T>(0.0f);
}

// The same row with the next-row prices and the first 64*IPL indicators
// already in registers (q0/q1: prices of this lane's stocks; ind[m]:
// indicator lane + 64 m); indicators beyond that are read from irow.
template <typename T, int IPL>
__device__ __forceinline__ void write_obs_row_regs(T *row, const EnvConst &C,
                                                   double cash, int h0, int h1,
                                                   float q0, float q1,
                                                   const float (&ind)[IPL],
                                                   const float *irow, int lane)
{
    const int n = C.n, nI = C.nI, S = 1 + 2 * n + nI;
    const int i0 = 2 * lane, i1 = i0 + 1;
    if (lane == 0) row[0] = obs_cvt<T>((float)(cash * (double)C.cash_scale));
    if (i0 < n) {
        row[1 + i0] = obs_cvt<T>(q0 * C.price_scale);
        row[1 + n + i0] = obs_cvt<T>((float)h0 * C.share_scale);
    }
    if (i1 < n) {
        row[1 + i1] = obs_cvt<T>(q1 * C.price_scale);
        row[1 + n + i1] = obs_cvt<T>((float)h1 * C.share_scale);
    }
    T *ri = row + 1 + 2 * n;
#pragma unroll
    for (int m = 0; m < IPL; ++m) {
        const int k = lane + WAVE * m;
        if (k < nI) ri[k] = obs_cvt<T>(ind[m]);
    }
    for (int k = WAVE * IPL + lane; k < nI; k += WAVE) ri[k] = obs_cvt<T>(irow[k]);
    for (int k = S + lane; k < C.K_pad; k += WAVE) row[k] = obs_cvt<T>(0.0f);
}

// Copy `bytes` (a multiple of 16) from LDS to global with 16-byte accesses,
// lanes [l0, l0 + nl) of the calling group participating.
__device__ __forceinline__ void copy16(void *dst, const void *src, size_t bytes,
                                       int l, int nl)
{
    const uint4 *s = (const uint4 *)src;
    uint4 *d = (uint4 *)dst;
    for (size_t i = l; i < bytes / 16; i += nl) d[i] = s[i];
}

}  // namespace tpk
