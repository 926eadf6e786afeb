// The stock-trading env step (paper Section 3, eqs. (2)-(4)) on one 16-lane
// DPP row: a 64-lane wavefront steps four envs at once, env r on lanes
// 16r .. 16r+15.  Lane s of a row holds stocks 8s .. 8s+7 (n <= 128), so
// stock order equals (lane, slot) order and a row's lane-order prefix sum is
// a prefix sum in stock index order.  Every cross-lane step stays inside a
// row (row_shr scans, quad_perm / mirror butterflies), so the four envs share
// one instruction stream and never exchange data.
//
// The arithmetic is the half-wave env step's (env.hpp), with the same exact
// fp64 sums: every p*q with q <= 128 and p in [2^-2, 2^13) is a multiple of
// 2^-25 below 2^20, so S, G and all their partial sums are exact in any
// order, and the sign-exact buy test fma(f_b, X, -b_s) <= 0 decides every
// purchase as a serial loop would.  Balances and share counts therefore
// agree bit for bit with the serial definition.
//
// Compared with the half-wave version a row carries twice the stocks per
// lane but a wave carries twice the envs, so per-stock work per env is the
// same while the cross-lane steps (one fewer level, no cross-row carries, no
// lane broadcasts) and the per-wave control cost half as much per env.
#pragma once

#include "device.hpp"
#include "internal.hpp"

namespace tpk {

constexpr int RL = 16;    // lanes per env (one DPP row)
constexpr int SPR = 8;    // stocks per lane

// DPP lane moves of a 64-bit value within 16-lane rows.  Lanes without a
// source (row_shr past the row start) receive 0.
enum : int {
    DPP_QP_XOR1 = 0xB1,       // quad_perm [1,0,3,2]
    DPP_QP_XOR2 = 0x4E,       // quad_perm [2,3,0,1]
    DPP_ROW_SHR1 = 0x111,
    DPP_ROW_ROR1 = 0x121,
    DPP_ROW_MIRROR = 0x140,   // lane i <- lane 15 - i
    DPP_ROW_HMIRROR = 0x141,  // lane i <- lane 7 - i within each half-row
};

template <int CTRL>
__device__ __forceinline__ double dpp64(double x)
{
    const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(x), CTRL, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(x), CTRL, 0xF, 0xF, false);
    return __hiloint2double(hi, lo);
}

template <int CTRL>
__device__ __forceinline__ float dpp32f(float x)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

template <int CTRL>
__device__ __forceinline__ int dpp32i(int x)
{
    return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xF, 0xF, false);
}

// Sum over the 16 lanes of each row, returned to every lane of the row.  A
// butterfly: each level adds a lane to its partner, and both partners add
// the same two values, so every lane ends with the same bits.
__device__ __forceinline__ double row_sum(double v)
{
    v += dpp64<DPP_QP_XOR1>(v);
    v += dpp64<DPP_QP_XOR2>(v);
    v += dpp64<DPP_ROW_HMIRROR>(v);
    v += dpp64<DPP_ROW_MIRROR>(v);
    return v;
}

// Inclusive prefix sum within each row, in lane order.
__device__ __forceinline__ double row_inclusive_scan(double v)
{
    v += dpp64<0x111>(v);
    v += dpp64<0x112>(v);
    v += dpp64<0x114>(v);
    v += dpp64<0x118>(v);
    return v;
}

// 1 on lanes below which (in their row) some lane has x != 0.
__device__ __forceinline__ int row_any_below(int x)
{
    int v = x != 0;
    v |= dpp32i<0x111>(v);
    v |= dpp32i<0x112>(v);
    v |= dpp32i<0x114>(v);
    v |= dpp32i<0x118>(v);
    return dpp32i<0x111>(v);   // exclusive: shift the inclusive OR by one lane
}

// Per-env state held by the owning row: lane s keeps stocks 8s .. 8s+7.
struct RowEnv {
    double cash;      // balance (same on every lane of the row)
    double value;     // total asset b + p^T h at the current row
    int h[SPR];       // holdings (0 for stocks >= n)
    double pd[SPR];   // prices at the current row (0 for stocks >= n)
};

// k = trunc(clip(a, -1, 1) * hmax), NaN -> 0 (the fp32 product truncated
// toward zero).
__device__ __forceinline__ int row_shares_from_action(float a, float hmaxf)
{
    const float u = __builtin_amdgcn_fmed3f(a, -1.0f, 1.0f);
    const int k = (int)(u * hmaxf);
    return a == a ? k : 0;
}

// One transition of the env owned by this lane's row.  a[c]: raw actions of
// this lane's stocks (0 for stocks >= n and for rows not stepped, which then
// trade nothing); qd[c]: their prices at the next row.  Returns the reward
// (same on every lane of the row).  All 64 lanes call it.
__device__ __forceinline__ float env_step_row(const EnvConst &C, RowEnv &s, const float (&a)[SPR],
                                              const double (&qd)[SPR])
{
    const double fb = C.f_b;
    const float hmaxf = (float)C.hmax;
    int k[SPR];
#pragma unroll
    for (int c = 0; c < SPR; ++c) k[c] = row_shares_from_action(a[c], hmaxf);

    // sells (all exact in fp64)
    int h[SPR];
    double sv = 0.0;
#pragma unroll
    for (int c = 0; c < SPR; ++c) {
        const int sc = min(max(-k[c], 0), s.h[c]);
        h[c] = s.h[c] - sc;
        sv = fma(s.pd[c], (double)sc, sv);
    }
    const double S = row_sum(sv);
    const double b_s = fma(S, C.f_s, s.cash);

    // buys: the greedy in ascending stock order, each stock buying the
    // largest q <= k the balance still covers.
    //
    // (1) One bulk round.  Drop every stock that cannot pay for one share
    // (at G = 0 it buys nothing, and G only grows), then find the first
    // pending stock whose full order no longer fits (the misfit): every
    // pending stock before it is bought in full, the misfit buys its largest
    // affordable q < k.
    // (2) The tail, after a misfit: each iteration takes the lowest-index
    // pending stock that can still pay for one share and buys its largest
    // affordable q <= k.  Every purchase so far is of a lower-index stock, so
    // a stock skipped as unaffordable sees the G the serial greedy would give
    // it.  Pending stocks as an 8-bit mask per lane (bit c = stock 8s + c).
    //
    // largest q in [lo, hi] with f_b (g + p q) <= b_s, the answer known to
    // lie in [lo, hi]: an fp32 estimate of (b_s - f_b g) / (f_b p) (off by at
    // most one: the quotient is below 2^15, after a misfit the balance is
    // below one share of it, and the estimate's relative error is about
    // 2^-21), then one step up and one step down with the sign-exact test
    auto largest_q = [&](double g, double p, int lo, int hi) {
        const float rem = (float)fma(-fb, g, b_s);
        const float est = floorf(rem * __builtin_amdgcn_rcpf((float)(p * fb)));
        int qq = (int)fminf(fmaxf(est, (float)lo), (float)hi);
        qq += (qq < hi && fma(fb, g + p * (double)(qq + 1), -b_s) <= 0.0) ? 1 : 0;
        qq -= (qq > lo && fma(fb, g + p * (double)qq, -b_s) > 0.0) ? 1 : 0;
        return qq;
    };

    double costp[SPR], pre[SPR], acc = 0.0;
    int pm = 0;
#pragma unroll
    for (int c = 0; c < SPR; ++c) {
        const bool pend = k[c] > 0 && fma(fb, s.pd[c], -b_s) <= 0.0;
        costp[c] = pend ? s.pd[c] * (double)k[c] : 0.0;
        pm |= pend ? 1 << c : 0;
        acc += costp[c];
        pre[c] = acc;
    }
    double G = 0.0;
    if (__ballot(pm != 0) != 0) {
        // exclusive prefix of lane totals within the row (exact)
        const double base = row_inclusive_scan(acc) - acc;
        int bad = 0;   // pending stocks whose prefix no longer fits
#pragma unroll
        for (int c = 0; c < SPR; ++c) bad |= fma(fb, base + pre[c], -b_s) > 0.0 ? 1 << c : 0;
        bad &= pm;
        const int below = row_any_below(bad);
        const bool after = below != 0;          // a lower lane holds the misfit
        const bool at = !after && bad != 0;     // this lane holds it
        const int cf = __builtin_ctz(bad | 0x100);    // its stock on this lane
        const int full = after ? 0 : (at ? pm & ((1 << cf) - 1) : pm);
        double gl = 0.0, gf = 0.0, pf = 0.0;
        int kf = 0;
#pragma unroll
        for (int c = 0; c < SPR; ++c) {
            const bool fc = (full >> c) & 1;
            h[c] += fc ? k[c] : 0;
            gl += fc ? costp[c] : 0.0;
            const bool sel = c == cf;
            gf = sel ? base + pre[c] - costp[c] : gf;
            pf = sel ? s.pd[c] : pf;
            kf = sel ? k[c] : kf;
        }
        // the misfit's purchase, computed by every lane (uniform code) and
        // kept on the misfit's lane
        const int qf = largest_q(gf, pf, 0, kf > 0 ? kf - 1 : 0);
        if (at) {
#pragma unroll
            for (int c = 0; c < SPR; ++c) h[c] += c == cf ? qf : 0;
            gl += pf * (double)qf;
        }
        pm &= ~full & ~(at ? 1 << cf : 0);
        G = row_sum(gl);
        // the tail (no iteration runs for a row without a misfit: its
        // pending mask is empty)
        for (;;) {
            int aff = 0;
#pragma unroll
            for (int c = 0; c < SPR; ++c) aff |= fma(fb, G + s.pd[c], -b_s) <= 0.0 ? 1 << c : 0;
            aff &= pm;
            pm = aff;
            if (__ballot(aff != 0) == 0) break;
            // (the row scan runs on every lane: a cross-lane move must not sit
            // behind a per-lane condition)
            const int below = row_any_below(aff);
            const bool hit = aff != 0 && below == 0;
            const int ct = __builtin_ctz(aff | 0x100);
            double pt = 0.0;
            int kt = 1;
#pragma unroll
            for (int c = 0; c < SPR; ++c) {
                const bool sel = c == ct;
                pt = sel ? s.pd[c] : pt;
                kt = sel ? k[c] : kt;
            }
            const int qt = largest_q(G, pt, 1, kt > 0 ? kt : 1);
            double dg = 0.0;
            if (hit) {
#pragma unroll
                for (int c = 0; c < SPR; ++c) h[c] += c == ct ? qt : 0;
                pm &= ~(1 << ct);
                dg = pt * (double)qt;
            }
            G += row_sum(dg);
        }
    }
    double nb = fma(-fb, G, b_s);
    if (nb < 0.0) nb = 0.0;

    double hv1 = 0.0;
#pragma unroll
    for (int c = 0; c < SPR; ++c) hv1 = fma((double)h[c], qd[c], hv1);
    const double V1 = nb + row_sum(hv1);
    const float r = (float)(C.reward_scale * (V1 - s.value));
    s.cash = nb;
    s.value = V1;
#pragma unroll
    for (int c = 0; c < SPR; ++c) {
        s.h[c] = h[c];
        s.pd[c] = qd[c];
    }
    return r;
}

}  // namespace tpk
