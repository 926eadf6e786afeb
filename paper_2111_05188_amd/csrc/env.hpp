// The stock-trading env step (paper Section 3, eqs. (2)-(4)) on half a
// wavefront.
//
// A 64-lane wavefront steps two envs at once: lanes 0-31 own env A, lanes
// 32-63 env B.  Lane h of a half holds stocks 4h .. 4h+3 (n <= 128), so stock
// order equals (lane, slot) order and a half's lane-order prefix sum is a
// prefix sum in stock index order.  Every collective below works on both
// halves independently, so the two envs share one instruction stream.
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
// the lane-level sums and scans below give the same bits as a serial loop.
// The buy test fma(f_b, X, -b_s) <= 0 rounds once, so its sign is the sign
// of the exact f_b*X - b_s.  Balances therefore agree bit for bit with a
// serial implementation, and so do share counts.
#pragma once

#include "device.hpp"
#include "internal.hpp"

namespace tpk {

constexpr int HALF = 32;   // lanes per env
constexpr int SPL = 4;     // stocks per lane

__device__ __forceinline__ int shares_from_action(float a, int hmax)
{
    const float u = isnan(a) ? 0.0f : fminf(fmaxf(a, -1.0f), 1.0f);
    return (int)truncf(u * (float)hmax);
}

// ---------------------------------------------------------------------------
// Half-wave collectives (all 64 lanes active; each half independent)
// ---------------------------------------------------------------------------

// Inclusive prefix sum within each 32-lane half, in lane order.
__device__ __forceinline__ double half_inclusive_scan(double v)
{
    v += dpp_f64<DPP_ROW_SHR + 1>(v);
    v += dpp_f64<DPP_ROW_SHR + 2>(v);
    v += dpp_f64<DPP_ROW_SHR + 4>(v);
    v += dpp_f64<DPP_ROW_SHR + 8>(v);
    v += dpp_f64<DPP_ROW_BCAST15, 0xA>(v);   // row 0 -> row 1, row 2 -> row 3
    return v;
}

// The value of lane `la` (half A) or 32 + `lb` (half B), seen by its half.
template <typename T>
__device__ __forceinline__ T half_value(T v, int la, int lb, bool upper)
{
    const T a = lane_value(v, la), b = lane_value(v, HALF + lb);
    return upper ? b : a;
}

__device__ __forceinline__ double half_sum(double v, bool upper)
{
    v = half_inclusive_scan(v);
    return half_value(v, HALF - 1, HALF - 1, upper);
}

// Per-env state held by the owning half: lane h keeps stocks 4h .. 4h+3.
struct HalfEnv {
    double cash;      // balance (same on every lane of the half)
    int h[SPL];       // holdings (0 for stocks >= n)
    float p[SPL];     // prices at the current row (0 for stocks >= n)
    double value;     // total asset b + p^T h after the last step
};

// One transition of the env owned by this lane's half.  a[c]: raw actions of
// this lane's stocks; q[c]: their prices at the next row (0 for stocks >= n).
// `live`: this half holds an env to step (an idle half trades nothing).
// `extra`: a per-lane fp64 term summed over the half alongside the step's
// own sums (the caller's log-density); on return it holds the half's total.
// Returns the reward (same on every lane of the half).  All 64 lanes call it.
// NC > 0 fixes the stock count at compile time (C.n otherwise).
template <int NC = 0>
__device__ __forceinline__ float env_step_half(const EnvConst &C, HalfEnv &s,
                                               const float (&a)[SPL],
                                               const float (&q)[SPL], bool live,
                                               int lane, double &extra)
{
    const bool upper = lane >= HALF;
    const int hl = lane & (HALF - 1);
    const int n = NC > 0 ? NC : C.n;
    const double fb = C.f_b;
    int k[SPL];
    double pd[SPL];
#pragma unroll
    for (int c = 0; c < SPL; ++c) {
        const bool v = live && SPL * hl + c < n;
        k[c] = v ? shares_from_action(a[c], C.hmax) : 0;
        pd[c] = (double)s.p[c];
    }

    // value of the holdings before the step, and the sells (fp64; every
    // product p*h is exact); the three half sums share one pass
    double hv = 0.0, sv = 0.0;
    int h[SPL];
#pragma unroll
    for (int c = 0; c < SPL; ++c) {
        hv += (double)s.h[c] * pd[c];
        const int sc = k[c] < 0 ? min(-k[c], s.h[c]) : 0;
        h[c] = s.h[c] - sc;
        sv += pd[c] * (double)sc;
    }
    hv = half_inclusive_scan(hv);
    sv = half_inclusive_scan(sv);
    extra = half_inclusive_scan(extra);
    const double V = s.cash + half_value(hv, HALF - 1, HALF - 1, upper);
    const double S = half_value(sv, HALF - 1, HALF - 1, upper);   // exact
    extra = half_value(extra, HALF - 1, HALF - 1, upper);
    const double b_s = fma(S, C.f_s, s.cash);

    // buys: the greedy in ascending stock order, each stock buying the
    // largest q <= k the balance still covers.  Both halves run the same
    // instruction stream; a half without work idles.
    //
    // (1) One bulk round.  Drop every stock that cannot pay for one share
    // (at G = 0 it buys nothing), then find the first pending stock whose
    // full order no longer fits (the misfit): every pending stock before it
    // is bought in full, the misfit buys its largest affordable q < k.
    // (2) The tail, after a misfit: the remaining balance is below one
    // share of the misfit, so few stocks can still buy.  Each iteration
    // takes the lowest-index pending stock that can pay for one share and
    // buys its largest affordable q <= k.  Every purchase so far is of a
    // lower-index stock, so a stock skipped as unaffordable sees the G the
    // serial greedy would give it, and G only grows: it stays at zero.
    // Pending stocks as a 4-bit mask per lane (bit c = stock 4 hl + c).
    double cost[SPL];
    int pm = 0;
#pragma unroll
    for (int c = 0; c < SPL; ++c) {
        cost[c] = k[c] > 0 ? pd[c] * (double)k[c] : 0.0;
        pm |= k[c] > 0 ? 1 << c : 0;
    }
    // largest q in [lo, hi] with f_b (g + p q) <= b_s, the answer known to
    // lie in [lo, hi]: an fp32 estimate of (b_s - f_b g) / (f_b p) (off by at
    // most one: the quotient is below 2^15, after a misfit the balance is
    // below one share of it, and the relative error of the estimate is about
    // 2^-21), then one step up and one step down with the sign-exact test
    // (g + p q is exact in fp64)
    auto largest_q = [&](double g, double p, int lo, int hi) {
        const float rem = (float)fma(-fb, g, b_s);
        const float est = floorf(rem * __builtin_amdgcn_rcpf((float)(p * fb)));
        int qq = (int)fminf(fmaxf(est, (float)lo), (float)hi);
        qq += (qq < hi && fma(fb, g + p * (double)(qq + 1), -b_s) <= 0.0) ? 1 : 0;
        qq -= (qq > lo && fma(fb, g + p * (double)qq, -b_s) > 0.0) ? 1 : 0;
        return qq;
    };
    double G = 0.0;
#pragma unroll
    for (int c = 0; c < SPL; ++c)
        pm &= fma(fb, pd[c], -b_s) > 0.0 ? ~(1 << c) : ~0;
    if (__ballot(pm != 0) != 0) {
        // lane-local inclusive prefix of the pending full costs, then the
        // half's exclusive prefix of lane totals (all exact)
        double pre[SPL], acc = 0.0;
#pragma unroll
        for (int c = 0; c < SPL; ++c) {
            acc += (pm >> c) & 1 ? cost[c] : 0.0;
            pre[c] = acc;
        }
        const double base = half_inclusive_scan(acc) - acc;
        int bad = 0;   // pending stocks whose prefix no longer fits
#pragma unroll
        for (int c = 0; c < SPL; ++c)
            bad |= fma(fb, base + pre[c], -b_s) > 0.0 ? 1 << c : 0;
        bad &= pm;
        const uint64_t m = __ballot(bad != 0);
        const uint32_t ma = (uint32_t)m, mb = (uint32_t)(m >> 32);
        // the misfit's lane in each half (the last lane when there is none:
        // its running total is then the half's G)
        const int fla = ma ? __ffs(ma) - 1 : HALF - 1;
        const int flb = mb ? __ffs(mb) - 1 : HALF - 1;
        const bool has = (upper ? mb : ma) != 0;
        const int fl = upper ? flb : fla;
        const bool at = has && hl == fl;
        const int cf = bad ? __ffs(bad) - 1 : 0;   // on the misfit's lane: its stock
        // every pending stock before the misfit is bought in full
        const int full = pm & (!has || hl < fl ? 0xF : (at ? (1 << cf) - 1 : 0));
#pragma unroll
        for (int c = 0; c < SPL; ++c) h[c] += (full >> c) & 1 ? k[c] : 0;
        pm &= ~full;
        // the misfit's purchase, computed by every lane for its own first
        // misfitting stock (uniform code) and kept on the misfit's lane
        double gf = base, pf = pd[0];
        int kf = k[0];
#pragma unroll
        for (int c = 0; c < SPL; ++c)
            if (c == cf) {
                pf = pd[c];
                kf = k[c];
                gf = base + pre[c] - cost[c];
            }
        const int qf = largest_q(gf, pf, 0, kf > 0 ? kf - 1 : 0);
        double gnew = base + acc;
        if (at) {
#pragma unroll
            for (int c = 0; c < SPL; ++c) h[c] += c == cf ? qf : 0;
            pm &= ~(1 << cf);
            gnew = gf + pf * (double)qf;
        }
        G = half_value(gnew, fla, flb, upper);
        // the tail (no iteration runs for a half without a misfit: its
        // pending mask is empty)
        for (;;) {
            int aff = 0;
#pragma unroll
            for (int c = 0; c < SPL; ++c)
                aff |= ((pm >> c) & 1) && fma(fb, G + pd[c], -b_s) <= 0.0 ? 1 << c : 0;
            pm = aff;
            const uint64_t mt = __ballot(aff != 0);
            if (mt == 0) break;
            const uint32_t ta = (uint32_t)mt, tb = (uint32_t)(mt >> 32);
            const int la = ta ? __ffs(ta) - 1 : 0, lb = tb ? __ffs(tb) - 1 : 0;
            const bool hit = (upper ? tb : ta) != 0 && hl == (upper ? lb : la);
            const int ct = aff ? __ffs(aff) - 1 : 0;
            double pt = pd[0];
            int kt = k[0];
#pragma unroll
            for (int c = 1; c < SPL; ++c)
                if (c == ct) {
                    pt = pd[c];
                    kt = k[c];
                }
            const int qt = largest_q(G, pt, 1, kt > 0 ? kt : 1);
            double dg = 0.0;
            if (hit) {
#pragma unroll
                for (int c = 0; c < SPL; ++c) h[c] += c == ct ? qt : 0;
                pm &= ~(1 << ct);
                dg = pt * (double)qt;
            }
            G += half_value(dg, la, lb, upper);
        }
    }
    double nb = fma(-fb, G, b_s);
    if (nb < 0.0) nb = 0.0;

    double hv1 = 0.0;
#pragma unroll
    for (int c = 0; c < SPL; ++c) hv1 += (double)h[c] * (double)q[c];
    const double V1 = nb + half_sum(hv1, upper);
    s.cash = nb;
    s.value = V1;
#pragma unroll
    for (int c = 0; c < SPL; ++c) {
        s.h[c] = h[c];
        s.p[c] = q[c];
    }
    return (float)(C.reward_scale * (V1 - V));
}

template <typename T> __device__ __forceinline__ T obs_cvt(float x);
template <> __device__ __forceinline__ float obs_cvt<float>(float x) { return x; }
template <> __device__ __forceinline__ __bf16 obs_cvt<__bf16>(float x) { return to_bf16(x); }

// Observation row [b*cs, p*ps (n), h*ss (n), ind (nI), 0 ... K_pad) written
// by one half: prices and holdings of the lane's stocks, `ind[m]` =
// indicator hl + 32 m for m < IPL, the rest read from `irow` (LDS or
// global).  All lanes of the half call it.
template <typename T, int IPL>
__device__ __forceinline__ void write_obs_half(T *row, const EnvConst &C, double cash,
                                               const int (&h)[SPL], const float (&p)[SPL],
                                               const float (&ind)[IPL], const float *irow,
                                               int hl)
{
    const int n = C.n, nI = C.nI, S = 1 + 2 * n + nI;
    if (hl == 0) row[0] = obs_cvt<T>((float)(cash * (double)C.cash_scale));
#pragma unroll
    for (int c = 0; c < SPL; ++c) {
        const int i = SPL * hl + c;
        if (i < n) {
            row[1 + i] = obs_cvt<T>(p[c] * C.price_scale);
            row[1 + n + i] = obs_cvt<T>((float)h[c] * C.share_scale);
        }
    }
    T *ri = row + 1 + 2 * n;
#pragma unroll
    for (int m = 0; m < IPL; ++m) {
        const int kk = hl + HALF * m;
        if (kk < nI) ri[kk] = obs_cvt<T>(ind[m]);
    }
    for (int kk = HALF * IPL + hl; kk < nI; kk += HALF) ri[kk] = obs_cvt<T>(irow[kk]);
    for (int kk = S + hl; kk < C.K_pad; kk += HALF) row[kk] = obs_cvt<T>(0.0f);
}

// The same row for bf16 observations when n and nI are multiples of 4 and
// the indicator rows are 16-byte aligned, in aligned 8-byte stores of
// columns 4k .. 4k+3: the value of column 4k belongs to the neighbouring
// chunk's owner and comes by shuffle.  Lane s < n/4 (stocks 4s .. 4s+3)
// writes columns 4s .. +3 = [price 4s-1, prices 4s .. 4s+2] and n + 4s ..
// +3 = [holding 4s-1, holdings 4s .. 4s+2] (lane 0: the balance, the last
// price); indicator chunk k (lane k % 32) writes columns 2n + 4k .. +3 =
// [indicator 4k-1, indicators 4k .. 4k+2] (chunk 0: the last holding),
// zeros past the last indicator; then the zero padding.  Every lane of
// the wave calls it (it shuffles; irow must be readable for every half);
// halves with `live` false store nothing.
// Indicator chunks of the aligned writer below, loaded ahead of use: round
// m holds chunk hl + 32 m of the row (clamped to the last chunk), for up to
// MAXR rounds (nI / 4 + 1 <= 32 MAXR).  Issuing these loads before the env
// step lets their latency overlap the step's arithmetic.
template <int MAXR>
struct IndChunks {
    float __attribute__((ext_vector_type(4))) v[MAXR];
};

template <int MAXR>
__device__ __forceinline__ IndChunks<MAXR> load_ind_chunks(const EnvConst &C, const float *irow, int hl)
{
    typedef float f4 __attribute__((ext_vector_type(4)));
    IndChunks<MAXR> r;
    const int nch = C.nI / 4 + 1, rounds = (nch + HALF - 1) / HALF;
#pragma unroll
    for (int m = 0; m < MAXR; ++m)
        r.v[m] = m < rounds ? *(const f4 *)(irow + 4 * min(hl + HALF * m, C.nI / 4 - 1))
                            : f4{0.f, 0.f, 0.f, 0.f};
    return r;
}

// The same row for bf16 observations when n and nI are multiples of 4 (nI
// > 0) and the indicator rows are 16-byte aligned, in aligned 8-byte stores
// of columns 4k .. 4k+3: the value of column 4k belongs to the neighbouring
// chunk's owner and comes by shuffle.  Lane s < n/4 (stocks 4s .. 4s+3)
// writes columns 4s .. +3 = [price 4s-1, prices 4s .. 4s+2] and n + 4s ..
// +3 = [holding 4s-1, holdings 4s .. 4s+2] (lane 0: the balance, the last
// price); indicator chunk k (lane k % 32) writes columns 2n + 4k .. +3 =
// [indicator 4k-1, indicators 4k .. 4k+2] (chunk 0: the last holding),
// zeros past the last indicator; then the zero padding.  `ind` holds the
// row's chunks (load_ind_chunks).  Every lane of the wave calls it (it
// shuffles); halves with `live` false store nothing.
template <int MAXR>
__device__ __forceinline__ void write_obs_half_aligned(__bf16 *row, const EnvConst &C, double cash,
                                                       const int (&h)[SPL],
                                                       const float (&p)[SPL],
                                                       const IndChunks<MAXR> &ind, int lane,
                                                       int hl, bool live)
{
    typedef float f4 __attribute__((ext_vector_type(4)));
    const int n = C.n, nI = C.nI, nq = n / 4, base = lane - hl;
    float pv[SPL], hv[SPL];
#pragma unroll
    for (int c = 0; c < SPL; ++c) {
        pv[c] = p[c] * C.price_scale;
        hv[c] = (float)h[c] * C.share_scale;
    }
    const int up = lane - (hl > 0);
    const float p_up = __shfl(pv[3], up), h_up = __shfl(hv[3], up);
    const float p_last = __shfl(pv[3], base + nq - 1), h_last = __shfl(hv[3], base + nq - 1);
    const int nch = nI / 4 + 1, rounds = (nch + HALF - 1) / HALF;
    float last3 = 0.f;
#pragma unroll
    for (int m = 0; m < MAXR; ++m) {   // the same trip count in every lane
        if (m >= rounds) break;
        const int k = hl + HALF * m;
        const f4 v = ind.v[m];
        const float v_up = __shfl(v[3], up), v_wrap = __shfl(last3, base + HALF - 1);
        const float first = hl > 0 ? v_up : (m > 0 ? v_wrap : h_last);
        if (live && k < nch) {
            const bool own = k < nI / 4;
            *(bf16x4 *)(row + 2 * n + 4 * k) =
                bf16x4{to_bf16(first), to_bf16(own ? v[0] : 0.f), to_bf16(own ? v[1] : 0.f),
                       to_bf16(own ? v[2] : 0.f)};
        }
        last3 = v[3];
    }
    if (!live) return;
    if (hl < nq) {
        const float bal = (float)(cash * (double)C.cash_scale);
        *(bf16x4 *)(row + 4 * hl) = bf16x4{to_bf16(hl > 0 ? p_up : bal), to_bf16(pv[0]),
                                           to_bf16(pv[1]), to_bf16(pv[2])};
        *(bf16x4 *)(row + n + 4 * hl) = bf16x4{to_bf16(hl > 0 ? h_up : p_last), to_bf16(hv[0]),
                                               to_bf16(hv[1]), to_bf16(hv[2])};
    }
    const bf16x4 zero = {to_bf16(0.f), to_bf16(0.f), to_bf16(0.f), to_bf16(0.f)};
    for (int c4 = (2 * n) / 4 + nch + hl; c4 < C.K_pad / 4; c4 += HALF)
        *(bf16x4 *)(row + 4 * c4) = zero;
}

// Copy `bytes` (a multiple of 16) with 16-byte accesses, lanes l = 0..nl-1
// of the calling group participating.
__device__ __forceinline__ void copy16(void *dst, const void *src, size_t bytes,
                                       int l, int nl)
{
    const uint4 *s = (const uint4 *)src;
    uint4 *d = (uint4 *)dst;
    for (size_t i = l; i < bytes / 16; i += nl) d[i] = s[i];
}

}  // namespace tpk
