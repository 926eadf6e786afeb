// Role-split fused rollout kernel for bf16 actors of the shapes in use
// (1001 inputs from 100 stocks with 8 indicators each, 512- or 1024-wide
// hidden layers).  One launch runs all L lockstep steps of a block of 16 envs.
//
// Why split roles.  A workgroup owns 16 envs, the N dimension of one MFMA
// tile, so every step streams the whole actor (1.65 MB at 1001-512-512-100)
// from L2 into the CU.  That stream, not the MFMAs, bounds the actor, and the
// env step is VALU work of about the same length.  Run back to back they add
// up; here they overlap.  The observation is [balance, prices, holdings,
// indicators] (Section 3, "State space"), and layer 1's columns past the
// first KSB k-steps of 32 hold only indicators of the market row.  Those do
// not depend on the actions, so their share of layer 1 for step j+1 can be
// computed while the env step of step j runs.  Only the first KSB k-steps of
// layer 1, layers 2 and 3 remain on the step-to-step chain.
//
// Waves.  Four matrix waves (one per SIMD) compute every actor layer; eight
// env waves (two per SIMD) own two envs each, one per 32-lane half, four
// stocks per lane.  Each role runs its own loop with the same barrier
// sequence: per step, four slots separated by workgroup barriers:
//
//   slot   matrix waves                         env waves
//   A      Z = W1[:, KSB..] x_j  (indicators)   env step j-1, trajectory row j-1,
//                                               balance/prices/holdings of x_j;
//                                               x_j to HBM; loads of row t+j+1
//   B      h1 = tanh(Z + W1[:, ..KSB] x_j + b1) -
//   L2     h2 = tanh(W2 h1 + b2)                indicators of row t+j+1 into x_{j+1};
//                                               Philox + Box-Muller normals of step j
//   L3     mu = W3 h2 + b3                      -
//
// LDS: x rows (bf16), h1 (bf16), Z (fp32) sharing its space with h2 (their
// lifetimes, slots A->B and L2->L3, do not overlap), mu (fp32), biases.
//
// Weight stream.  A matrix wave consumes a fixed sequence of F weight
// fragments per step (1 KiB each: one 16x32 A-operand of
// v_mfma_f32_16x16x32_bf16, 16 bytes per lane) through a ring of R fragment
// registers: consuming fragment f issues the load of fragment f + R, wrapping
// into the next step's sequence (the weights do not change during a
// rollout), so loads stay in flight across group ends, layer ends and
// barriers, and nothing is read twice.  Fragments come through buffer loads
// with a wave-uniform scalar offset.
#include <type_traits>

#include "device.hpp"
#include "env.hpp"
#include "internal.hpp"

namespace tpk {
namespace rs {

constexpr int MW = 4;            // matrix waves
constexpr int VW = 8;            // env waves
constexpr int NWAVES = MW + VW;
constexpr int MB = 2 * VW;       // envs per workgroup
constexpr int G = 4;             // output tiles per group in layers 1 and 2

template <int I> using ic = std::integral_constant<int, I>;

typedef float f4v __attribute__((ext_vector_type(4)));
typedef int i4v __attribute__((ext_vector_type(4)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));

// Market rows and trajectory rows are touched once per step; streaming
// (non-temporal) accesses keep them from evicting the actor's weights,
// which every step reads again, from L2.
__device__ __forceinline__ f4v load_stream(const float *p)
{
    return __builtin_nontemporal_load((const f4v *)p);
}
template <class T>
__device__ __forceinline__ void store_stream(T v, T *p)
{
    __builtin_nontemporal_store(v, p);
}

template <int B, int E, typename Fn>
__device__ __forceinline__ void static_for(Fn &&fn)
{
    if constexpr (B < E) {
        fn(ic<B>{});
        static_for<B + 1, E>(fn);
    }
}

// Actor shape.  NS stocks with NI indicator values per market row; KS1
// k-steps of 32 inputs in layer 1, the first KSB of which hold the balance,
// prices and holdings; NT1, NT2, NT3 output tiles of 16; a ring of R weight
// fragments per matrix wave.
template <int NS_, int NI_, int KS1_, int KSB_, int NT1_, int NT2_, int NT3_, int R_>
struct Shape {
    static constexpr int NS = NS_, NI = NI_;   // stocks, indicator values per row
    static constexpr int R = R_;
    static constexpr int KS1 = KS1_, KSB = KSB_, KSA = KS1_ - KSB_;
    static constexpr int NT1 = NT1_, NT2 = NT2_, NT3 = NT3_;
    static constexpr int KS2 = NT1 / 2, KS3 = NT2 / 2;
    static constexpr int NG1 = NT1 / (MW * G), NG2 = NT2 / (MW * G), NG3 = NT3 / MW;
    static_assert(NT1 % (MW * G) == 0 && NT2 % (MW * G) == 0 && NT3 % MW == 0,
                  "tiles must split evenly over the matrix waves");
    // fragments per step of one matrix wave, in consumption order A, B, L2, L3
    static constexpr int FA = NG1 * KSA * G, FB = NG1 * KSB * G;
    static constexpr int F2 = NG2 * KS2 * G, F3 = NG3 * KS3;
    static constexpr int F = FA + FB + F2 + F3;
    static_assert(F % R == 0, "the ring must map every fragment to a fixed slot");

    // layer of fragment f, and its byte offset from the wave's base in that
    // layer (the wave's first tile; groups are MW * G tiles apart in layers
    // 1 and 2, MW tiles apart in layer 3)
    static constexpr int layer(int f) { return f < FA + FB ? 0 : (f < FA + FB + F2 ? 1 : 2); }
    static constexpr int offset(int f)
    {
        if (f < FA) {
            const int g = f / (KSA * G), r = f % (KSA * G);
            return ((g * MW * G + r % G) * KS1 + KSB + r / G) * 1024;
        }
        f -= FA;
        if (f < FB) {
            const int g = f / (KSB * G), r = f % (KSB * G);
            return ((g * MW * G + r % G) * KS1 + r / G) * 1024;
        }
        f -= FB;
        if (f < F2) {
            const int g = f / (KS2 * G), r = f % (KS2 * G);
            return ((g * MW * G + r % G) * KS2 + r / G) * 1024;
        }
        f -= F2;
        return ((f / KS3) * MW * KS3 + f % KS3) * 1024;
    }
};

__device__ __forceinline__ bf16x8 as_bf16x8(uint32_t __attribute__((ext_vector_type(4))) v)
{
    return __builtin_bit_cast(bf16x8, v);
}

struct Lds {
    __bf16 *X;      // [MB][ldx]   observations
    __bf16 *H1;     // [MB][ldh1]  hidden layer 1
    float *Z;       // [MB][ldz]   indicator part of layer 1 (shares space with H2)
    __bf16 *H2;     // [MB][ldh2]  hidden layer 2
    float *MU;      // [MB][ldmu]  action means
    float *BIAS;    // b1 | b2 | b3
    int ldx, ldh1, ldz, ldh2, ldmu;
};

// ---------------------------------------------------------------------------
// Matrix role
// ---------------------------------------------------------------------------
// One matrix wave's weight stream.  Fragment i of the step sequence lives in
// ring slot i % R; consuming fragment i first refills the slot fragment i-1
// left (its MFMA has issued), then multiplies, so R-1 loads stay in flight.
template <class S>
struct Stream {
    static constexpr int R = S::R;
    __amdgpu_buffer_rsrc_t rsrc;
    int wb0, wb1, wb2;   // wave's byte base in each layer
    int voff;
    bf16x8 ring[R];

    template <int I>
    __device__ __forceinline__ void fetch()
    {
        constexpr int f = I % S::F, slot = I % R, L = S::layer(f);
        const int base = L == 0 ? wb0 : (L == 1 ? wb1 : wb2);
        ring[slot] = as_bf16x8(
            __builtin_amdgcn_raw_buffer_load_b128(rsrc, voff, base + S::offset(f), 0));
    }

    template <int I>
    __device__ __forceinline__ void mma(const bf16x8 &x, floatx4 &acc)
    {
        fetch<I + R - 1>();
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ring[I % R], x, acc, 0, 0, 0);
    }

    // The fragment offsets base + constant are loop-invariant; hoisted out
    // of the step loop they would need one scalar register each.  Hiding
    // the bases from the optimiser at every slot keeps each offset next to
    // its load.
    __device__ __forceinline__ void launder() { asm volatile("" : "+s"(wb0), "+s"(wb1), "+s"(wb2)); }

    // One slot's work: NG groups of GT output tiles over KS k-steps that
    // start at k-step K0 of the input rows `xb` (this lane's row and column
    // offset).  init(g, acc) and epi(g, t, acc) set up and store group g.
    // With DEFER the epilogue of group g runs tile by tile inside the first
    // GT k-steps of group g+1, so the weight stream keeps moving through it.
    template <int FB0, int NG, int KS, int K0, int GT, bool DEFER, class InitF, class EpiF>
    __device__ __forceinline__ void seg(const __bf16 *xb, InitF &&init, EpiF &&epi)
    {
        static_assert(!DEFER || KS >= GT, "deferred epilogue needs a k-step per tile");
        floatx4 acc[GT], prev[GT];
        static_for<0, NG>([&](auto gi) {
            constexpr int g = decltype(gi)::value;
            init(g, acc);
            bf16x8 x = *(const bf16x8 *)(xb + K0 * 32);
            static_for<0, KS>([&](auto ki) {
                constexpr int k = decltype(ki)::value;
                bf16x8 xn;
                if constexpr (k + 1 < KS) xn = *(const bf16x8 *)(xb + (K0 + k + 1) * 32);
                static_for<0, GT>([&](auto ti) {
                    constexpr int t = decltype(ti)::value;
                    mma<FB0 + (g * KS + k) * GT + t>(x, acc[t]);
                });
                if constexpr (DEFER && g > 0 && k < GT) epi(g - 1, k, prev[k]);
                if constexpr (k + 1 < KS) x = xn;
                __builtin_amdgcn_sched_barrier(0);
            });
            if constexpr (DEFER && g + 1 < NG) {
#pragma unroll
                for (int t = 0; t < GT; ++t) prev[t] = acc[t];
            } else {
#pragma unroll
                for (int t = 0; t < GT; ++t) epi(g, t, acc[t]);
            }
        });
    }
};

template <class S>
__device__ __forceinline__ void matrix_role(const RolloutArgs &A, const Lds &s,
                                            const uint8_t *pk, int m, int lane)
{
    const PackedLayout &P = A.lay;
    const int r16 = lane & 15, kq = lane >> 4;
    // biases in LDS; those of the tanh layers pre-scaled by -2 log2(e)
    float *b1 = s.BIAS, *b2 = b1 + S::NT1 * 16, *b3 = b2 + S::NT2 * 16;
    {
        const float *src = (const float *)(pk + P.off_b[0]);
        for (int i = m * WAVE + lane; i < S::NT1 * 16; i += MW * WAVE) b1[i] = NEG_2LOG2E * src[i];
        src = (const float *)(pk + P.off_b[1]);
        for (int i = m * WAVE + lane; i < S::NT2 * 16; i += MW * WAVE) b2[i] = NEG_2LOG2E * src[i];
        src = (const float *)(pk + P.off_b[2]);
        for (int i = m * WAVE + lane; i < S::NT3 * 16; i += MW * WAVE) b3[i] = src[i];
    }

    Stream<S> st;
    st.rsrc = __builtin_amdgcn_make_buffer_rsrc((void *)pk, (short)0, (int)P.agent_stride,
                                                0x00020000);
    st.wb0 = (int)P.off_W[0] + m * G * S::KS1 * 1024;
    st.wb1 = (int)P.off_W[1] + m * G * S::KS2 * 1024;
    st.wb2 = (int)P.off_W[2] + m * S::KS3 * 1024;
    st.voff = lane * 16;

    const __bf16 *xb = s.X + r16 * s.ldx + kq * 8;
    const __bf16 *h1b = s.H1 + r16 * s.ldh1 + kq * 8;
    const __bf16 *h2b = s.H2 + r16 * s.ldh2 + kq * 8;
    // output column of tile t of group g, for this lane, in layers 1-2 / 3
    auto col12 = [&](int g, int t) { return ((g * MW + m) * G + t) * 16 + kq * 4; };
    auto col3 = [&](int g) { return (g * MW + m) * 16 + kq * 4; };
    auto zero = [&](int, floatx4 *acc) {
#pragma unroll
        for (int t = 0; t < G; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
    };
    auto tanh_store = [&](const floatx4 &a, const float *bs, __bf16 *Y, int o) {
        const floatx4 bv = *(const floatx4 *)(bs + o);
        const bf16x4 h = {to_bf16(tanh_from_e2(fmaf(a[0], NEG_2LOG2E, bv[0]))),
                          to_bf16(tanh_from_e2(fmaf(a[1], NEG_2LOG2E, bv[1]))),
                          to_bf16(tanh_from_e2(fmaf(a[2], NEG_2LOG2E, bv[2]))),
                          to_bf16(tanh_from_e2(fmaf(a[3], NEG_2LOG2E, bv[3])))};
        *(bf16x4 *)(Y + o) = h;
    };

    // slot A: Z = W1[:, KSB..] x (fp32, no bias)
    auto seg_A = [&]() {
        st.template seg<0, S::NG1, S::KSA, S::KSB, G, false>(
            xb, zero, [&](int g, int t, const floatx4 &a) {
                *(floatx4 *)(s.Z + r16 * s.ldz + col12(g, t)) = a;
            });
    };
    // slot B: h1 = tanh(Z + W1[:, ..KSB] x + b1)
    auto seg_B = [&]() {
        st.template seg<S::FA, S::NG1, S::KSB, 0, G, true>(
            xb,
            [&](int g, floatx4 *acc) {
#pragma unroll
                for (int t = 0; t < G; ++t) acc[t] = *(const floatx4 *)(s.Z + r16 * s.ldz + col12(g, t));
            },
            [&](int g, int t, const floatx4 &a) { tanh_store(a, b1, s.H1 + r16 * s.ldh1, col12(g, t)); });
    };
    // slot L2: h2 = tanh(W2 h1 + b2)
    auto seg_L2 = [&]() {
        st.template seg<S::FA + S::FB, S::NG2, S::KS2, 0, G, true>(
            h1b, zero,
            [&](int g, int t, const floatx4 &a) { tanh_store(a, b2, s.H2 + r16 * s.ldh2, col12(g, t)); });
    };
    // slot L3: mu = W3 h2 + b3
    auto seg_L3 = [&]() {
        st.template seg<S::FA + S::FB + S::F2, S::NG3, S::KS3, 0, 1, false>(
            h2b, [&](int, floatx4 *acc) { acc[0] = floatx4{0.f, 0.f, 0.f, 0.f}; },
            [&](int g, int, const floatx4 &a) {
                const int o = col3(g);
                const floatx4 bv = *(const floatx4 *)(b3 + o);
                *(floatx4 *)(s.MU + r16 * s.ldmu + o) =
                    floatx4{a[0] + bv[0], a[1] + bv[1], a[2] + bv[2], a[3] + bv[3]};
            });
    };

    // the first R-1 fragments; the rest is fetched one slot behind use
    static_for<0, S::R - 1>([&](auto i) { st.template fetch<decltype(i)::value>(); });
    __syncthreads();   // observations of step 0 and the biases are in LDS
    for (int j = 0; j < A.L; ++j) {
        st.launder();
        seg_A();
        __syncthreads();
        st.launder();
        seg_B();
        __syncthreads();
        st.launder();
        seg_L2();
        __syncthreads();
        st.launder();
        seg_L3();
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// Env role
// ---------------------------------------------------------------------------
// Balance, prices and holdings of an observation row (the indicator part is
// written separately, one slot earlier).
// Balance, prices and holdings of an observation row (columns 0 .. 2n; the
// indicator part is written separately, one slot earlier), in aligned
// 8-byte stores: lane s (s < n / 4, owner of stocks 4s .. 4s+3) writes
// columns 4s .. 4s+3 = [price 4s-1 (lane s-1's last), prices 4s .. 4s+2]
// and columns n + 4s .. n + 4s + 3 = [holding 4s-1, holdings 4s .. 4s+2];
// lane 0 starts the first with the balance and the second with the last
// price; column 2n (the last holding) is one 2-byte store.  All lanes of
// the wave call it (it shuffles); only `live` halves store.
template <int n>
__device__ __forceinline__ void write_obs_state(__bf16 *row, const EnvConst &C, double cash,
                                                const int (&h)[SPL], const float (&p)[SPL],
                                                int lane, int hl, bool live)
{
    static_assert(n % 4 == 0 && n / 4 <= HALF, "one chunk of each kind per lane");
    float pv[SPL], hv[SPL];
#pragma unroll
    for (int c = 0; c < SPL; ++c) {
        pv[c] = p[c] * C.price_scale;
        hv[c] = (float)h[c] * C.share_scale;
    }
    const int base = lane - hl;
    const float p_up = __shfl(pv[3], lane - (hl > 0)), h_up = __shfl(hv[3], lane - (hl > 0));
    const float p_last = __shfl(pv[3], base + n / 4 - 1), h_last = __shfl(hv[3], base + n / 4 - 1);
    if (!live || hl >= n / 4) return;
    const float bal = (float)(cash * (double)C.cash_scale);
    *(bf16x4 *)(row + 4 * hl) = bf16x4{to_bf16(hl > 0 ? p_up : bal), to_bf16(pv[0]), to_bf16(pv[1]),
                                       to_bf16(pv[2])};
    *(bf16x4 *)(row + n + 4 * hl) = bf16x4{to_bf16(hl > 0 ? h_up : p_last), to_bf16(hv[0]),
                                           to_bf16(hv[1]), to_bf16(hv[2])};
    if (hl == n / 4 - 1) row[2 * n] = to_bf16(h_last);
}

template <int NS, int NI, int KPAD>
__device__ __forceinline__ void env_role(const RolloutArgs &A, const Lds &s, const uint8_t *pk,
                                         int agent, int ebase, int nenv, int v, int lane)
{
    // NS stocks (a multiple of 4, at most 128), NI = NS * indicators (a
    // multiple of 4), observation rows of KPAD elements
    static_assert(NS % SPL == 0 && NS <= SPL * HALF && NI % 4 == 0, "shape");
    constexpr int IPC = (NI / 4 + HALF - 1) / HALF;   // 16-byte indicator chunks per lane
    constexpr int OBS_CHUNKS = KPAD * 2 / 16;         // 16-byte chunks of an observation row
    const EnvConst &C = A.env;
    const PackedLayout &P = A.lay;
    constexpr int n = NS, nI = NI;
    const int half = lane / HALF, hl = lane % HALF;
    const int sl = 2 * v + half;
    const bool mine = sl < nenv;
    const int e = ebase + sl;
    __bf16 *xrow = s.X + sl * s.ldx;
    const size_t E = (size_t)A.E;
    const float qnan = __builtin_nanf("");

    float ls[SPL], sg[SPL];
    {
        const float *lsd = (const float *)(pk + P.off_ls);
#pragma unroll
        for (int c = 0; c < SPL; ++c) {
            const int i = SPL * hl + c;
            ls[c] = i < n ? lsd[i] : 0.f;
            sg[c] = expf(ls[c]);
        }
    }

    // state of this half's env, kept in registers for the whole rollout
    HalfEnv st;
    st.cash = 0.0;
    int64_t t0 = 0;
    bool live = false;
#pragma unroll
    for (int c = 0; c < SPL; ++c) {
        st.h[c] = 0;
        st.p[c] = 0.f;
    }
    if (mine) {
        t0 = A.t[e];
        live = t0 >= 0 && t0 + A.L <= C.T1 - 1;
        if (A.n_invalid && !live && hl == 0) atomicAdd(A.n_invalid, 1);
        st.cash = A.cash[e];
#pragma unroll
        for (int c = 0; c < SPL; ++c) {
            const int i = SPL * hl + c;
            st.h[c] = i < n ? A.shares[(size_t)e * n + i] : 0;
        }
        if (live) {
            const float *prow = C.price + (size_t)t0 * n;
            const float *irow = C.ind + (size_t)t0 * nI;
#pragma unroll
            for (int c = 0; c < SPL; ++c) {
                const int i = SPL * hl + c;
                st.p[c] = i < n ? prow[i] : 0.f;
            }
            float ind1[1];
            ind1[0] = hl < nI ? irow[hl] : 0.f;
            write_obs_half<__bf16, 1>(xrow, C, st.cash, st.h, st.p, ind1, irow, hl);
        }
    }
    const bool wave_live = __ballot(live) != 0;
    const double half_log2pi_n = 0.5 * (double)n * 1.8378770664093454836;
    const int obs_bytes = C.K_pad * 2;

    float z[SPL], q[SPL];
#pragma unroll
    for (int c = 0; c < SPL; ++c) z[c] = q[c] = 0.f;

    // env step of step jj: action, log-density, trade, trajectory row jj and
    // the balance / prices / holdings of observation jj + 1
    auto step_env = [&](int jj) {
        const float *mu = s.MU + sl * s.ldmu;
        float a[SPL];
        double lp = 0.0;
#pragma unroll
        for (int c = 0; c < SPL; ++c) {
            const int i = SPL * hl + c;
            const bool ok = live && i < n;
            a[c] = ok ? mu[i] + sg[c] * z[c] : 0.f;
            if (ok) lp += -0.5 * (double)z[c] * (double)z[c] - (double)ls[c];
        }
        float qq[SPL];
#pragma unroll
        for (int c = 0; c < SPL; ++c) qq[c] = (live && SPL * hl + c < n) ? q[c] : 0.f;
        float r = 0.f;
        if (wave_live) r = env_step_half<NS>(C, st, a, qq, live, lane, lp);
        lp -= half_log2pi_n;
        write_obs_state<NS>(xrow, C, st.cash, st.h, st.p, lane, hl, live);
        if (!mine) return;
        const size_t row = (size_t)jj * E + e;
        const uint8_t done = (uint8_t)(A.step0 + (uint64_t)jj + 1 == (uint64_t)C.horizon);
        // this lane's 4 stocks are 16 contiguous bytes of the action row
        if (hl < NS / SPL) {
            const f4v av = live ? f4v{a[0], a[1], a[2], a[3]} : f4v{qnan, qnan, qnan, qnan};
            store_stream(av, (f4v *)(A.action + row * n) + hl);
            if (A.mu_tap)
                store_stream(live ? *(const f4v *)(mu + SPL * hl) : f4v{qnan, qnan, qnan, qnan},
                             (f4v *)(A.mu_tap + row * n) + hl);
            if (A.shares_tap)
                store_stream(i4v{st.h[0], st.h[1], st.h[2], st.h[3]},
                             (i4v *)(A.shares_tap + row * n) + hl);
        }
        if (hl == 0) {
            store_stream(live ? (float)lp : qnan, A.logp + row);
            store_stream(live ? r : qnan, A.reward + row);
            store_stream(live ? done : (uint8_t)0, A.done + row);
            if (A.cash_tap) store_stream(st.cash, A.cash_tap + row);
            if (A.asset_tap) store_stream(live ? st.value : (double)qnan, A.asset_tap + row);
        }
    };

    __syncthreads();   // observations of step 0 are in LDS
    f4v ind[IPC];
    for (int j = 0; j < A.L; ++j) {
        // slot A: env step of step j-1, which completes x_j (the matrix
        // waves read only the indicator columns of x_j meanwhile); then
        // this step's memory traffic, kept out of the short slot B where
        // it would hold up the weight stream: x_j to HBM, loads of row
        // t0+j+1 (which exists for a stepped env; others read row 0)
        if (j > 0) step_env(j - 1);
        if (live && A.obs) {
            const u4v *src = (const u4v *)xrow;
            u4v *dst = (u4v *)((__bf16 *)A.obs + ((size_t)j * E + e) * A.ld_obs);
#pragma unroll
            for (int c = hl; c < OBS_CHUNKS; c += HALF) store_stream(src[c], dst + c);
        }
        {
            const int64_t t1 = live ? t0 + j + 1 : 0;
            const float *pr = C.price + (size_t)t1 * NS;
            const float *ir = C.ind + (size_t)t1 * NI;
            const f4v qv = load_stream(pr + SPL * min(hl, NS / SPL - 1));
#pragma unroll
            for (int c = 0; c < SPL; ++c) q[c] = qv[c];
#pragma unroll
            for (int mm = 0; mm < IPC; ++mm) ind[mm] = load_stream(ir + 4 * min(hl + HALF * mm, NI / 4 - 1));
        }
        __syncthreads();

        // slot B: nothing for the env waves
        __syncthreads();

        // slot L2: indicators of row t0+j+1 into x_{j+1} (the matrix waves
        // are done with x_j); the normals of step j
        {
            // 8-byte stores of columns 2n + 4k .. +3 for chunks k = hl + HALF mm
            // <= nI / 4: indicator values 4k - 1 .. 4k + 2 (indicator i sits in
            // column 2n + 1 + i).  Value 4k - 1 is element 3 of chunk k - 1, from
            // the neighbouring lane of this half-wave.  Column 2n (the last
            // holding) gets a placeholder that slot A overwrites before anything
            // reads it; the columns past the last indicator are zero padding.
            static_assert(n % 4 == 0, "chunk starts are 8-byte aligned");
            constexpr int NCH = nI / 4 + 1;
            constexpr int IPW = (NCH + HALF - 1) / HALF;
            const int base = lane - hl;   // this half-wave's first lane
            float prev[IPW];
#pragma unroll
            for (int mm = 0; mm < IPW; ++mm) {
                const float up = mm < IPC ? __shfl(ind[mm < IPC ? mm : 0][3], lane - (hl > 0)) : 0.f;
                const float wrap = mm > 0 ? __shfl(ind[mm - 1 < IPC ? mm - 1 : 0][3], base + HALF - 1)
                                          : 0.f;
                prev[mm] = hl > 0 ? up : wrap;
            }
            if (live) {
                __bf16 *rc = xrow + 2 * n;
#pragma unroll
                for (int mm = 0; mm < IPW; ++mm) {
                    const int k = hl + HALF * mm;
                    if (k < NCH) {
                        const bool own = k < nI / 4;
                        const f4v v = mm < IPC ? ind[mm < IPC ? mm : 0] : f4v{0.f, 0.f, 0.f, 0.f};
                        *(bf16x4 *)(rc + 4 * k) =
                            bf16x4{to_bf16(prev[mm]), to_bf16(own ? v[0] : 0.f),
                                   to_bf16(own ? v[1] : 0.f), to_bf16(own ? v[2] : 0.f)};
                    }
                }
            }
        }
        {
            const U4 w = philox4x32_10(
                U4{(uint32_t)hl, (uint32_t)e, (uint32_t)(A.step0 + (uint64_t)j), (uint32_t)agent},
                A.key_lo, A.key_hi);
            box_muller_hw(uniform_open01(w.x), uniform_open01(w.y), z[0], z[1]);
            box_muller_hw(uniform_open01(w.z), uniform_open01(w.w), z[2], z[3]);
        }
        __syncthreads();

        // slot L3: nothing for the env waves
        __syncthreads();
    }
    step_env(A.L - 1);

    if (mine && live) {
        if (A.obs_last) copy16((__bf16 *)A.obs_last + (size_t)e * A.ld_obs, xrow, obs_bytes, hl, HALF);
        if (hl == 0) {
            A.cash[e] = st.cash;
            A.t[e] = t0 + A.L;
        }
#pragma unroll
        for (int c = 0; c < SPL; ++c) {
            const int i = SPL * hl + c;
            if (i < n) A.shares[(size_t)e * n + i] = st.h[c];
        }
    }
}

template <class S>
__global__ __launch_bounds__(NWAVES *WAVE) void rollout_rs_kernel(RolloutArgs A)
{
    extern __shared__ __align__(16) uint8_t smem[];
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / WAVE));
    const int lane = threadIdx.x % WAVE;

    // XCD-aware block order (consecutive dispatch slots of one XCD take
    // consecutive logical blocks)
    const int nb = gridDim.x;
    const int logical = (blockIdx.x % 8) * (nb / 8) + blockIdx.x / 8;
    if (logical >= A.n_agents * A.blocks_per_agent) return;
    const int agent = logical / A.blocks_per_agent;
    const int blk = logical % A.blocks_per_agent;
    const int ebase = agent * A.envs_per_agent + blk * MB;
    const int nenv = min(MB, A.envs_per_agent - blk * MB);
    const uint8_t *pk = A.packed + (size_t)agent * A.lay.agent_stride;

    Lds s;
    s.X = (__bf16 *)(smem + A.lds_X);
    s.H1 = (__bf16 *)(smem + A.lds_H);
    s.Z = (float *)(smem + A.lds_Z);
    s.H2 = (__bf16 *)(smem + A.lds_Z);
    s.MU = (float *)(smem + A.lds_MU);
    s.BIAS = (float *)(smem + A.lds_B);
    s.ldx = A.ldx;
    s.ldh1 = A.ldh;
    s.ldz = A.ldz;
    s.ldh2 = A.ldh2;
    s.ldmu = A.ldmu;

    // zero the observation rows (padding columns and rows of absent envs
    // stay zero)
    for (int i = threadIdx.x; i < MB * s.ldx * 2 / 16; i += NWAVES * WAVE)
        ((uint4 *)s.X)[i] = uint4{0, 0, 0, 0};
    __syncthreads();

    if (wave < MW)
        matrix_role<S>(A, s, pk, wave, lane);
    else
        env_role<S::NS, S::NI, S::KS1 * 32>(A, s, pk, agent, ebase, nenv, wave - MW, lane);
}

template <class S>
hipError_t launch(RolloutArgs &a, hipStream_t st)
{
    const PackedLayout &P = a.lay;
    a.ldx = S::KS1 * 32 + 8;
    a.ldh = S::NT1 * 16 + 8;
    a.ldz = S::NT1 * 16 + 4;
    a.ldh2 = S::NT2 * 16 + 8;
    a.ldmu = S::NT3 * 16 + 4;
    auto al = [](size_t x) { return (x + 15) & ~(size_t)15; };
    size_t off = 0;
    a.lds_X = off;  off = al(off + (size_t)MB * a.ldx * 2);
    a.lds_H = off;  off = al(off + (size_t)MB * a.ldh * 2);
    a.lds_Z = off;
    {
        const size_t z = (size_t)MB * a.ldz * 4, h2 = (size_t)MB * a.ldh2 * 2;
        off = al(off + (z > h2 ? z : h2));
    }
    a.lds_MU = off; off = al(off + (size_t)MB * a.ldmu * 4);
    a.lds_B = off;  off = al(off + (size_t)(S::NT1 + S::NT2 + S::NT3) * 16 * 4);
    a.lds_bytes = off;
    if (off > LDS_LIMIT) return hipErrorInvalidConfiguration;
    if (P.KS[0] != S::KS1 || P.NT[0] != S::NT1 || P.NT[1] != S::NT2 || P.NT[2] != S::NT3 ||
        P.KS[1] != S::KS2 || P.KS[2] != S::KS3)
        return hipErrorInvalidValue;
    a.blocks_per_agent = (a.envs_per_agent + MB - 1) / MB;
    int nblk = a.n_agents * a.blocks_per_agent;
    nblk = (nblk + 7) & ~7;
    auto k = rollout_rs_kernel<S>;
    hipError_t e = hipFuncSetAttribute((const void *)k,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)off);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k, dim3(nblk), dim3(NWAVES * WAVE), off, st, a);
    return hipGetLastError();
}

}  // namespace rs

// The role-split kernel covers bf16 actors with 100 stocks of 8 indicators
// (1001 inputs: KS1 = 32, the balance/prices/holdings in the first 7
// k-steps) and hidden widths 512 or 1024; returns hipErrorNotSupported for
// other shapes.
bool rollout_rs_shape(const PackedLayout &P, int nI)
{
    return P.dtype == TP_BF16 && P.n == 100 && P.S == 1001 && nI == 800 && P.KS[0] == 32 &&
           P.NT[2] == 8 && ((P.H1 == 512 && P.H2 == 512) || (P.H1 == 1024 && P.H2 == 1024));
}

hipError_t launch_rollout_rs(RolloutArgs &a, hipStream_t s)
{
    const PackedLayout &P = a.lay;
    if (!rollout_rs_shape(P, a.env.nI)) return hipErrorNotSupported;
    // the env waves move prices, indicators, actions and holdings in
    // 16-byte accesses
    if ((uintptr_t)a.env.price % 16 || (uintptr_t)a.env.ind % 16 || (uintptr_t)a.action % 16 ||
        (uintptr_t)a.shares_tap % 16 || (uintptr_t)a.mu_tap % 16)
        return hipErrorNotSupported;
    if (P.H1 == 512 && P.H2 == 512) return rs::launch<rs::Shape<100, 800, 32, 7, 32, 32, 8, 16>>(a, s);
    if (P.H1 == 1024 && P.H2 == 1024) return rs::launch<rs::Shape<100, 800, 32, 7, 64, 64, 8, 16>>(a, s);
    return hipErrorNotSupported;
}

}  // namespace tpk
