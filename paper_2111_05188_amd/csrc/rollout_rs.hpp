// Role-split fused rollout kernel for bf16 actors of a 100-stock market
// (4, 8 or 10 indicators per stock: 601, 1001 or 1201 inputs) with two
// hidden layers of the same width, 256, 512, 768 or 1024.  One launch runs
// all L lockstep steps of a block of 16 envs.  The kernel is a template over
// the shape; rollout_rs.hip (8 indicators) and rollout_rs_i4.hip,
// rollout_rs_i10.hip, rollout_rs_i10_wide.hip instantiate it.
//
// Why split roles.  A workgroup owns 16 envs, the N dimension of one MFMA
// tile, so every step streams the actor's weights from L2 into the CU.  That
// stream, not the MFMAs, bounds the actor, and the env step is VALU work
// that would add to it if the two ran one after the other.  Here they
// overlap.  The observation is [balance, prices, holdings, indicators]
// (Section 3, "State space").  Only the balance and the holdings depend on
// the actions; the k-steps of 32 layer-1 inputs that hold neither (the
// market k-steps: prices and indicators only) can be multiplied as soon as
// the market row is known, which is before the env step that completes the
// observation.  Only the other k-steps of layer 1 (the action k-steps),
// layers 2 and 3 remain on the step-to-step chain.
//
// Market k-steps in batches.  The market k-steps of J consecutive steps
// (1 to 3, as the registers and the LDS allow: Pick below) are multiplied
// together, each weight fragment against every step's rows (J MFMAs per
// fragment), so the market part of layer 1 streams once per J steps.  The
// batch's partial sums wait in accumulator registers for their step's
// action k-steps.
//
// Waves.  Four matrix waves (one per SIMD) compute every actor layer; four
// env waves (one per SIMD) own four envs each, one per 16-lane row, eight
// stocks per lane (env_row.hpp).  Each role runs its own loop with the same
// barrier sequence: per step j, four slots separated by workgroup barriers:
//
//   slot  matrix waves                             env waves
//   A     market k-steps of x_j .. x_{j+J-1}       loads of row t0+j+J (in slot B when the
//         (once every J steps)                     step starts a batch); env step j-1:
//                                                  balance and holdings of x_j, trajectory
//                                                  row j-1
//   B     h1 = tanh(Z_j + W1[:, action] x_j + b1)   -
//   L2    h2 = tanh(W2 h1 + b2)                    x_j to HBM; normals of step j
//   L3    mu = W3 h2 + b3                          prices and indicators of row t0+j+J
//                                                  into x_{j+J}
//
// LDS: J observation rows per env (x_j lives in buffer j % J: its market
// columns are written J steps ahead, the balance and holdings by the env
// step that completes it), h1, h2 (bf16), mu (fp32), biases.
//
// Weight stream.  A matrix wave consumes a fixed sequence of weight
// fragments (1 KiB each: one 16x32 A-operand of v_mfma_f32_16x16x32_bf16, 16
// bytes per lane) through a ring of R fragment registers: consuming fragment
// f issues the load of fragment f + R - 1, wrapping into the next period
// (the weights do not change during a rollout), so loads stay in flight
// across layer ends and barriers, and nothing is read twice.  Fragments come
// through buffer loads with a wave-uniform scalar offset.
#pragma once

#include <type_traits>

#include "device.hpp"
#include "env_row.hpp"
#include "internal.hpp"

namespace tpk {
namespace rs {

constexpr int MW = 4;            // matrix waves
constexpr int VW = 4;            // env waves
constexpr int NWAVES = MW + VW;
constexpr int EPW = WAVE / RL;   // envs per env wave
constexpr int MB = EPW * VW;     // envs per workgroup
constexpr int G = 4;             // output tiles per group in layers 1 and 2
static_assert(MB == 16, "one MFMA tile of envs per workgroup");

template <int I> using ic = std::integral_constant<int, I>;

typedef float f4v __attribute__((ext_vector_type(4)));
typedef int i4v __attribute__((ext_vector_type(4)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

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
// k-steps of 32 inputs in layer 1; NT1, NT2, NT3 output tiles of 16; a ring
// of R weight fragments per matrix wave; market k-steps of J steps (1 to 3)
// multiplied together.
template <int NS_, int NI_, int KS1_, int NT1_, int NT2_, int NT3_, int R_, int J_>
struct Shape {
    static constexpr int NS = NS_, NI = NI_;   // stocks, indicator values per row
    static constexpr int R = R_, J = J_;
    static constexpr int KS1 = KS1_;
    static constexpr int NT1 = NT1_, NT2 = NT2_, NT3 = NT3_;
    static constexpr int KS2 = NT1 / 2, KS3 = NT2 / 2;
    static constexpr int NG1 = NT1 / (MW * G), NG2 = NT2 / (MW * G), NG3 = NT3 / MW;
    static_assert(NT1 % (MW * G) == 0 && NT2 % (MW * G) == 0 && NT3 % MW == 0,
                  "tiles must split evenly over the matrix waves");
    static_assert(J >= 1 && J <= 3, "one to three steps per market pass");

    // k-step s holds the balance (column 0) or a holding (columns NS+1 .. 2NS)
    static constexpr bool is_action(int s) { return s == 0 || (32 * s <= 2 * NS && 32 * s + 31 >= NS + 1); }
    static constexpr int count_action()
    {
        int c = 0;
        for (int s = 0; s < KS1; ++s) c += is_action(s);
        return c;
    }
    static constexpr int KSB = count_action(), KSA = KS1 - KSB;
    // the i-th action / market k-step
    static constexpr int aks(int i)
    {
        for (int s = 0; s < KS1; ++s)
            if (is_action(s) && i-- == 0) return s;
        return -1;
    }
    static constexpr int mks(int i)
    {
        for (int s = 0; s < KS1; ++s)
            if (!is_action(s) && i-- == 0) return s;
        return -1;
    }

    // fragments of one matrix wave, in consumption order: the market
    // k-steps (once per J steps), then per step the action k-steps, layer 2
    // and layer 3
    static constexpr int FM = NG1 * KSA * G, FB = NG1 * KSB * G;
    static constexpr int F2 = NG2 * KS2 * G, F3 = NG3 * KS3;
    static constexpr int FS = FB + F2 + F3;
    static constexpr int F = FM + J * FS;   // one period
    static_assert(F % R == 0, "the ring must map every fragment to a fixed slot");
    static_assert(KSB >= G, "the deferred epilogue needs a k-step per tile");

    // layer of fragment f, and its byte offset from the wave's base in that
    // layer (the wave's first tile; groups are MW * G tiles apart in layers
    // 1 and 2, MW tiles apart in layer 3)
    static constexpr int layer(int f)
    {
        if (f < FM) return 0;
        f = (f - FM) % FS;
        return f < FB ? 0 : (f < FB + F2 ? 1 : 2);
    }
    static constexpr int offset(int f)
    {
        if (f < FM) {
            const int g = f / (KSA * G), r = f % (KSA * G);
            return ((g * MW * G + r % G) * KS1 + mks(r / G)) * 1024;
        }
        f = (f - FM) % FS;
        if (f < FB) {
            const int g = f / (KSB * G), r = f % (KSB * G);
            return ((g * MW * G + r % G) * KS1 + aks(r / G)) * 1024;
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
    __bf16 *X;      // [J][MB][ldx] observation rows (x_j in buffer j % J)
    __bf16 *H1;     // [MB][ldh1]  hidden layer 1
    __bf16 *H2;     // [MB][ldh2]  hidden layer 2
    float *MU;      // [MB][ldmu]  action means
    float *BIAS;    // b1 | b2 | b3
    float *LS;      // log sigma | sigma of the actor, per stock slot (RL * SPR each)
    int ldx, ldh1, ldh2, ldmu;
    // row `sl` of observation buffer b (0 <= b < J)
    __device__ __forceinline__ __bf16 *xrow(int b, int sl) const { return X + (b * MB + sl) * ldx; }
};

// k-step k of a segment at input column 32 * col(k)
struct KPlain {
    static constexpr int col(int k) { return k; }
};
template <class S> struct KAction {
    static constexpr int col(int k) { return S::aks(k); }
};
template <class S> struct KMarket {
    static constexpr int col(int k) { return S::mks(k); }
};

// ---------------------------------------------------------------------------
// Matrix role
// ---------------------------------------------------------------------------
// One matrix wave's weight stream.  Fragment i of the period lives in ring
// slot i % R; consuming fragment i first refills the slot fragment i-1 left
// (its MFMAs have issued), then multiplies, so R-1 loads stay in flight.
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
        // (offsets and columns below are bound to constexpr names: the
        // helpers loop over the k-steps, and left in a runtime expression
        // they are not always folded)
        constexpr int f = I % S::F, slot = I % R, L = S::layer(f), off = S::offset(f);
        const int base = L == 0 ? wb0 : (L == 1 ? wb1 : wb2);
        ring[slot] = as_bf16x8(__builtin_amdgcn_raw_buffer_load_b128(rsrc, voff, base + off, 0));
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

    // One slot's work: NG groups of GT output tiles over KS k-steps (k-step
    // k at input column 32 * KM::col(k) of the rows `xb`, this lane's row and
    // column offset).  init(g, acc) and epi(g, t, acc) set up and store group
    // g.  With DEFER the epilogue of group g runs tile by tile inside the
    // first GT k-steps of group g+1, so the weight stream keeps moving
    // through it.
    template <int FB0, int NG, int KS, class KM, int GT, bool DEFER, class InitF, class EpiF>
    __device__ __forceinline__ void seg(const __bf16 *xb, InitF &&init, EpiF &&epi)
    {
        static_assert(!DEFER || KS >= GT, "deferred epilogue needs a k-step per tile");
        floatx4 acc[GT], prev[GT];
        static_for<0, NG>([&](auto gi) {
            constexpr int g = decltype(gi)::value;
            init(g, acc);
            constexpr int c0 = KM::col(0);
            bf16x8 x = *(const bf16x8 *)(xb + c0 * 32);
            static_for<0, KS>([&](auto ki) {
                constexpr int k = decltype(ki)::value;
                bf16x8 xn;
                if constexpr (k + 1 < KS) {
                    constexpr int c1 = KM::col(k + 1);
                    xn = *(const bf16x8 *)(xb + c1 * 32);
                }
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

    // The market k-steps of layer 1 for the rows of NT consecutive steps
    // (tile i from the rows x0b + i * bstride into Z[i]), no bias: every
    // weight fragment is multiplied against all NT tiles.
    template <int FB0, int NT>
    __device__ __forceinline__ void market(const __bf16 *x0b, int bstride,
                                           floatx4 (&Z)[S::J][S::NG1][G])
    {
        static_for<0, S::NG1>([&](auto gi) {
            constexpr int g = decltype(gi)::value;
#pragma unroll
            for (int i = 0; i < NT; ++i)
#pragma unroll
                for (int t = 0; t < G; ++t) Z[i][g][t] = floatx4{0.f, 0.f, 0.f, 0.f};
            bf16x8 x[NT];
            constexpr int c0 = S::mks(0);
#pragma unroll
            for (int i = 0; i < NT; ++i) x[i] = *(const bf16x8 *)(x0b + i * bstride + c0 * 32);
            static_for<0, S::KSA>([&](auto ki) {
                constexpr int k = decltype(ki)::value;
                bf16x8 xn[NT];
                if constexpr (k + 1 < S::KSA) {
                    constexpr int c1 = S::mks(k + 1);
#pragma unroll
                    for (int i = 0; i < NT; ++i) xn[i] = *(const bf16x8 *)(x0b + i * bstride + c1 * 32);
                }
                static_for<0, G>([&](auto ti) {
                    constexpr int t = decltype(ti)::value;
                    constexpr int f = FB0 + (g * S::KSA + k) * G + t;
                    fetch<f + R - 1>();
#pragma unroll
                    for (int i = 0; i < NT; ++i)
                        Z[i][g][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ring[f % R], x[i], Z[i][g][t], 0, 0, 0);
                });
                if constexpr (k + 1 < S::KSA) {
#pragma unroll
                    for (int i = 0; i < NT; ++i) x[i] = xn[i];
                }
                __builtin_amdgcn_sched_barrier(0);
            });
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

    const __bf16 *xb0 = s.xrow(0, r16) + kq * 8;   // buffer i: xb0 + i * bstride
    const int bstride = MB * s.ldx;
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

    // market partial sums of layer 1 for the J steps of a period
    floatx4 Z[S::J][S::NG1][G];

    // one step's chain from fragment FB0 on: h1 from the action k-steps of
    // the rows `xb` on top of Zs, then layers 2 and 3
    auto chain = [&](auto fb0, const __bf16 *xb, floatx4 (&Zs)[S::NG1][G]) {
        constexpr int F0 = decltype(fb0)::value;
        // slot B: h1 = tanh(Z + W1[:, action] x + b1)
        st.launder();
        st.template seg<F0, S::NG1, S::KSB, KAction<S>, G, true>(
            xb,
            [&](int g, floatx4 *acc) {
#pragma unroll
                for (int t = 0; t < G; ++t) acc[t] = Zs[g][t];
            },
            [&](int g, int t, const floatx4 &a) { tanh_store(a, b1, s.H1 + r16 * s.ldh1, col12(g, t)); });
        __syncthreads();
        // slot L2: h2 = tanh(W2 h1 + b2)
        st.launder();
        st.template seg<F0 + S::FB, S::NG2, S::KS2, KPlain, G, true>(
            h1b, zero,
            [&](int g, int t, const floatx4 &a) { tanh_store(a, b2, s.H2 + r16 * s.ldh2, col12(g, t)); });
        __syncthreads();
        // slot L3: mu = W3 h2 + b3
        st.launder();
        st.template seg<F0 + S::FB + S::F2, S::NG3, S::KS3, KPlain, 1, false>(
            h2b, [&](int, floatx4 *acc) { acc[0] = floatx4{0.f, 0.f, 0.f, 0.f}; },
            [&](int g, int, const floatx4 &a) {
                const int o = col3(g);
                const floatx4 bv = *(const floatx4 *)(b3 + o);
                *(floatx4 *)(s.MU + r16 * s.ldmu + o) =
                    floatx4{a[0] + bv[0], a[1] + bv[1], a[2] + bv[2], a[3] + bv[3]};
            });
        __syncthreads();
    };

    // the first R-1 fragments; the rest is fetched one slot behind use
    static_for<0, S::R - 1>([&](auto i) { st.template fetch<decltype(i)::value>(); });
    __syncthreads();   // observation rows of steps 0 and 1 and the biases are in LDS
    for (int j = 0; j < A.L; j += S::J) {
        // slot A of step j: the market k-steps of steps j .. j+J-1 (their
        // rows are in buffers 0 .. J-1)
        st.launder();
        st.template market<0, S::J>(xb0, bstride, Z);
        __syncthreads();
        static_for<0, S::J>([&](auto ii) {
            constexpr int i = decltype(ii)::value;
            if (i == 0 || j + i < A.L) {
                if constexpr (i > 0) __syncthreads();   // slot A of step j+i: nothing here
                chain(ic<S::FM + i * S::FS>{}, xb0 + i * bstride, Z[i]);
            }
        });
    }
}

// ---------------------------------------------------------------------------
// Env role
// ---------------------------------------------------------------------------
template <class S>
__device__ __forceinline__ void env_role(const RolloutArgs &A, const Lds &s, const uint8_t *pk,
                                         int agent, int ebase, int nenv, int v, int lane)
{
    constexpr int n = S::NS, nI = S::NI, J = S::J;
    static_assert(n % 4 == 0 && n <= RL * SPR && nI % 4 == 0 && nI > 0, "shape");
    constexpr int NPC = n / 4;                         // 16-byte price chunks of a row
    constexpr int NICH = nI / 4;                       // 16-byte indicator chunks of a row
    constexpr int IPL = (NICH + RL - 1) / RL;          // indicator chunks per lane
    // 16-byte chunks of an observation row as stored (K_pad = the inputs
    // rounded up to 32 columns; the k-steps of layer 1 run to a multiple of
    // 128, and the columns past K_pad stay in LDS)
    constexpr int OBS_CHUNKS = (1 + 2 * n + nI + 31) / 32 * 32 / 8;
    const EnvConst &C = A.env;
    const PackedLayout &P = A.lay;
    const int r = lane / RL, sl16 = lane % RL;
    const int sl = EPW * v + r;   // env slot in the workgroup
    const bool mine = sl < nenv;
    const int e = ebase + sl;
    const size_t E = (size_t)A.E;
    const float qnan = __builtin_nanf("");
    // this lane's stocks SPR * sl16 + c: all eight, the first four (the
    // lane holding the row's last four stocks when n % 8 == 4) or none
    const bool has8 = SPR * sl16 + 8 <= n, has4 = SPR * sl16 + 4 <= n;
    // ... which are 16-byte chunks pc0, pc1 of a row (clamped to the row)
    const int pc0 = min(2 * sl16, NPC - 1), pc1 = min(2 * sl16 + 1, NPC - 1);

    // log sigma and sigma per stock slot (0 and 1 past n) go to LDS once;
    // the normals' slot reads them back each step (16 registers the env
    // waves do not hold through the trade)
    if (v == 0) {
        const float *lsd = (const float *)(pk + P.off_ls);
        for (int i = lane; i < RL * SPR; i += WAVE) {
            const float l = i < n ? lsd[i] : 0.f;
            s.LS[i] = l;
            s.LS[RL * SPR + i] = expf(l);
        }
    }

    // state of this row's env, kept in registers for the whole rollout
    RowEnv st;
    st.cash = 0.0;
    st.value = 0.0;
    int64_t t0 = 0;
    bool live = false;
#pragma unroll
    for (int c = 0; c < SPR; ++c) {
        st.h[c] = 0;
        st.pd[c] = 0.0;
    }
    if (mine) {
        t0 = A.t[e];
        live = t0 >= 0 && t0 + A.L <= C.T1 - 1;
        if (A.n_invalid && !live && sl16 == 0) atomicAdd(A.n_invalid, 1);
        st.cash = A.cash[e];
#pragma unroll
        for (int c = 0; c < SPR; ++c) {
            const int i = SPR * sl16 + c;
            st.h[c] = i < n ? A.shares[(size_t)e * n + i] : 0;
        }
    }
    const bool wave_live = __ballot(live) != 0;
    const double half_log2pi_n = 0.5 * (double)n * 1.8378770664093454836;

    // prices of row t, 8 per lane; row 0 for envs not stepped.  Slots of
    // stocks past n repeat the row's last chunk: such a stock holds no
    // shares and its order is zero, so its price never enters a sum (and
    // leaving the loaded values as they are lets the loads stay in flight
    // until first use)
    auto load_prices = [&](int64_t t, float (&p)[SPR]) {
        const float *pr = C.price + (size_t)(live ? t : 0) * n;
        const f4v a = load_stream(pr + 4 * pc0), b = load_stream(pr + 4 * pc1);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            p[c] = a[c];
            p[4 + c] = b[c];
        }
    };
    // indicator chunks sl16 + 16 m of row t (clamped to the row)
    auto load_ind = [&](int64_t t, f4v (&ind)[IPL]) {
        const float *ir = C.ind + (size_t)(live ? t : 0) * nI;
#pragma unroll
        for (int mm = 0; mm < IPL; ++mm) ind[mm] = load_stream(ir + 4 * min(sl16 + RL * mm, NICH - 1));
    };
    // this lane's stock values v[c] as bf16 at columns col0 + SPR * sl16 + c
    // (col0 odd): 2-, 4-, 4-, 4- and 2-byte stores for eight stocks
    auto put_stocks = [&](__bf16 *row, int col0, const float (&v)[SPR]) {
        __bf16 *q = row + col0 + SPR * sl16;
        if (has8) {
            q[0] = to_bf16(v[0]);
            *(bf16x2 *)(q + 1) = bf16x2{to_bf16(v[1]), to_bf16(v[2])};
            *(bf16x2 *)(q + 3) = bf16x2{to_bf16(v[3]), to_bf16(v[4])};
            *(bf16x2 *)(q + 5) = bf16x2{to_bf16(v[5]), to_bf16(v[6])};
            q[7] = to_bf16(v[7]);
        } else if (has4) {
            q[0] = to_bf16(v[0]);
            *(bf16x2 *)(q + 1) = bf16x2{to_bf16(v[1]), to_bf16(v[2])};
            q[3] = to_bf16(v[3]);
        }
    };
    // the market columns of an observation row (prices 1 .. n, indicators
    // 2n+1 .. 2n+nI) in bf16; the balance, the holdings and the zero padding
    // are left alone.  Indicators go in aligned 8-byte stores of columns
    // 2n + 4w .. +3 = [indicator 4w-1, indicators 4w .. 4w+2] (chunk w of the
    // row; value 4w-1 is the last of chunk w-1, held by the previous lane of
    // the row, or by lane 15 one round earlier); chunk 0 skips column 2n
    // (the last holding) and the last indicator is one 2-byte store.  All
    // lanes call it (it moves values between lanes); only live rows store.
    auto write_market = [&](__bf16 *row, const float (&p)[SPR], const f4v (&ind)[IPL]) {
        float last = 0.f;   // element 3 of this lane's previous chunk
#pragma unroll
        for (int mm = 0; mm < IPL; ++mm) {
            const f4v vv = ind[mm];
            const float src = sl16 == RL - 1 ? last : vv[3];
            const float prev = dpp32f<DPP_ROW_ROR1>(src);
            last = vv[3];
            const int w = sl16 + RL * mm;
            if (live && w < NICH) {
                __bf16 *q = row + 2 * n + 4 * w;
                if (w > 0) {
                    *(bf16x4 *)q = bf16x4{to_bf16(prev), to_bf16(vv[0]), to_bf16(vv[1]), to_bf16(vv[2])};
                } else {
                    q[1] = to_bf16(vv[0]);
                    *(bf16x2 *)(q + 2) = bf16x2{to_bf16(vv[1]), to_bf16(vv[2])};
                }
                if (w == NICH - 1) q[4] = to_bf16(vv[3]);
            }
        }
        float ps[SPR];
#pragma unroll
        for (int c = 0; c < SPR; ++c) ps[c] = p[c] * C.price_scale;
        if (live) put_stocks(row, 1, ps);
    };
    // the balance and the holdings of an observation row
    auto write_state = [&](__bf16 *row) {
        float hs[SPR];
#pragma unroll
        for (int c = 0; c < SPR; ++c) hs[c] = (float)st.h[c] * C.share_scale;
        if (!live) return;
        if (sl16 == 0) row[0] = to_bf16((float)(st.cash * (double)C.cash_scale));
        put_stocks(row, 1 + n, hs);
    };
    auto xr = [&](int b) { return s.xrow(b, sl); };

    // Prices the coming env steps need: at the start of step j, pj[i]
    // holds row t0 + j + i (pj[0]: the next row of env step j-1).  Rows are
    // loaded J steps ahead, with the market columns of x_{j+J}.
    float pj[J][SPR];
    f4v ind[IPL];
    {
        // observation rows of steps 0 (complete) and 1 .. J-1 (market
        // columns); the total asset at the start row
        load_prices(t0, pj[0]);
        load_ind(t0, ind);
        write_market(xr(0), pj[0], ind);
        write_state(xr(0));
        double hv = 0.0;
#pragma unroll
        for (int c = 0; c < SPR; ++c) {
            st.pd[c] = (double)pj[0][c];
            hv = fma((double)st.h[c], st.pd[c], hv);
        }
        st.value = st.cash + row_sum(hv);
#pragma unroll
        for (int m = 1; m < J; ++m) {
            if (m <= A.L) {
                load_prices(t0 + m, pj[m]);
                load_ind(t0 + m, ind);
                write_market(xr(m), pj[m], ind);
            }
        }
    }

    float sz[SPR];
    double lp = 0.0;
#pragma unroll
    for (int c = 0; c < SPR; ++c) sz[c] = 0.f;

    // env step of step jj (pn: the prices of row t0 + jj + 1): action and
    // mean rows, the trade, the balance and holdings of x_{jj+1}, the rest
    // of trajectory row jj
    auto step_env = [&](int jj, const float (&pn)[SPR]) {
        const size_t row = (size_t)jj * E + e;
        float ain[SPR];
        {
            const float *mu = s.MU + sl * s.ldmu + SPR * sl16;
            const f4v m0 = *(const f4v *)mu, m1 = *(const f4v *)(mu + 4);
            float a[SPR];
#pragma unroll
            for (int c = 0; c < SPR; ++c) {
                a[c] = (c < 4 ? m0[c] : m1[c - 4]) + sz[c];
                ain[c] = (live && SPR * sl16 + c < n) ? a[c] : 0.f;
            }
            // this lane's stocks are 16-byte chunks pc0, pc1 of the rows
            if (mine && has4) {
                const f4v nanv = {qnan, qnan, qnan, qnan};
                f4v *arow = (f4v *)(A.action + row * n);
                store_stream(live ? f4v{a[0], a[1], a[2], a[3]} : nanv, arow + pc0);
                if (has8) store_stream(live ? f4v{a[4], a[5], a[6], a[7]} : nanv, arow + pc1);
                if (A.mu_tap) {
                    f4v *mrow = (f4v *)(A.mu_tap + row * n);
                    store_stream(live ? m0 : nanv, mrow + pc0);
                    if (has8) store_stream(live ? m1 : nanv, mrow + pc1);
                }
            }
        }
        double qd[SPR];
#pragma unroll
        for (int c = 0; c < SPR; ++c) qd[c] = (double)pn[c];
        float rw = 0.f;
        if (wave_live) rw = env_step_row(C, st, ain, qd);
        write_state(xr((jj + 1) % J));
        if (!mine) return;
        const uint8_t done = (uint8_t)(A.step0 + (uint64_t)jj + 1 == (uint64_t)C.horizon);
        if (A.shares_tap && has4) {
            i4v *srow = (i4v *)(A.shares_tap + row * n);
            store_stream(i4v{st.h[0], st.h[1], st.h[2], st.h[3]}, srow + pc0);
            if (has8) store_stream(i4v{st.h[4], st.h[5], st.h[6], st.h[7]}, srow + pc1);
        }
        if (sl16 == 0) {
            store_stream(live ? (float)lp : qnan, A.logp + row);
            store_stream(live ? rw : qnan, A.reward + row);
            store_stream(live ? done : (uint8_t)0, A.done + row);
            if (A.cash_tap) store_stream(st.cash, A.cash_tap + row);
            if (A.asset_tap) store_stream(live ? st.value : (double)qnan, A.asset_tap + row);
        }
    };

    __syncthreads();   // observation rows of steps 0 .. J-1 are in LDS
    int bj = 0;        // j % J: the buffer of x_j
    for (int j = 0; j < A.L; ++j) {
        // slot A: the env step of step j-1, which completes x_j (the matrix
        // waves read only the market k-steps meanwhile)
        float pnext[SPR];
#pragma unroll
        for (int c = 0; c < SPR; ++c) pnext[c] = pj[0][c];
#pragma unroll
        for (int i = 0; i + 1 < J; ++i)
#pragma unroll
            for (int c = 0; c < SPR; ++c) pj[i][c] = pj[i + 1][c];
        // Loads of row t0 + j + J (when a step of this rollout needs it;
        // written in slot L3).  These rows miss in L2 and hold their memory
        // requests for a full HBM round trip, which slows a weight stream
        // running beside them: they go out first in slot A, where the
        // matrix waves stream nothing, except in the steps that start a
        // market batch, where they wait for slot B.
        const bool ahead = j + J <= A.L;
        if (ahead && bj != 0) {
            load_prices(t0 + j + J, pj[J - 1]);
            load_ind(t0 + j + J, ind);
        }
        if (j > 0) step_env(j - 1, pnext);
        __syncthreads();

        // slot B: the row loads of a step that starts a market batch
        if (ahead && bj == 0) {
            load_prices(t0 + j + J, pj[J - 1]);
            load_ind(t0 + j + J, ind);
        }
        __syncthreads();

        // slot L2: x_j to HBM; the normals of step j and their log-density
        if (live && A.obs) {
            const u4v *src = (const u4v *)xr(bj);
            u4v *dst = (u4v *)((__bf16 *)A.obs + ((size_t)j * E + e) * A.ld_obs);
            if constexpr (OBS_CHUNKS % RL == 0) {
#pragma unroll
                for (int c = sl16; c < OBS_CHUNKS; c += RL) store_stream(src[c], dst + c);
            } else {
#pragma unroll
                for (int m = 0; m < (OBS_CHUNKS + RL - 1) / RL; ++m)
                    if (sl16 + RL * m < OBS_CHUNKS) store_stream(src[sl16 + RL * m], dst + sl16 + RL * m);
            }
        }
        {
            float z[SPR];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const U4 w = philox4x32_10(U4{(uint32_t)(2 * sl16 + h), (uint32_t)e,
                                              (uint32_t)(A.step0 + (uint64_t)j), (uint32_t)agent},
                                           A.key_lo, A.key_hi);
                box_muller_hw(uniform_open01(w.x), uniform_open01(w.y), z[4 * h], z[4 * h + 1]);
                box_muller_hw(uniform_open01(w.z), uniform_open01(w.w), z[4 * h + 2], z[4 * h + 3]);
            }
            const float *lsr = s.LS + SPR * sl16;
            const f4v l0 = *(const f4v *)lsr, l1 = *(const f4v *)(lsr + 4);
            const f4v g0 = *(const f4v *)(lsr + RL * SPR), g1 = *(const f4v *)(lsr + RL * SPR + 4);
            double l = 0.0;
#pragma unroll
            for (int c = 0; c < SPR; ++c) {
                const float lsc = c < 4 ? l0[c] : l1[c - 4], sgc = c < 4 ? g0[c] : g1[c - 4];
                sz[c] = sgc * z[c];
                if (SPR * sl16 + c < n) l += -0.5 * (double)z[c] * (double)z[c] - (double)lsc;
            }
            lp = row_sum(l) - half_log2pi_n;
        }
        __syncthreads();

        // slot L3: market columns of x_{j+J} into buffer j % J (x_j has left
        // it: its action k-steps were read in slot B, its copy went out in
        // slot L2)
        if (ahead) write_market(xr(bj), pj[J - 1], ind);
        __syncthreads();
        bj = bj + 1 == J ? 0 : bj + 1;
    }
    step_env(A.L - 1, pj[0]);

    if (mine && live) {
        if (A.obs_last) {
            const u4v *src = (const u4v *)xr(A.L % J);
            u4v *dst = (u4v *)((__bf16 *)A.obs_last + (size_t)e * A.ld_obs);
            if constexpr (OBS_CHUNKS % RL == 0) {
#pragma unroll
                for (int c = sl16; c < OBS_CHUNKS; c += RL) dst[c] = src[c];
            } else {
#pragma unroll
                for (int m = 0; m < (OBS_CHUNKS + RL - 1) / RL; ++m)
                    if (sl16 + RL * m < OBS_CHUNKS) dst[sl16 + RL * m] = src[sl16 + RL * m];
            }
        }
        if (sl16 == 0) {
            A.cash[e] = st.cash;
            A.t[e] = t0 + A.L;
        }
#pragma unroll
        for (int c = 0; c < SPR; ++c) {
            const int i = SPR * sl16 + c;
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
    s.H2 = (__bf16 *)(smem + A.lds_Z);
    s.MU = (float *)(smem + A.lds_MU);
    s.BIAS = (float *)(smem + A.lds_B);
    s.LS = s.BIAS + (S::NT1 + S::NT2 + S::NT3) * 16;
    s.ldx = A.ldx;
    s.ldh1 = A.ldh;
    s.ldh2 = A.ldh2;
    s.ldmu = A.ldmu;

    // zero the observation buffers (padding columns and rows of absent
    // envs stay zero)
    for (int i = threadIdx.x; i < S::J * MB * s.ldx * 2 / 16; i += NWAVES * WAVE)
        ((uint4 *)s.X)[i] = uint4{0, 0, 0, 0};
    __syncthreads();

    if (wave < MW)
        matrix_role<S>(A, s, pk, wave, lane);
    else
        env_role<S>(A, s, pk, agent, ebase, nenv, wave - MW, lane);
}

template <class S>
hipError_t launch(RolloutArgs &a, hipStream_t st)
{
    const PackedLayout &P = a.lay;
    a.ldx = S::KS1 * 32 + 8;
    a.ldh = S::NT1 * 16 + 8;
    a.ldh2 = S::NT2 * 16 + 8;
    a.ldmu = S::NT3 * 16 + 4;
    a.ldz = 0;
    auto al = [](size_t x) { return (x + 15) & ~(size_t)15; };
    size_t off = 0;
    a.lds_X = off;  off = al(off + (size_t)S::J * MB * a.ldx * 2);
    a.lds_H = off;  off = al(off + (size_t)MB * a.ldh * 2);
    a.lds_Z = off;  off = al(off + (size_t)MB * a.ldh2 * 2);
    a.lds_MU = off; off = al(off + (size_t)MB * a.ldmu * 4);
    a.lds_B = off;  off = al(off + ((size_t)(S::NT1 + S::NT2 + S::NT3) * 16 + 2 * RL * SPR) * 4);
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

// The launch configuration of a market of NS stocks with NI indicator
// values per row and an actor with two hidden layers of width H:
//  - J, the market batch: the largest of 3, 2, 1 whose J observation rows
//    per env fit the LDS with h1, h2, mu, the biases and log sigma,
//    whose partial sums (J * NT1 accumulator registers per matrix wave)
//    leave room for a ring of at least 16 fragments in 192 registers, and
//    whose price rows (8 J registers) fit beside the indicator chunks
//    (4 IPL) in the env waves' budget of 92;
//  - R, the ring depth: the largest in 16 .. 24 that divides the period of
//    fragments (every fragment then has a fixed ring slot).
template <int NS, int NI, int H>
struct Pick {
    static constexpr int S = 1 + 2 * NS + NI;
    static constexpr int KS1 = (S + 127) / 128 * 4;
    static constexpr int NT = H / 16, NT3 = ((NS + 15) / 16 + 3) / 4 * 4;
    static constexpr int IPL = (NI / 4 + RL - 1) / RL;
    static constexpr size_t lds(int J)
    {
        auto al = [](size_t x) { return (x + 15) & ~(size_t)15; };
        return al((size_t)J * MB * (KS1 * 32 + 8) * 2) + 2 * al((size_t)MB * (NT * 16 + 8) * 2) +
               al((size_t)MB * (NT3 * 16 + 4) * 4) + al(((size_t)(2 * NT + NT3) * 16 + 2 * RL * SPR) * 4);
    }
    template <int J>
    static constexpr int ring()
    {
        constexpr int F = Shape<NS, NI, KS1, NT, NT, NT3, 1, J>::F;
        const int cap = (192 - J * NT) / 4;
        for (int R = cap < 24 ? cap : 24; R >= 16; --R)
            if (F % R == 0) return R;
        return 0;
    }
    template <int J>
    static constexpr bool fits()
    {
        return lds(J) <= LDS_LIMIT && J * NT <= 128 && 4 * IPL + 8 * J <= 92 && ring<J>() > 0;
    }
    static constexpr int J = fits<3>() ? 3 : (fits<2>() ? 2 : (fits<1>() ? 1 : 0));
    static_assert(J > 0, "no launch configuration fits this shape");
    static constexpr int R = J == 3 ? ring<3>() : (J == 2 ? ring<2>() : ring<1>());
    using type = Shape<NS, NI, KS1, NT, NT, NT3, R, J>;
};

// The role-split rollout of the 100-stock market with NI indicator values
// per row and hidden width H (a translation unit may instantiate some
// widths and declare the rest extern, to split the compile).
template <int NI, int H>
hipError_t launch_shape(RolloutArgs &a, hipStream_t s)
{
    return launch<typename Pick<100, NI, H>::type>(a, s);
}

// ... by hidden width; hipErrorNotSupported for other widths.
template <int NI>
hipError_t launch_market(RolloutArgs &a, hipStream_t s)
{
    switch (a.lay.H1) {
    case 256: return launch_shape<NI, 256>(a, s);
    case 512: return launch_shape<NI, 512>(a, s);
    case 768: return launch_shape<NI, 768>(a, s);
    case 1024: return launch_shape<NI, 1024>(a, s);
    }
    return hipErrorNotSupported;
}

}  // namespace rs
}  // namespace tpk
