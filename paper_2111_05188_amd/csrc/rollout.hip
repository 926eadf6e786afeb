// Fused rollout kernel: L lockstep steps of a block of envs in one launch.
//
// A workgroup owns MB envs of one agent for the whole rollout (envs are
// independent, so workgroups never synchronise with each other).  Per step:
//   layer 1..3 of the actor on the block's observations (bf16 MFMA or fp32
//   VALU), Philox + Box-Muller sampling, the env step, the next observation.
// Observations, hidden activations and the action means stay in LDS; the
// only HBM traffic is the market row of the next bar, the weights (served
// from L2 after the first block reads them), the trajectory writes and the
// state at entry/exit.
//
// Every wave owns EPW envs for the per-env work and computes a share of the
// output tiles of every actor layer.  Within a step the waves' global memory
// traffic is phased: the actor layers stream weights only; the per-env phase
// loads the next market row at its start (the weight stream is over, so its
// latency hides behind the sampling and trade logic) and stores the
// trajectory rows at its end (their acknowledgements overlap the barrier and
// the next layer's first weight loads).
#include "device.hpp"
#include "env.hpp"
#include "internal.hpp"

namespace tpk {

// ---------------------------------------------------------------------------
// Actor layers
// ---------------------------------------------------------------------------

// bf16 MFMA layer: Y[env][o] = act(sum_k W[o][k] X[env][k] + b[o]).
// A operand = packed weight fragment (16 outputs x 32 k), B operand = the
// observations (32 k x 16 envs) read from LDS; the 16x16 fp32 result gives
// each lane 4 consecutive outputs of one env.  Wave w computes tile groups
// g = w, w + nwaves, ... of G tiles each (NT % G == 0).  Weight fragments are
// software-pipelined D k-steps ahead in a register ring (KS % D == 0), so a
// wave keeps D*G KiB of weight loads in flight while its MFMAs run.
constexpr int PIPE = 4;

template <int MT, int G, bool HIDDEN, int KSC>
__device__ __forceinline__ void mfma_layer(const bf16x8 *__restrict__ W,
                                           const float *__restrict__ bias,
                                           int NT, int KSr, const __bf16 *Xs,
                                           int ldx, void *Y, int ldy, int wave,
                                           int nwaves, int lane)
{
    constexpr int D = PIPE;
    // KSC > 0: k-steps known at compile time, the k loop unrolls completely
    // and every wait for a weight fragment is exact
    const int KS = KSC > 0 ? KSC : KSr;
    const int r16 = lane & 15, kq = lane >> 4;
    for (int g0 = wave * G; g0 < NT; g0 += nwaves * G) {
        floatx4 acc[MT][G];
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
            for (int t = 0; t < G; ++t) acc[m][t] = floatx4{0.f, 0.f, 0.f, 0.f};
        const bf16x8 *wt[G];
#pragma unroll
        for (int t = 0; t < G; ++t) wt[t] = W + ((size_t)(g0 + t) * KS) * WAVE + lane;
        const __bf16 *xb = Xs + r16 * ldx + kq * 8;
        bf16x8 buf[D][G];
#pragma unroll
        for (int d = 0; d < D; ++d)
#pragma unroll
            for (int t = 0; t < G; ++t) buf[d][t] = wt[t][d * WAVE];
#pragma unroll
        for (int ks0 = 0; ks0 < (KSC > 0 ? KSC : KS); ks0 += D) {
#pragma unroll
            for (int d = 0; d < D; ++d) {
                const int ks = ks0 + d;
                bf16x8 xf[MT];
#pragma unroll
                for (int m = 0; m < MT; ++m)
                    xf[m] = *(const bf16x8 *)(xb + m * 16 * ldx + ks * 32);
#pragma unroll
                for (int t = 0; t < G; ++t)
#pragma unroll
                    for (int m = 0; m < MT; ++m)
                        acc[m][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(buf[d][t], xf[m], acc[m][t], 0, 0, 0);
                // refill this slot with k-step ks + D.  Past a tile's last
                // k-step this reads the next tile (or the guard the layout
                // leaves after every layer); those values are never used.
#pragma unroll
                for (int t = 0; t < G; ++t) buf[d][t] = wt[t][(size_t)(ks + D) * WAVE];
                // keep the refill here: the scheduler must not sink it next
                // to its use D k-steps later
                __builtin_amdgcn_sched_barrier(0);
            }
        }
#pragma unroll
        for (int t = 0; t < G; ++t) {
            const int o = (g0 + t) * 16 + kq * 4;
            const float4 bv = *(const float4 *)(bias + o);
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                const int env = m * 16 + r16;
                float v0 = acc[m][t][0] + bv.x, v1 = acc[m][t][1] + bv.y;
                float v2 = acc[m][t][2] + bv.z, v3 = acc[m][t][3] + bv.w;
                if (HIDDEN) {
                    bf16x4 h = {to_bf16(tanhf(v0)), to_bf16(tanhf(v1)),
                                to_bf16(tanhf(v2)), to_bf16(tanhf(v3))};
                    *(bf16x4 *)((__bf16 *)Y + env * ldy + o) = h;
                } else {
                    *(float4 *)((float *)Y + env * ldy + o) = float4{v0, v1, v2, v3};
                }
            }
        }
    }
}

// fp32 VALU layer: thread o computes output o for all MB envs; weights are
// k-blocked transposes so consecutive threads read consecutive 16 bytes.
// A layer with at most half as many outputs as threads (the action means)
// gives each output T consecutive lanes (T the largest power of two with
// out * T <= nthr, at most 64) that split its k-blocks and combine by xor
// shuffles in a fixed order: 10% faster on the 30-stock daily shape, where
// 30 threads would otherwise walk 64 k-blocks each.  Deeper unrolling of
// the k loop measured slower.
template <int MB, bool HIDDEN>
__device__ __forceinline__ void valu_layer(const float4 *__restrict__ Wt,
                                           const float *__restrict__ bias,
                                           int K4, int out, const float *Xs,
                                           int ldx, float *Y, int ldy, int tid,
                                           int nthr)
{
    if (out * 2 <= nthr) {
        int T = 1;
        while (T < WAVE && out * T * 2 <= nthr) T *= 2;
        const int span = (out * T + nthr - 1) / nthr * nthr;
        for (int q = tid; q < span; q += nthr) {
            const int o = q / T, sub = q % T;
            const bool live = o < out;
            const int oc = live ? o : out - 1;
            float acc[MB];
#pragma unroll
            for (int m = 0; m < MB; ++m) acc[m] = 0.f;
            for (int k4 = sub; k4 < K4; k4 += T) {
                const float4 w = Wt[(size_t)k4 * out + oc];
#pragma unroll
                for (int m = 0; m < MB; ++m) {
                    const float4 x = *(const float4 *)(Xs + m * ldx + 4 * k4);
                    acc[m] = fmaf(w.x, x.x, acc[m]);
                    acc[m] = fmaf(w.y, x.y, acc[m]);
                    acc[m] = fmaf(w.z, x.z, acc[m]);
                    acc[m] = fmaf(w.w, x.w, acc[m]);
                }
            }
            for (int d = 1; d < T; d *= 2)
#pragma unroll
                for (int m = 0; m < MB; ++m) acc[m] += __shfl_xor(acc[m], d);
            if (live && sub == 0) {
                const float bo = bias[o];
#pragma unroll
                for (int m = 0; m < MB; ++m) {
                    const float v = acc[m] + bo;
                    Y[m * ldy + o] = HIDDEN ? tanhf(v) : v;
                }
            }
        }
        return;
    }
    for (int o = tid; o < out; o += nthr) {
        float acc[MB];
#pragma unroll
        for (int m = 0; m < MB; ++m) acc[m] = 0.f;
#pragma unroll 4
        for (int k4 = 0; k4 < K4; ++k4) {
            const float4 w = Wt[(size_t)k4 * out + o];
#pragma unroll
            for (int m = 0; m < MB; ++m) {
                const float4 x = *(const float4 *)(Xs + m * ldx + 4 * k4);
                acc[m] = fmaf(w.x, x.x, acc[m]);
                acc[m] = fmaf(w.y, x.y, acc[m]);
                acc[m] = fmaf(w.z, x.z, acc[m]);
                acc[m] = fmaf(w.w, x.w, acc[m]);
            }
        }
        const float bo = bias[o];
#pragma unroll
        for (int m = 0; m < MB; ++m) {
            const float v = acc[m] + bo;
            Y[m * ldy + o] = HIDDEN ? tanhf(v) : v;
        }
    }
}

// ---------------------------------------------------------------------------
// The rollout kernel.  OT = observation element type (__bf16 with the MFMA
// actor, float with the VALU actor).
// ---------------------------------------------------------------------------
template <typename OT, int EPW, int NWM, int KS1, int KS2, int KS3>
__global__ __launch_bounds__(NWM *WAVE) void rollout_kernel(RolloutArgs A)
{
    constexpr int MB = EPW * NWM;
    constexpr bool BF16 = sizeof(OT) == 2;
    constexpr int IPL = 32;  // indicators held per lane (n * n_ind <= 1024)
    static_assert(EPW == 1 || EPW == 2, "one env per half wave");
    extern __shared__ __align__(16) uint8_t smem[];

    const EnvConst &C = A.env;
    const PackedLayout &P = A.lay;
    const int n = C.n, nI = C.nI;
    const int tid = threadIdx.x, wave = tid / WAVE, lane = tid % WAVE;

    // XCD-aware block order: consecutive dispatch slots of one XCD (block id
    // mod 8) take consecutive logical blocks, so one agent's blocks share an
    // XCD and its L2.
    const int nb = gridDim.x;
    const int logical = (blockIdx.x % 8) * (nb / 8) + blockIdx.x / 8;
    if (logical >= A.n_agents * A.blocks_per_agent) return;
    const int agent = logical / A.blocks_per_agent;
    const int blk = logical % A.blocks_per_agent;
    const int ebase = agent * A.envs_per_agent + blk * MB;
    const int nenv = min(MB, A.envs_per_agent - blk * MB);

    const uint8_t *pk = A.packed + (size_t)agent * P.agent_stride;
    const float *b1 = (const float *)(pk + P.off_b[0]);
    const float *b2 = (const float *)(pk + P.off_b[1]);
    const float *b3 = (const float *)(pk + P.off_b[2]);
    const float *lsd = (const float *)(pk + P.off_ls);

    OT *X = (OT *)(smem + A.lds_X);              // [MB][ldx] observations (H2 aliases it)
    OT *Hd = (OT *)(smem + A.lds_H);             // [MB][ldh] hidden layer 1
    float *MU = (float *)(smem + A.lds_MU);      // [MB][ldmu] action means
    int32_t *OS = (int32_t *)(smem + A.lds_OS);  // [MB][n] holdings
    float *PT = (float *)(smem + A.lds_PT);      // [MB][n] prices at the current row
    int64_t *T0 = (int64_t *)(smem + A.lds_scal);  // [MB] start rows
    double *OC = (double *)(T0 + MB);            // [MB] balances
    int *ACT = (int *)(OC + MB);                 // [MB] env is stepped

    const int ldx = A.ldx, ldh = A.ldh, ldmu = A.ldmu;
    const size_t E = (size_t)A.E;
    const int obs_chunks = C.K_pad * (int)sizeof(OT) / 16;

    // this lane's half of the wave: env slot `sl` (EPW == 1 leaves the upper
    // half idle), lane `hl` within it, stocks 4 hl .. 4 hl + 3
    const int half = lane / HALF, hl = lane % HALF;
    const int sl = wave * EPW + (half < EPW ? half : 0);
    const bool mine = half < EPW && sl < nenv;

    // copy slot sl's observation row from X to the global row `dst`
    auto store_obs_row = [&](OT *dst) {
        const uint4 *x = (const uint4 *)(X + sl * ldx);
        for (int c = hl; c < obs_chunks; c += HALF) ((uint4 *)dst)[c] = x[c];
    };

    // ---- prologue: state into LDS, obs_0 into X and HBM ----------------------
    for (int i = tid; i < MB * ldx * (int)sizeof(OT) / 16; i += blockDim.x)
        ((uint4 *)X)[i] = uint4{0, 0, 0, 0};
    __syncthreads();
    float ls[SPL], sg[SPL];
#pragma unroll
    for (int c = 0; c < SPL; ++c) {
        const int i = SPL * hl + c;
        ls[c] = i < n ? lsd[i] : 0.f;
        sg[c] = expf(ls[c]);
    }
    bool live = false;   // this half's env is stepped
    if (mine) {
        const int e = ebase + sl;
        const int64_t tt = A.t[e];
        live = tt >= 0 && tt + A.L <= C.T1 - 1;
        if (A.n_invalid && !live && hl == 0) atomicAdd(A.n_invalid, 1);
        // state (also for envs that are not stepped: their taps repeat it)
        for (int i = hl; i < n; i += HALF) OS[sl * n + i] = A.shares[(size_t)e * n + i];
        if (hl == 0) {
            OC[sl] = A.cash[e];
            T0[sl] = tt;
            ACT[sl] = live;
        }
        if (live) {
            const float *prow = C.price + (size_t)tt * n;
            int h[SPL];
            float p[SPL], ind1[1];
#pragma unroll
            for (int c = 0; c < SPL; ++c) {
                const int i = SPL * hl + c;
                h[c] = i < n ? OS[sl * n + i] : 0;
                p[c] = i < n ? prow[i] : 0.f;
                if (i < n) PT[sl * n + i] = p[c];
            }
            const float *irow = C.ind + (size_t)tt * nI;
            ind1[0] = hl < nI ? irow[hl] : 0.f;
            write_obs_half<OT, 1>(X + sl * ldx, C, OC[sl], h, p, ind1, irow, hl);
            if (A.obs) store_obs_row((OT *)A.obs + ((size_t)ebase + sl) * A.ld_obs);
        }
    }
    __syncthreads();

    const double half_log2pi_n = 0.5 * (double)n * 1.8378770664093454836;
    const float qnan = __builtin_nanf("");

    for (int j = 0; j < A.L; ++j) {
        // ---- actor ---------------------------------------------------------
        if constexpr (BF16) {
            constexpr int MT = MB / 16;
            mfma_layer<MT, 4, true, KS1>((const bf16x8 *)(pk + P.off_W[0]), b1, P.NT[0], P.KS[0],
                                         (const __bf16 *)X, ldx, Hd, ldh, wave, NWM, lane);
            __syncthreads();
            mfma_layer<MT, 4, true, KS2>((const bf16x8 *)(pk + P.off_W[1]), b2, P.NT[1], P.KS[1],
                                         (const __bf16 *)Hd, ldh, X, ldx, wave, NWM, lane);
            __syncthreads();
            mfma_layer<MT, 1, false, KS3>((const bf16x8 *)(pk + P.off_W[2]), b3, P.NT[2], P.KS[2],
                                          (const __bf16 *)X, ldx, MU, ldmu, wave, NWM, lane);
        } else {
            valu_layer<MB, true>((const float4 *)(pk + P.off_W[0]), b1, P.KS[0], P.H1,
                                 (const float *)X, ldx, (float *)Hd, ldh, tid, NWM * WAVE);
            __syncthreads();
            valu_layer<MB, true>((const float4 *)(pk + P.off_W[1]), b2, P.KS[1], P.H2,
                                 (const float *)Hd, ldh, (float *)X, ldx, tid, NWM * WAVE);
            __syncthreads();
            valu_layer<MB, false>((const float4 *)(pk + P.off_W[2]), b3, P.KS[2], P.n,
                                  (const float *)X, ldx, MU, ldmu, tid, NWM * WAVE);
        }
        __syncthreads();

        // ---- sampling, env step, trajectory rows, next observation ---------
        // Both envs of the wave are stepped together (one per half).  Order:
        // next-row market loads first, then the compute, then the stores, so
        // that every load is issued before any store (vmcnt counts both, in
        // issue order).
        const uint32_t step = (uint32_t)(A.step0 + (uint64_t)j);
        const uint8_t done = (uint8_t)(A.step0 + (uint64_t)j + 1 == (uint64_t)C.horizon);
        // branch-free loads from valid addresses (clamped index; row 0 for a
        // half without a stepped env), so they issue back to back
        const int64_t t1 = live ? T0[sl] + j + 1 : 0;
        const float *pr = C.price + (size_t)t1 * n;
        const float *ir = nI > 0 ? C.ind + (size_t)t1 * nI : pr;
        const int last = (nI > 0 ? nI : n) - 1;
        float q[SPL], ind[IPL];
#pragma unroll
        for (int c = 0; c < SPL; ++c) q[c] = pr[min(SPL * hl + c, n - 1)];
#pragma unroll
        for (int m = 0; m < IPL; ++m) ind[m] = ir[min(hl + HALF * m, last)];

        // Philox counter (i/4, env, step, agent): lane hl owns stocks 4 hl ..
        // 4 hl + 3 = counter hl, the two Box-Muller pairs of its 4 words
        const int e = ebase + sl;
        const U4 w = philox4x32_10(U4{(uint32_t)hl, (uint32_t)e, step, (uint32_t)agent},
                                   A.key_lo, A.key_hi);
        float z[SPL];
        box_muller(uniform_open01(w.x), uniform_open01(w.y), z[0], z[1]);
        box_muller(uniform_open01(w.z), uniform_open01(w.w), z[2], z[3]);
        const float *mu = MU + sl * ldmu;
        HalfEnv st;
        st.cash = live ? OC[sl] : 0.0;
        float a[SPL];
        double lp = 0.0;
#pragma unroll
        for (int c = 0; c < SPL; ++c) {
            const int i = SPL * hl + c;
            const bool v = live && i < n;
            a[c] = v ? mu[i] + sg[c] * z[c] : 0.f;
            if (v) lp += -0.5 * (double)z[c] * (double)z[c] - (double)ls[c];
            st.h[c] = v ? OS[sl * n + i] : 0;
            st.p[c] = v ? PT[sl * n + i] : 0.f;
            if (!v) q[c] = 0.f;
        }
        const float r = env_step_half(C, st, a, q, live, lane, lp);
        lp -= half_log2pi_n;
        if (live) {
            if (hl == 0) OC[sl] = st.cash;
#pragma unroll
            for (int c = 0; c < SPL; ++c) {
                const int i = SPL * hl + c;
                if (i < n) {
                    OS[sl * n + i] = st.h[c];
                    PT[sl * n + i] = q[c];
                }
            }
            write_obs_half<OT, IPL>(X + sl * ldx, C, st.cash, st.h, q, ind, ir, hl);
        }

        // trajectory row j; observation row j+1 (or the bootstrap one)
        if (mine) {
            const size_t row = (size_t)j * E + e;
            float *ga = A.action + row * n;
            float *gm = A.mu_tap ? A.mu_tap + row * n : nullptr;
            int32_t *gs = A.shares_tap ? A.shares_tap + row * n : nullptr;
            if (!live) {
                // not stepped: NaN rows, done = 0, taps repeat the state
                for (int i = hl; i < n; i += HALF) {
                    ga[i] = qnan;
                    if (gm) gm[i] = qnan;
                    if (gs) gs[i] = OS[sl * n + i];
                }
                if (hl == 0) {
                    A.logp[row] = qnan;
                    A.reward[row] = qnan;
                    A.done[row] = 0;
                    if (A.cash_tap) A.cash_tap[row] = OC[sl];
                    if (A.asset_tap) A.asset_tap[row] = (double)qnan;
                }
            } else {
#pragma unroll
                for (int c = 0; c < SPL; ++c) {
                    const int i = SPL * hl + c;
                    if (i < n) {
                        ga[i] = a[c];
                        if (gm) gm[i] = mu[i];
                        if (gs) gs[i] = st.h[c];
                    }
                }
                if (hl == 0) {
                    A.logp[row] = (float)lp;
                    A.reward[row] = r;
                    A.done[row] = done;
                    if (A.cash_tap) A.cash_tap[row] = st.cash;
                    if (A.asset_tap) A.asset_tap[row] = st.value;
                }
                if (j + 1 < A.L) {
                    if (A.obs) store_obs_row((OT *)A.obs + (row + E) * A.ld_obs);
                } else if (A.obs_last) {
                    store_obs_row((OT *)A.obs_last + (size_t)e * A.ld_obs);
                }
            }
        }
        __syncthreads();
    }

    // ---- epilogue: state back to HBM -----------------------------------------
    if (mine && live) {
        const int e = ebase + sl;
        if (hl == 0) {
            A.cash[e] = OC[sl];
            A.t[e] = T0[sl] + A.L;
        }
        for (int i = hl; i < n; i += HALF) A.shares[(size_t)e * n + i] = OS[sl * n + i];
    }
}

// ---------------------------------------------------------------------------
// Launcher
// ---------------------------------------------------------------------------
static size_t align16(size_t x) { return (x + 15) & ~(size_t)15; }

template <typename OT, int EPW, int NWM, int KS1 = 0, int KS2 = 0, int KS3 = 0>
static hipError_t launch_cfg(RolloutArgs &a, hipStream_t s)
{
    constexpr int MB = EPW * NWM;
    const EnvConst &C = a.env;
    const PackedLayout &P = a.lay;
    const int esz = (int)sizeof(OT);
    if (esz == 2) {
        const int K1 = P.KS[0] * 32;  // layer-1 inputs incl. pipeline padding
        a.ldx = (K1 > P.H2 ? K1 : P.H2) + 8;
        a.ldh = P.H1 + 8;
        a.ldmu = P.NT[2] * 16;
    } else {
        a.ldx = (P.K_pad > P.H2 ? P.K_pad : P.H2) + 4;
        a.ldh = P.H1 + 4;
        a.ldmu = P.n + (4 - P.n % 4) % 4;
    }
    size_t off = 0;
    a.lds_X = off;   off = align16(off + (size_t)MB * a.ldx * esz);
    a.lds_H = off;   off = align16(off + (size_t)MB * a.ldh * esz);
    a.lds_MU = off;  off = align16(off + (size_t)MB * a.ldmu * 4);
    a.lds_OS = off;  off = align16(off + (size_t)MB * C.n * 4);
    a.lds_PT = off;  off = align16(off + (size_t)MB * C.n * 4);
    a.lds_scal = off;
    off = align16(off + (size_t)MB * (8 + 8 + 4));
    a.lds_bytes = off;
    if (off > LDS_LIMIT) return hipErrorInvalidConfiguration;
    a.blocks_per_agent = (a.envs_per_agent + MB - 1) / MB;
    int nblk = a.n_agents * a.blocks_per_agent;
    nblk = (nblk + 7) & ~7;
    auto k = rollout_kernel<OT, EPW, NWM, KS1, KS2, KS3>;
    hipError_t e = hipFuncSetAttribute((const void *)k,
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)off);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k, dim3(nblk), dim3(NWM * WAVE), off, s, a);
    return hipGetLastError();
}

hipError_t launch_rollout(RolloutArgs &a, hipStream_t s)
{
    if (a.n_invalid) {
        const hipError_t e = launch_zero_i32(a.n_invalid, s);
        if (e != hipSuccess) return e;
    }
    if (a.lay.dtype == TP_BF16) {
        const hipError_t e = launch_rollout_rs(a, s);
        if (e != hipErrorNotSupported) return e;
        const int *k = a.lay.KS;
        // fully unrolled variants for the actor shapes in use
        if (k[0] == 32 && k[1] == 16 && k[2] == 16) return launch_cfg<__bf16, 2, 8, 32, 16, 16>(a, s);
        if (k[0] == 32 && k[1] == 32 && k[2] == 32) return launch_cfg<__bf16, 2, 8, 32, 32, 32>(a, s);
        return launch_cfg<__bf16, 2, 8>(a, s);
    }
    return launch_cfg<float, 1, 4>(a, s);
}

}  // namespace tpk
