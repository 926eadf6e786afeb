// Critic (value network) forward over a time-major block of observations:
// V(x) = w3 . tanh(W2 tanh(W1 x + b1) + b2) + b3 for every row (t, e).
//
// A workgroup owns a block of rows of one time step and one agent (envs
// e0 .. e0 + BM - 1 of that agent), so the weights it streams serve BM rows.
//
// MFMA kernel (bf16, hidden widths 512 or 1024, observation rows of 1024
// columns).  Eight waves, two per SIMD; wave w owns output tiles
// w*OT .. w*OT+OT-1 of both hidden layers (OT = H / 128) for all
// BM = 512 / OT rows, a 4x8 or 8x4 register block of 16x16 fp32
// accumulators (128 registers).  The MFMA is
// v_mfma_f32_16x16x32_bf16 with A = a packed weight fragment (16 outputs x
// 32 inputs, streamed from L2 two k-steps ahead) and B = 32 inputs x 16 rows
// from LDS.  Layer 1 stages the observation block through LDS in chunks of
// 128 columns (double-buffered; the next chunk's global loads are in flight
// while the current one is multiplied); h1 then replaces the staging
// buffers in LDS.  Layer 2's tanh outputs are rounded to bf16 and reduced
// with w3 straight from the accumulators: per lane, across the four lane
// groups of a tile, then across the eight waves in LDS, always in the same
// order, so the result is deterministic.
//
// Generic kernel (fp32, or bf16 shapes the MFMA kernel does not take):
// 16 rows per workgroup, one thread per output unit, weights transposed so
// consecutive threads read consecutive addresses.
#include "device.hpp"
#include "internal.hpp"

// MFMA kernel configuration: waves per workgroup and 16x16 accumulator
// tiles per wave (each 4 registers).
#ifndef CRITIC_NW
#define CRITIC_NW 8
#endif
#ifndef CRITIC_ACC_TILES
#define CRITIC_ACC_TILES 32
#endif
#ifndef CRITIC_MIN_WAVES
#define CRITIC_MIN_WAVES 2
#endif


namespace tpk {

namespace {

typedef uint32_t u4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8 as_bf16x8(u4v v) { return __builtin_bit_cast(bf16x8, v); }

// row block of workgroup b: (time step, agent, first env, rows)
struct RowBlock {
    int64_t t;
    int agent, e0, nrow;
};

__device__ __forceinline__ RowBlock row_block(const CriticArgs &A, int BM)
{
    const int bpa = (A.envs_per_agent + BM - 1) / BM;
    int64_t b = blockIdx.x;
    const int eb = (int)(b % bpa);
    b /= bpa;
    RowBlock r;
    r.agent = (int)(b % A.n_agents);
    r.t = b / A.n_agents;
    r.e0 = r.agent * A.envs_per_agent + eb * BM;
    r.nrow = min(BM, A.envs_per_agent - eb * BM);
    return r;
}

// NW waves, each OT output tiles x RT row tiles of accumulators; KS1
// k-steps of 32 inputs in layer 1 (a multiple of 4).
template <int NW, int OT, int RT, int KS1>
__global__ __launch_bounds__(NW *WAVE, CRITIC_MIN_WAVES) void critic_mfma_kernel(CriticArgs A)
{
    constexpr int NTH = NW * WAVE;
    constexpr int H = 16 * NW * OT;    // hidden width (both layers)
    constexpr int BM = 16 * RT;        // rows per workgroup
    constexpr int KC = 128;            // columns per staged chunk (4 k-steps)
    constexpr int NCH = KS1 / 4;
    constexpr int LDX = KC + 8;        // staged row pitch (conflict-free reads)
    constexpr int LDH = H + 8;
    constexpr int KS2 = H / 32;
    constexpr int SPT = BM * (KC / 8) / NTH;   // 16-byte staging loads per thread
    static_assert(KS1 % 4 == 0 && KS2 % 2 == 0 && SPT >= 1, "shape");
    extern __shared__ __align__(16) uint8_t smem[];
    __bf16 *Xs = (__bf16 *)smem;       // [2][BM][LDX]
    __bf16 *H1s = (__bf16 *)smem;      // [BM][LDH] (after layer 1)
    constexpr size_t XBYTES = 2 * BM * LDX * 2, HBYTES = (size_t)BM * LDH * 2;
    float *vred = (float *)(smem + (XBYTES > HBYTES ? XBYTES : HBYTES));   // [NW][BM]

    const CriticLayout &P = A.lay;
    const int tid = threadIdx.x, lane = tid % WAVE;
    const int w = __builtin_amdgcn_readfirstlane(tid / WAVE);
    const int r16 = lane & 15, kq = lane >> 4;
    const RowBlock rb = row_block(A, BM);
    const uint8_t *pk = A.packed + (size_t)rb.agent * P.agent_stride;
    const __bf16 *rows = (const __bf16 *)A.obs + ((size_t)rb.t * A.E + rb.e0) * A.ld_obs;

    // weight fragments, two k-steps ahead in a ring of two slots
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        (void *)pk, (short)0, (int)P.agent_stride, 0x00020000);
    const int voff = lane * 16;
    const int base1 = (int)P.off_W[0] + w * OT * KS1 * 1024;
    const int base2 = (int)P.off_W[1] + w * OT * KS2 * 1024;
    bf16x8 wr[2][OT];
    auto fetch1 = [&](int slot, int k) {
#pragma unroll
        for (int ot = 0; ot < OT; ++ot)
            wr[slot][ot] = as_bf16x8(__builtin_amdgcn_raw_buffer_load_b128(
                rsrc, voff, base1 + (ot * KS1 + k) * 1024, 0));
    };
    auto fetch2 = [&](int slot, int k) {
#pragma unroll
        for (int ot = 0; ot < OT; ++ot)
            wr[slot][ot] = as_bf16x8(__builtin_amdgcn_raw_buffer_load_b128(
                rsrc, voff, base2 + (ot * KS2 + k) * 1024, 0));
    };

    // observation staging: thread tid moves the 16-byte pieces tid + NTH i
    // of a 128-column chunk (row idx / 16, piece idx % 16); rows past the
    // block's last read its last row (never stored)
    const __bf16 *src[SPT];
#pragma unroll
    for (int i = 0; i < SPT; ++i) {
        const int idx = tid + NTH * i, row = min(idx >> 4, rb.nrow - 1), part = idx & 15;
        src[i] = rows + (size_t)row * A.ld_obs + part * 8;
    }
    u4v st[SPT];
    auto load_chunk = [&](int c) {
#pragma unroll
        for (int i = 0; i < SPT; ++i)
            st[i] = __builtin_nontemporal_load((const u4v *)(src[i] + c * KC));
    };
    auto store_chunk = [&](int buf) {
#pragma unroll
        for (int i = 0; i < SPT; ++i) {
            const int idx = tid + NTH * i, row = idx >> 4, part = idx & 15;
            *(u4v *)(Xs + (size_t)buf * BM * LDX + row * LDX + part * 8) = st[i];
        }
    };

    fetch1(0, 0);
    fetch1(1, 1);
    load_chunk(0);
    store_chunk(0);
    __syncthreads();

    // ---- layer 1 ----------------------------------------------------------
    floatx4 acc[OT][RT];
    // one k-step: B fragments row tile by row tile (the next one read
    // while the current one is multiplied), each against the OT weights
    auto mma_kstep = [&](const __bf16 *xk, int ld, int slot) {
        bf16x8 x = *(const bf16x8 *)xk;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            bf16x8 xn;
            if (rt + 1 < RT) xn = *(const bf16x8 *)(xk + (rt + 1) * 16 * ld);
#pragma unroll
            for (int ot = 0; ot < OT; ++ot)
                acc[ot][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wr[slot][ot], x, acc[ot][rt],
                                                                      0, 0, 0);
            if (rt + 1 < RT) x = xn;
        }
    };
#pragma unroll
    for (int ot = 0; ot < OT; ++ot)
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) acc[ot][rt] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c < NCH; ++c) {
        const bool more = c + 1 < NCH;
        if (more) load_chunk(c + 1);
        const __bf16 *xb = Xs + (size_t)(c & 1) * BM * LDX + r16 * LDX + kq * 8;
        mma_kstep(xb, LDX, 0);
        fetch1(0, c * 4 + 2);
        mma_kstep(xb + 32, LDX, 1);
        fetch1(1, c * 4 + 3);
        mma_kstep(xb + 64, LDX, 0);
        if (more) fetch1(0, c * 4 + 4);
        else fetch2(0, 0);
        mma_kstep(xb + 96, LDX, 1);
        if (more) fetch1(1, c * 4 + 5);
        else fetch2(1, 1);
        if (more) store_chunk((c + 1) & 1);
        __syncthreads();
    }

    // h1 = tanh(acc + b1) in bf16, over the staging buffers
    {
        const float *b1 = (const float *)(pk + P.off_b[0]);
#pragma unroll
        for (int ot = 0; ot < OT; ++ot) {
            const int o = (w * OT + ot) * 16 + kq * 4;
            const floatx4 bv = *(const floatx4 *)(b1 + o);
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                const bf16x4 h = {to_bf16(tanh_from_e2(NEG_2LOG2E * (acc[ot][rt][0] + bv[0]))),
                                  to_bf16(tanh_from_e2(NEG_2LOG2E * (acc[ot][rt][1] + bv[1]))),
                                  to_bf16(tanh_from_e2(NEG_2LOG2E * (acc[ot][rt][2] + bv[2]))),
                                  to_bf16(tanh_from_e2(NEG_2LOG2E * (acc[ot][rt][3] + bv[3])))};
                *(bf16x4 *)(H1s + (rt * 16 + r16) * LDH + o) = h;
            }
        }
    }
    __syncthreads();

    // ---- layer 2 (k-steps continue the fragment stream at KS1) -------------
#pragma unroll
    for (int ot = 0; ot < OT; ++ot)
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) acc[ot][rt] = floatx4{0.f, 0.f, 0.f, 0.f};
    {
        // layer-2 k-step ks sits in ring slot ks & 1
        const __bf16 *hb = H1s + r16 * LDH + kq * 8;
        for (int ks = 0; ks < KS2; ks += 2) {
            const bool more = ks + 2 < KS2;
            mma_kstep(hb + ks * 32, LDH, 0);
            if (more) fetch2(0, ks + 2);
            mma_kstep(hb + (ks + 1) * 32, LDH, 1);
            if (more) fetch2(1, ks + 3);
        }
    }

    // ---- h2 = bf16(tanh(acc + b2)); V = w3 . h2 + b3 ------------------------
    {
        const float *b2 = (const float *)(pk + P.off_b[1]);
        const float *w3 = (const float *)(pk + P.off_W[2]);
        float part[RT];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) part[rt] = 0.f;
#pragma unroll
        for (int ot = 0; ot < OT; ++ot) {
            const int o = (w * OT + ot) * 16 + kq * 4;
            const floatx4 bv = *(const floatx4 *)(b2 + o);
            const floatx4 wv = *(const floatx4 *)(w3 + o);
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float h = (float)to_bf16(tanh_from_e2(NEG_2LOG2E * (acc[ot][rt][i] + bv[i])));
                    part[rt] = fmaf(wv[i], h, part[rt]);
                }
        }
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            part[rt] += __shfl_xor(part[rt], 16);
            part[rt] += __shfl_xor(part[rt], 32);
        }
        if (kq == 0)
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) vred[w * BM + rt * 16 + r16] = part[rt];
    }
    __syncthreads();
    if (tid < rb.nrow) {
        float v = *(const float *)(pk + P.off_b[2]);
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) v += vred[ww * BM + tid];
        A.value[(size_t)rb.t * A.E + rb.e0 + tid] = v;
    }
}

// Generic kernel: 16 rows, 256 threads, fp32 arithmetic on the (bf16-
// rounded, for TP_BF16) transposed weights W1T [K_pad][H1], W2T [H1][H2].
constexpr int GEN_BM = 16;
constexpr int GEN_THREADS = 256;

template <bool BF16>
__global__ __launch_bounds__(GEN_THREADS) void critic_generic_kernel(CriticArgs A)
{
    extern __shared__ __align__(16) uint8_t smem[];
    const CriticLayout &P = A.lay;
    const int S = P.S, K = P.K_pad, H1 = P.H1, H2 = P.H2;
    float *xs = (float *)smem;                 // [GEN_BM][K]
    float *h1 = xs + GEN_BM * K;               // [GEN_BM][H1]
    float *red = h1 + GEN_BM * H1;             // [GEN_THREADS][GEN_BM]
    const int tid = threadIdx.x;
    const RowBlock rb = row_block(A, GEN_BM);
    const uint8_t *pk = A.packed + (size_t)rb.agent * P.agent_stride;
    const float *W1T = (const float *)(pk + P.off_W[0]);
    const float *W2T = (const float *)(pk + P.off_W[1]);
    const float *w3 = (const float *)(pk + P.off_W[2]);
    const float *b1 = (const float *)(pk + P.off_b[0]);
    const float *b2 = (const float *)(pk + P.off_b[1]);

    for (int i = tid; i < GEN_BM * K; i += GEN_THREADS) {
        const int r = i / K, k = i % K;
        float v = 0.f;
        if (r < rb.nrow && k < S) {
            const size_t at = ((size_t)rb.t * A.E + rb.e0 + r) * A.ld_obs + k;
            v = BF16 ? (float)((const __bf16 *)A.obs)[at] : ((const float *)A.obs)[at];
        }
        xs[i] = v;
    }
    __syncthreads();
    for (int o = tid; o < H1; o += GEN_THREADS) {
        float acc[GEN_BM];
#pragma unroll
        for (int r = 0; r < GEN_BM; ++r) acc[r] = 0.f;
        for (int k = 0; k < S; ++k) {
            const float wk = W1T[(size_t)k * H1 + o];
#pragma unroll
            for (int r = 0; r < GEN_BM; ++r) acc[r] = fmaf(wk, xs[r * K + k], acc[r]);
        }
#pragma unroll
        for (int r = 0; r < GEN_BM; ++r) {
            const float h = tanhf(acc[r] + b1[o]);
            h1[r * H1 + o] = BF16 ? (float)to_bf16(h) : h;
        }
    }
    __syncthreads();
    float part[GEN_BM];
#pragma unroll
    for (int r = 0; r < GEN_BM; ++r) part[r] = 0.f;
    for (int o = tid; o < H2; o += GEN_THREADS) {
        float acc[GEN_BM];
#pragma unroll
        for (int r = 0; r < GEN_BM; ++r) acc[r] = 0.f;
        for (int k = 0; k < H1; ++k) {
            const float wk = W2T[(size_t)k * H2 + o];
#pragma unroll
            for (int r = 0; r < GEN_BM; ++r) acc[r] = fmaf(wk, h1[r * H1 + k], acc[r]);
        }
#pragma unroll
        for (int r = 0; r < GEN_BM; ++r) {
            float h = tanhf(acc[r] + b2[o]);
            if (BF16) h = (float)to_bf16(h);
            part[r] = fmaf(w3[o], h, part[r]);
        }
    }
#pragma unroll
    for (int r = 0; r < GEN_BM; ++r) red[tid * GEN_BM + r] = part[r];
    __syncthreads();
    if (tid < rb.nrow) {
        float v = *(const float *)(pk + P.off_b[2]);
        for (int th = 0; th < GEN_THREADS; ++th) v += red[th * GEN_BM + tid];
        A.value[(size_t)rb.t * A.E + rb.e0 + tid] = v;
    }
}

template <class K>
hipError_t launch_with_lds(K k, size_t nblk, int threads, size_t lds, const CriticArgs &a,
                           hipStream_t s)
{
    if (lds > LDS_LIMIT) return hipErrorInvalidConfiguration;
    if (nblk > 0x7fffffffULL) return hipErrorInvalidConfiguration;
    hipError_t e = hipFuncSetAttribute((const void *)k,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k, dim3((unsigned)nblk), dim3(threads), lds, s, a);
    return hipGetLastError();
}

}  // namespace

bool critic_mfma_shape(const CriticLayout &L)
{
    return L.dtype == TP_BF16 && L.H1 == L.H2 && (L.H1 == 512 || L.H1 == 1024) &&
           L.K_pad == 1024;
}

hipError_t launch_critic_value(const CriticArgs &a, hipStream_t s)
{
    const CriticLayout &L = a.lay;
    if (L.mfma) {
        constexpr int NW = CRITIC_NW;
        const int OT = L.H1 / (16 * NW), RT = CRITIC_ACC_TILES / OT, BM = 16 * RT;
        const size_t nblk = (size_t)a.T * a.n_agents * ((a.envs_per_agent + BM - 1) / BM);
        const size_t xb = 2 * (size_t)BM * (128 + 8) * 2, hb = (size_t)BM * (L.H1 + 8) * 2;
        const size_t lds = (xb > hb ? xb : hb) + NW * (size_t)BM * 4;
        constexpr int T512 = 512 / (16 * NW), T1024 = 1024 / (16 * NW);
        if (L.H1 == 512)
            return launch_with_lds(critic_mfma_kernel<NW, T512, CRITIC_ACC_TILES / T512, 32>,
                                   nblk, NW * WAVE, lds, a, s);
        return launch_with_lds(critic_mfma_kernel<NW, T1024, CRITIC_ACC_TILES / T1024, 32>, nblk,
                               NW * WAVE, lds, a, s);
    }
    const size_t nblk = (size_t)a.T * a.n_agents * ((a.envs_per_agent + GEN_BM - 1) / GEN_BM);
    const size_t lds = ((size_t)GEN_BM * (L.K_pad + L.H1) + (size_t)GEN_THREADS * GEN_BM) * 4;
    if (L.dtype == TP_BF16)
        return launch_with_lds(critic_generic_kernel<true>, nblk, GEN_THREADS, lds, a, s);
    return launch_with_lds(critic_generic_kernel<false>, nblk, GEN_THREADS, lds, a, s);
}

}  // namespace tpk
