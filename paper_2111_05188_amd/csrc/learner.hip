// PPO learner update (PPO, Section 5.2; hyper-parameters of Table 2; the
// learner trains the networks on the stored transitions, Section 4.3) for
// one agent's flat fp32 parameter vector, on minibatches of B transitions
// gathered from a time-major trajectory.
//
// Every matrix product of the forward and backward passes is one "NT"
// product C[M][N] = A[M][K] B[N][K]^T with both operands K-contiguous:
//   forward   Z = X W^T                      (A = activations, B = weights)
//   backward  dH = dZ W   = dZ (W^T)^T       (B = a transposed weight copy)
//   weights   dW = dZ^T X = (dZ^T)(X^T)^T    (both transposed activations)
// so the epilogues that produce activations also write their transposes
// (the MFMA result layout gives each lane four consecutive rows of one
// column, one 8-byte store).  Actor and critic take the same minibatch
// rows, so their first layers run as one product over the concatenated
// weights [W1; Wc1]; the other products of a stage are grouped into one
// launch.  bf16 configs use bf16 operands (weights rounded from the fp32
// masters, observations as stored, hidden activations and backpropagated
// pre-activation gradients rounded to bf16) with fp32 MFMA accumulation;
// fp32 configs use an LDS-tiled fp32 kernel.  Bias, log-std and critic-head
// gradients are row sums of the transposed gradient blocks (one wave per
// row, fixed order).  Adam runs over 32x32 tiles of each weight matrix and
// rewrites the operand copies (and their transposes, through LDS) in the
// same pass.
#include <type_traits>

#include "device.hpp"
#include "internal.hpp"

namespace tpk {

namespace {

constexpr float LN_2PI_F = 1.8378770664093453f;

template <bool BF>
using Elem = typename std::conditional<BF, __bf16, float>::type;

template <bool BF>
__device__ __forceinline__ Elem<BF> to_elem(float x)
{
    if constexpr (BF) return to_bf16(x);
    else return x;
}

__device__ __forceinline__ float fast_tanh(float x) { return tanh_from_e2(NEG_2LOG2E * x); }

// ---------------------------------------------------------------------------
// Grouped NT products with fused epilogues
// ---------------------------------------------------------------------------

enum Epi : int {
    EPI_TANH = 0,   // h = tanh(acc + bias[col]) -> out[row][col], outT[col][row] (elem)
    EPI_BIAS = 1,   // out[row][col] = acc + bias[col]                   (fp32)
    EPI_GRAD = 2,   // gradient rows: row < gsplit -> g0, else g1; cols < gcols (fp32)
    EPI_DTANH = 3,  // v = acc (1 - h^2), h = hsrc[col][row] -> out, outT   (elem)
};

struct GemmProb {
    const void *A;
    const void *B;
    int64_t lda, ldb;
    int M, N, K;
    int mode;
    const float *bias0, *bias1;
    int bsplit;
    void *out;
    int64_t ldo;
    void *outT;
    int64_t ldt;
    float *g0, *g1;
    int64_t ldg;
    int gsplit, gcols;
    const void *hsrc;   // EPI_DTANH: the layer's activations, transposed ([col][row], 8-byte reads)
    int64_t ldh;
    int tiles_n, tile0;
};

constexpr int MAX_PROBS = 4;
struct GemmBatch {
    GemmProb p[MAX_PROBS];
    int np;
    int tiles, na;       // tiles per agent, agents
    int64_t aws, aprm;   // bytes between agents: workspace, parameters
};

// The (agent, tile) slot of this workgroup.  With several agents it is
// XCD-aware: workgroups are dealt round-robin over the 8 XCDs; the grid
// holds 8 per of them (per = gridDim.x / 8), and workgroup b takes slot
// (b % 8) per + b / 8, so each XCD walks a contiguous run of slots, whole
// agents whose operands stay in that XCD's L2.  One agent keeps slot b
// (measured faster there).  False for the padding slots past the last.
__device__ __forceinline__ bool gemm_slot(const GemmBatch &gb, int &agent, int &t)
{
    const int b = blockIdx.x, per = gridDim.x / 8;
    const int v = gb.na == 1 ? b : (b % 8) * per + b / 8;
    if (v >= gb.tiles * gb.na) return false;
    // uniform, but a division by a runtime value is computed on the vector
    // unit: move the results to scalar registers
    agent = __builtin_amdgcn_readfirstlane(v / gb.tiles);
    t = __builtin_amdgcn_readfirstlane(v % gb.tiles);
    return true;
}

// p + by bytes (null stays null), computed on the global address space.
// Pointers that reach a kernel inside a struct are generic to the compiler,
// so accesses through them become flat instructions; a flat load counts
// against the LDS counter too, and every wait for an LDS read would then
// also wait for the operand prefetches in flight.  Derived from a global
// pointer, they compile to global loads and stores.
template <class T>
__device__ __forceinline__ T *shifted(T *p, size_t by)
{
    typedef __attribute__((address_space(1))) char gchar;
    return (T *)((gchar *)p + (p ? by : 0));
}

// Problem pi for agent `agent`: the operands, outputs, gradient blocks and
// activation sources live in the agent's workspace, the biases in its
// parameters.
__device__ __forceinline__ GemmProb agent_prob(const GemmBatch &gb, int pi, int agent)
{
    GemmProb P = gb.p[pi];
    const size_t w = (size_t)agent * (size_t)gb.aws, q = (size_t)agent * (size_t)gb.aprm;
    P.A = shifted(P.A, w);
    P.B = shifted(P.B, w);
    P.out = shifted(P.out, w);
    P.outT = shifted(P.outT, w);
    P.g0 = shifted(P.g0, w);
    P.g1 = shifted(P.g1, w);
    P.hsrc = shifted(P.hsrc, w);
    P.bias0 = shifted(P.bias0, q);
    P.bias1 = shifted(P.bias1, q);
    return P;
}

constexpr int GT = 64;   // workgroup tile (rows and columns)

template <bool BF>
__device__ __forceinline__ void epi4(const GemmProb &P, int row0, int col, const float v[4])
{
    if (col >= P.N) return;
    const int mode = P.mode;
    if (mode == EPI_GRAD) {
        if (col >= P.gcols) return;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = row0 + i;
            if (r >= P.M) break;
            float *d = r < P.gsplit ? P.g0 + (size_t)r * P.ldg : P.g1 + (size_t)(r - P.gsplit) * P.ldg;
            d[col] = v[i];
        }
        return;
    }
    if (mode == EPI_BIAS) {
        const float b = col < P.bsplit ? P.bias0[col] : P.bias1[col - P.bsplit];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = row0 + i;
            if (r >= P.M) break;
            ((float *)P.out)[(size_t)r * P.ldo + col] = v[i] + b;
        }
        return;
    }
    Elem<BF> h[4];
    if (mode == EPI_TANH) {
        const float b = col < P.bsplit ? P.bias0[col] : P.bias1[col - P.bsplit];
#pragma unroll
        for (int i = 0; i < 4; ++i) h[i] = to_elem<BF>(fast_tanh(v[i] + b));
    } else {   // EPI_DTANH
        const Elem<BF> *hs = (const Elem<BF> *)P.hsrc;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = min(row0 + i, P.M - 1);
            const float y = (float)hs[(size_t)col * P.ldh + r];
            h[i] = to_elem<BF>(v[i] * (1.0f - y * y));
        }
    }
    if (P.out) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = row0 + i;
            if (r >= P.M) break;
            ((Elem<BF> *)P.out)[(size_t)r * P.ldo + col] = h[i];
        }
    }
    if (P.outT) {
        Elem<BF> *t = (Elem<BF> *)P.outT + (size_t)col * P.ldt + row0;
        if (row0 + 3 < P.M) {
            if constexpr (BF) {
                *(bf16x4 *)t = bf16x4{h[0], h[1], h[2], h[3]};
            } else {
                *(floatx4 *)t = floatx4{h[0], h[1], h[2], h[3]};
            }
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (row0 + i < P.M) t[i] = h[i];
        }
    }
}

__device__ __forceinline__ int find_prob(const GemmBatch &g, int t)
{
    int pi = 0;
#pragma unroll
    for (int q = 1; q < MAX_PROBS; ++q)
        if (q < g.np && t >= g.p[q].tile0) pi = q;
    return pi;
}

// bf16: four waves, each a 32x32 block of the 64x64 tile (2x2 MFMA tiles of
// 16x16, v_mfma_f32_16x16x32_bf16), fragments loaded straight from global
// memory (operands are small and L2-resident) through a ring of GEMM_PF
// k-steps of registers: consuming k-step k issues the loads of k + GEMM_PF,
// so that many k-steps are in flight to cover the L2 latency.
#ifndef GEMM_PF
#define GEMM_PF 8
#endif

template <int I>
using ic = std::integral_constant<int, I>;

template <int B, int E, typename Fn>
__device__ __forceinline__ void static_for(Fn &&fn)
{
    if constexpr (B < E) {
        fn(ic<B>{});
        static_for<B + 1, E>(fn);
    }
}

__device__ __forceinline__ void mma_2x2(const bf16x8 a[2], const bf16x8 b[2], floatx4 acc[2][2])
{
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
}

// NK k-steps fully unrolled: every ring slot is a compile-time register
// set, so each wait is for exactly the k-step about to be used.
template <int NK, int PF>
__device__ __forceinline__ void kloop_fixed(const __bf16 *const pa[2], const __bf16 *const pb[2],
                                            floatx4 acc[2][2])
{
    constexpr int D = NK < PF ? NK : PF;
    bf16x8 ra[D][2], rb[D][2];
    static_for<0, D>([&](auto q) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            ra[q][i] = *(const bf16x8 *)(pa[i] + q * 32);
            rb[q][i] = *(const bf16x8 *)(pb[i] + q * 32);
        }
    });
    // the scheduling barriers keep each refill where it is issued (the
    // scheduler would otherwise sink the loads next to their use and
    // shrink the ring to a step or two)
    __builtin_amdgcn_sched_barrier(0);
    static_for<0, NK>([&](auto k) {
        constexpr int slot = k % D;
        mma_2x2(ra[slot], rb[slot], acc);
        if constexpr (k + D < NK) {
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                ra[slot][i] = *(const bf16x8 *)(pa[i] + (k + D) * 32);
                rb[slot][i] = *(const bf16x8 *)(pb[i] + (k + D) * 32);
            }
        }
        __builtin_amdgcn_sched_barrier(0);
    });
}

// Any k-step count: the same ring under a runtime bound.
template <int PF>
__device__ __forceinline__ void kloop_any(const __bf16 *const pa[2], const __bf16 *const pb[2],
                                          floatx4 acc[2][2], int nk)
{
    bf16x8 ra[PF][2], rb[PF][2];
    static_for<0, PF>([&](auto q) {
        if (q < nk) {
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                ra[q][i] = *(const bf16x8 *)(pa[i] + q * 32);
                rb[q][i] = *(const bf16x8 *)(pb[i] + q * 32);
            }
        }
    });
    for (int kb = 0; kb < nk; kb += PF) {
        static_for<0, PF>([&](auto q) {
            const int k = kb + q;
            if (k < nk) {
                mma_2x2(ra[q], rb[q], acc);
                if (k + PF < nk) {
#pragma unroll
                    for (int i = 0; i < 2; ++i) {
                        ra[q][i] = *(const bf16x8 *)(pa[i] + (k + PF) * 32);
                        rb[q][i] = *(const bf16x8 *)(pb[i] + (k + PF) * 32);
                    }
                }
            }
        });
    }
}
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmBatch gb)
{
    constexpr int PF = GEMM_PF;
    int agent, t;
    if (!gemm_slot(gb, agent, t)) return;
    const int pi = find_prob(gb, t);
    const GemmProb P = agent_prob(gb, pi, agent);
    t -= P.tile0;
    const int tn = __builtin_amdgcn_readfirstlane(t % P.tiles_n);
    const int tm = __builtin_amdgcn_readfirstlane(t / P.tiles_n);
    const int wave = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
    const int m0 = tm * GT + (wave >> 1) * 32, n0 = tn * GT + (wave & 1) * 32;
    const int r16 = lane & 15, kq = lane >> 4;
    const __bf16 *A = (const __bf16 *)P.A, *B = (const __bf16 *)P.B;
    const __bf16 *pa[2], *pb[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        pa[i] = A + (size_t)min(m0 + i * 16 + r16, P.M - 1) * P.lda + kq * 8;
        pb[i] = B + (size_t)min(n0 + i * 16 + r16, P.N - 1) * P.ldb + kq * 8;
    }
    floatx4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    const int nk = P.K / 32;
    switch (nk) {   // the products in use have 4, 16 or 32 k-steps
    case 4: kloop_fixed<4, PF>(pa, pb, acc); break;
    case 16: kloop_fixed<16, PF>(pa, pb, acc); break;
    case 32: kloop_fixed<32, PF>(pa, pb, acc); break;
    default: kloop_any<PF>(pa, pb, acc, nk); break;
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
            epi4<true>(P, m0 + i * 16 + kq * 4, n0 + j * 16 + r16, v);
        }
}

// bf16 through LDS, for products whose K is a multiple of 128 (all of the
// bf16 learner's): chunks of 64 rows x 128 k of A and of B are staged in
// LDS (rows padded by 32 bytes, measured faster than 16 or 48), loaded
// with whole-line accesses (each wave instruction
// reads 4 rows x 256 contiguous bytes), GEMM_LD chunks ahead in registers
// (deeper prefetch measured slower); eight waves (a 2 x 4 grid of 32x16
// blocks: twice the waves of a 2 x 2 grid of 32x32 blocks, for latency
// hiding, at 1.5x the LDS fragment reads) read their fragments from LDS.
#ifndef GEMM_LD
#define GEMM_LD 2                     // chunks in flight in registers
#endif
#ifndef GEMM_LPAD
#define GEMM_LPAD 16                  // LDS row padding (bf16 elements)
#endif
constexpr int LBK = 128;              // k per chunk
constexpr int LROW = LBK + GEMM_LPAD; // padded LDS row (bf16)
constexpr int LTILE = GT * LROW;      // one operand's chunk (bf16)

typedef uint32_t v4u_t __attribute__((ext_vector_type(4)));

constexpr int LWAVES = 8;              // waves per workgroup: 2 (rows) x 4 (columns)
constexpr int LTHREADS = LWAVES * WAVE;

// Epilogues staged through LDS.  In the MFMA layout a lane holds four rows
// of one column, so stores straight from the accumulators give each
// instruction 16 separate 32-byte pieces of bf16 (64-byte pieces of the
// fp32 gradient rows).  Instead the fragments go into a 64 x 64 block in
// LDS (row-major and transposed), and a group of G threads stores whole
// rows of it: 128 contiguous bytes per bf16 row, 256 per fp32 row, 16
// bytes a thread where the output's rows are 16-byte aligned, else one
// element a thread, a row per 64 threads.  Same values as epi4, same bits.
constexpr int ER = 64 + 8;   // LDS row of a staged bf16 block (elements)
constexpr int EF = 64 + 4;   // LDS row of a staged fp32 block (floats)
constexpr int STAGE_BYTES = 2 * 64 * ER * 2;   // one block: T and R (F is smaller)

__device__ __forceinline__ bool rows16(const void *p, int64_t ld, int es)
{
    return (uintptr_t)p % 16 == 0 && (ld * es) % 16 == 0;
}

// Fragment piece (rows lr .. lr + 3, column lc of the block; global row0,
// col) into the staged block: the gradient rows' fp32 values into F, or
// the bf16 activation (EPI_TANH) or its pre-activation gradient
// (EPI_DTANH) into R (row-major) and T (transposed).
__device__ __forceinline__ void stage4(const GemmProb &P, const floatx4 &a, int row0, int col,
                                       int lr, int lc, void *blk)
{
    if (P.mode == EPI_GRAD) {
        float *F = (float *)blk;
#pragma unroll
        for (int e = 0; e < 4; ++e) F[(lr + e) * EF + lc] = a[e];
        return;
    }
    __bf16 *T = (__bf16 *)blk, *R = T + 64 * ER;
    col = min(col, P.N - 1);   // columns past N are staged but never stored
    __bf16 h[4];
    if (P.mode == EPI_TANH) {
        const float b = col < P.bsplit ? P.bias0[col] : P.bias1[col - P.bsplit];
#pragma unroll
        for (int e = 0; e < 4; ++e) h[e] = to_bf16(fast_tanh(a[e] + b));
    } else {
        const __bf16 *hs = (const __bf16 *)P.hsrc + (size_t)col * P.ldh;
        bf16x4 y4;
        if (row0 + 3 < P.M) y4 = *(const bf16x4 *)(hs + row0);
        else
#pragma unroll
            for (int e = 0; e < 4; ++e) y4[e] = hs[min(row0 + e, P.M - 1)];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float y = (float)y4[e];
            h[e] = to_bf16(a[e] * (1.0f - y * y));
        }
    }
    *(bf16x4 *)(T + lc * ER + lr) = bf16x4{h[0], h[1], h[2], h[3]};
#pragma unroll
    for (int e = 0; e < 4; ++e) R[(lr + e) * ER + lc] = h[e];
}

// Threads gt = 0 .. G - 1 store the staged block of rows bm .., columns
// bn .. (after a barrier that covers every write of stage4).
template <int G>
__device__ __forceinline__ void store_staged(const GemmProb &P, const void *blk, int bm, int bn,
                                             int gt)
{
    const int nrow = min(64, P.M - bm);
    if (P.mode == EPI_GRAD) {
        const float *F = (const float *)blk;
        const int ncol = min(64, min(P.N, P.gcols) - bn);
        if (nrow <= 0 || ncol <= 0) return;
        auto dst = [&](int r) {
            const int gr = bm + r;
            return gr < P.gsplit ? P.g0 + (size_t)gr * P.ldg : P.g1 + (size_t)(gr - P.gsplit) * P.ldg;
        };
        if (nrow == 64 && ncol == 64 && rows16(P.g0, P.ldg, 4) &&
            (P.gsplit >= P.M || rows16(P.g1, P.ldg, 4))) {
#pragma unroll
            for (int s = 0; s < 1024 / G; ++s) {
                const int r = (s * G + gt) / 16, c4 = (gt % 16) * 4;
                *(floatx4 *)(dst(r) + bn + c4) = *(const floatx4 *)(F + r * EF + c4);
            }
        } else {
            const int c = gt % 64;
            for (int r = gt / 64; r < nrow; r += G / 64)
                if (c < ncol) dst(r)[bn + c] = F[r * EF + c];
        }
        return;
    }
    const __bf16 *T = (const __bf16 *)blk, *R = T + 64 * ER;
    const int ncol = min(64, P.N - bn);
    if (nrow <= 0 || ncol <= 0) return;
    const bool full = nrow == 64 && ncol == 64;
    // block row (or column) x, 16-byte piece p8 of it
    auto put = [&](__bf16 *o, int64_t ld, const __bf16 *src, int nx, int ny) {
        if (full && rows16(o, ld, 2)) {
#pragma unroll
            for (int s = 0; s < 512 / G; ++s) {
                const int x = (s * G + gt) / 8, p8 = (gt % 8) * 8;
                *(v4u_t *)(o + (size_t)x * ld + p8) = *(const v4u_t *)(src + x * ER + p8);
            }
        } else {
            const int y = gt % 64;
            for (int x = gt / 64; x < nx; x += G / 64)
                if (y < ny) o[(size_t)x * ld + y] = src[x * ER + y];
        }
    };
    if (P.out) put((__bf16 *)P.out + (size_t)bm * P.ldo + bn, P.ldo, R, nrow, ncol);
    if (P.outT) put((__bf16 *)P.outT + (size_t)bn * P.ldt + bm, P.ldt, T, ncol, nrow);
}

// Chunk loop: LTHREADS threads move a 64 x 128 chunk of A and one of B
// (thread t: rows (t / 16) + 32 j, 16-byte piece t % 16); wave (wm, wn)
// multiplies rows 32 wm .. +31 by columns 16 wn .. +15 (two 16x16 tiles).
template <int NC>
__device__ __forceinline__ void lds_kloop(const __bf16 *const ga, const __bf16 *const gb,
                                          int64_t lda, int64_t ldb, int Mr, int Nr,
                                          __bf16 *smem, floatx4 acc[2])
{
    const int tid = threadIdx.x, lane = tid % WAVE, wave = tid / WAVE;
    const int r16 = lane & 15, kq = lane >> 4;
    const int lrow = tid >> 4, lpiece = tid & 15;
    const __bf16 *la[2], *lb[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        la[j] = ga + (size_t)min(lrow + 32 * j, Mr - 1) * lda + lpiece * 8;
        lb[j] = gb + (size_t)min(lrow + 32 * j, Nr - 1) * ldb + lpiece * 8;
    }
    constexpr int D = NC < GEMM_LD ? NC : GEMM_LD;   // chunks in flight in registers
    v4u_t ra[D][2], rb[D][2];
    auto load = [&](v4u_t (&xa)[2], v4u_t (&xb)[2], int c) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            xa[j] = *(const v4u_t *)(la[j] + c * LBK);
            xb[j] = *(const v4u_t *)(lb[j] + c * LBK);
        }
    };
    auto store = [&](const v4u_t (&xa)[2], const v4u_t (&xb)[2], int buf) {
        __bf16 *As = smem + buf * 2 * LTILE, *Bs = As + LTILE;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            *(v4u_t *)(As + (lrow + 32 * j) * LROW + lpiece * 8) = xa[j];
            *(v4u_t *)(Bs + (lrow + 32 * j) * LROW + lpiece * 8) = xb[j];
        }
    };
    static_for<0, D>([&](auto c) { load(ra[c], rb[c], c); });
    store(ra[0], rb[0], 0);
    if constexpr (D < NC) load(ra[0], rb[0], D);
    __syncthreads();
    const int am = (wave >> 2) * 32, bn = (wave & 3) * 16;
    // Per chunk c: read its fragments (all four k-steps); store chunk c + 1
    // into the other LDS buffer (free since the last barrier) and issue the
    // load of chunk c + 1 + D; then the MFMAs; one barrier.
    static_for<0, NC>([&](auto c) {
        constexpr int buf = c & 1;
        const __bf16 *As = smem + buf * 2 * LTILE, *Bs = As + LTILE;
        bf16x8 fa[LBK / 32][2], fb[LBK / 32];
#pragma unroll
        for (int q = 0; q < LBK / 32; ++q) {
#pragma unroll
            for (int i = 0; i < 2; ++i)
                fa[q][i] = *(const bf16x8 *)(As + (am + i * 16 + r16) * LROW + q * 32 + kq * 8);
            fb[q] = *(const bf16x8 *)(Bs + (bn + r16) * LROW + q * 32 + kq * 8);
        }
        if constexpr (c + 1 < NC) {
            // chunk c + 1 sits in register set (c + 1) % D; refill it with c + 1 + D
            constexpr int slot = (c + 1) % D;
            store(ra[slot], rb[slot], (c + 1) & 1);
            if constexpr (c + 1 + D < NC) load(ra[slot], rb[slot], c + 1 + D);
        }
#pragma unroll
        for (int q = 0; q < LBK / 32; ++q) {
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < 2; ++i)
                acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[q][i], fb[q], acc[i], 0, 0, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (c + 1 < NC) __syncthreads();
    });
}

__global__ __launch_bounds__(LTHREADS, 2) void gemm_lds_kernel(GemmBatch gb)
{
    __shared__ __attribute__((aligned(16))) __bf16 smem[2 * 2 * LTILE];
    int agent, t;
    if (!gemm_slot(gb, agent, t)) return;
    const int pi = find_prob(gb, t);
    const GemmProb P = agent_prob(gb, pi, agent);
    t -= P.tile0;
    const int tn = __builtin_amdgcn_readfirstlane(t % P.tiles_n);
    const int tm = __builtin_amdgcn_readfirstlane(t / P.tiles_n);
    const int wave = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
    const int m0 = tm * GT, n0 = tn * GT;
    const int r16 = lane & 15, kq = lane >> 4;
    const __bf16 *ga = (const __bf16 *)P.A + (size_t)m0 * P.lda;
    const __bf16 *gbp = (const __bf16 *)P.B + (size_t)n0 * P.ldb;
    floatx4 acc[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) acc[i] = floatx4{0.f, 0.f, 0.f, 0.f};
    const int Mr = P.M - m0, Nr = P.N - n0;     // rows left in this tile (>= 1)
    switch (P.K / LBK) {
    case 1: lds_kloop<1>(ga, gbp, P.lda, P.ldb, Mr, Nr, smem, acc); break;
    case 4: lds_kloop<4>(ga, gbp, P.lda, P.ldb, Mr, Nr, smem, acc); break;
    case 8: lds_kloop<8>(ga, gbp, P.lda, P.ldb, Mr, Nr, smem, acc); break;
    default: break;   // the launcher routes other K to gemm_bf16_kernel
    }
    const int wm = m0 + (wave >> 2) * 32, wn = n0 + (wave & 3) * 16;
    if (P.mode == EPI_BIAS) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const float v[4] = {acc[i][0], acc[i][1], acc[i][2], acc[i][3]};
            epi4<true>(P, wm + i * 16 + kq * 4, wn + r16, v);
        }
        return;
    }
    static_assert(STAGE_BYTES <= sizeof(smem), "the staged block fits");
    // the eight waves stage the 64 x 64 tile in LDS (free once every wave has
    // passed this barrier) and store it together
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 2; ++i)
        stage4(P, acc[i], wm + i * 16 + kq * 4, wn + r16, wm - m0 + i * 16 + kq * 4, wn - n0 + r16,
               smem);
    __syncthreads();
    store_staged<LTHREADS>(P, smem, m0, n0, threadIdx.x);
}

// Launches with many tiles (several agents): 256 x 128 workgroup tiles of
// eight 64 x 64 waves, k-chunks of 64 staged through LDS, one workgroup per
// CU.  A wave's 4 x 4 tiles of 16 x 16 use each fragment four times, 0.5 KiB
// of LDS reads per MFMA against 1.5 KiB in the eight-wave kernel above,
// whose reads exceed the LDS bandwidth once every CU is busy.  The operand
// loads bound this kernel (timing copies without them run 8% faster per
// update, without the MFMAs no faster): 256 x 128 loads 48 KiB per chunk
// for the work two 128 x 128 workgroups load 64 KiB for (measured 2% faster
// per update).  Rows padded by 32 bytes (measured faster than 16).
constexpr int BT = 128;               // workgroup tile: columns (rows of B)
constexpr int BM = 256;               // workgroup tile: rows (rows of A)
constexpr int BWAVES = 8;             // a 4 x 2 grid of 64 x 64 waves
constexpr int BTHREADS = BWAVES * WAVE;
#ifndef GEMM_BPAD
#define GEMM_BPAD 16                  // LDS row padding (bf16 elements)
#endif
constexpr int BBK = 64;               // k per chunk
constexpr int BROW = BBK + GEMM_BPAD; // padded LDS row (bf16)
constexpr int BBUF = (BM + BT) * BROW;   // one chunk of A and B (bf16)
constexpr int BIG_MIN_TILES = 512;    // launches with fewer 128 x 128 tiles keep 64 x 64

// Chunk loop: 512 threads move a 256 x 64 chunk of A and a 128 x 64 chunk
// of B (thread t: rows (t / 8) + 64 j, 16-byte piece t % 8; a wave
// instruction reads 8 rows x 128 contiguous bytes); wave (wm, wn)
// multiplies rows 64 wm .. +63 by columns 64 wn .. +63.
template <int NC>
__device__ __forceinline__ void big_kloop(const __bf16 *const ga, const __bf16 *const gb,
                                          int64_t lda, int64_t ldb, int Mr, int Nr,
                                          __bf16 *smem, floatx4 (&acc)[4][4])
{
    const int tid = threadIdx.x, lane = tid % WAVE, wave = tid / WAVE;
    const int r16 = lane & 15, kq = lane >> 4;
    constexpr int RS = BTHREADS / 8, JA = BM / RS, JB = BT / RS;
    const int lrow = tid >> 3, lpiece = tid & 7;
    const __bf16 *la[JA], *lb[JB];
#pragma unroll
    for (int j = 0; j < JA; ++j) la[j] = ga + (size_t)min(lrow + RS * j, Mr - 1) * lda + lpiece * 8;
#pragma unroll
    for (int j = 0; j < JB; ++j) lb[j] = gb + (size_t)min(lrow + RS * j, Nr - 1) * ldb + lpiece * 8;
    constexpr int D = NC < GEMM_LD ? NC : GEMM_LD;   // chunks in flight in registers
    v4u_t ra[D][JA], rb[D][JB];
    auto load = [&](v4u_t (&xa)[JA], v4u_t (&xb)[JB], int c) {
#pragma unroll
        for (int j = 0; j < JA; ++j) xa[j] = *(const v4u_t *)(la[j] + c * BBK);
#pragma unroll
        for (int j = 0; j < JB; ++j) xb[j] = *(const v4u_t *)(lb[j] + c * BBK);
    };
    auto store = [&](const v4u_t (&xa)[JA], const v4u_t (&xb)[JB], int buf) {
        __bf16 *As = smem + buf * BBUF, *Bs = As + BM * BROW;
#pragma unroll
        for (int j = 0; j < JA; ++j) *(v4u_t *)(As + (lrow + RS * j) * BROW + lpiece * 8) = xa[j];
#pragma unroll
        for (int j = 0; j < JB; ++j) *(v4u_t *)(Bs + (lrow + RS * j) * BROW + lpiece * 8) = xb[j];
    };
    static_for<0, D>([&](auto c) { load(ra[c], rb[c], c); });
    store(ra[0], rb[0], 0);
    if constexpr (D < NC) load(ra[0], rb[0], D);
    __syncthreads();
    const int am = (wave >> 1) * 64, bn = (wave & 1) * 64;
    // Per chunk c: read its fragments (both k-steps) and run its MFMAs; then
    // store chunk c + 1 into the other LDS buffer (free since the last
    // barrier: chunk c - 1's reads completed before it) and issue the load of
    // chunk c + 1 + D; one barrier.  With the stores after the MFMAs, a
    // chunk's loads have the MFMAs' time to land (measured 1% faster than
    // storing between the reads and the MFMAs).
    static_for<0, NC>([&](auto c) {
        constexpr int buf = c & 1;
        const __bf16 *As = smem + buf * BBUF, *Bs = As + BM * BROW;
        bf16x8 fa[BBK / 32][4], fb[BBK / 32][4];
#pragma unroll
        for (int q = 0; q < BBK / 32; ++q)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                fa[q][i] = *(const bf16x8 *)(As + (am + i * 16 + r16) * BROW + q * 32 + kq * 8);
                fb[q][i] = *(const bf16x8 *)(Bs + (bn + i * 16 + r16) * BROW + q * 32 + kq * 8);
            }
#pragma unroll
        for (int q = 0; q < BBK / 32; ++q) {
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[q][i], fb[q][j],
                                                                        acc[i][j], 0, 0, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (c + 1 < NC) {
            // chunk c + 1 sits in register set (c + 1) % D; refill it with c + 1 + D
            constexpr int slot = (c + 1) % D;
            store(ra[slot], rb[slot], (c + 1) & 1);
            if constexpr (c + 1 + D < NC) load(ra[slot], rb[slot], c + 1 + D);
        }
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (c + 1 < NC) __syncthreads();
    });
}

__global__ __launch_bounds__(BTHREADS, 1) void gemm_big_kernel(GemmBatch gb)
{
    constexpr int SM0 = 2 * BBUF, SM1 = BWAVES * STAGE_BYTES / 2;   // bf16 elements
    __shared__ __attribute__((aligned(16))) __bf16 smem[SM0 > SM1 ? SM0 : SM1];
    int agent, t;
    if (!gemm_slot(gb, agent, t)) return;
    const int pi = find_prob(gb, t);
    const GemmProb P = agent_prob(gb, pi, agent);
    t -= P.tile0;
    const int tn = __builtin_amdgcn_readfirstlane(t % P.tiles_n);
    const int tm = __builtin_amdgcn_readfirstlane(t / P.tiles_n);
    const int wave = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
    const int m0 = tm * BM, n0 = tn * BT;
    const int r16 = lane & 15, kq = lane >> 4;
    const __bf16 *ga = (const __bf16 *)P.A + (size_t)m0 * P.lda;
    const __bf16 *gbp = (const __bf16 *)P.B + (size_t)n0 * P.ldb;
    floatx4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    const int Mr = P.M - m0, Nr = P.N - n0;     // rows left in this tile (>= 1)
    switch (P.K / BBK) {
    case 2: big_kloop<2>(ga, gbp, P.lda, P.ldb, Mr, Nr, smem, acc); break;
    case 8: big_kloop<8>(ga, gbp, P.lda, P.ldb, Mr, Nr, smem, acc); break;
    case 16: big_kloop<16>(ga, gbp, P.lda, P.ldb, Mr, Nr, smem, acc); break;
    default: break;   // the launcher routes other K elsewhere
    }
    __builtin_amdgcn_sched_barrier(0);
    const int wm = m0 + (wave >> 1) * 64, wn = n0 + (wave & 1) * 64;
    if (P.mode == EPI_BIAS) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
                epi4<true>(P, wm + i * 16 + kq * 4, wn + j * 16 + r16, v);
            }
        return;
    }
    // each wave stages its 64 x 64 block in LDS (free once every wave has
    // passed this barrier: the last chunk's fragment reads are done) and
    // stores it
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));   // keep these lane terms out of the chunk loop's live set
    const int el = tid % WAVE, ew = tid / WAVE;
    static_assert(BWAVES * STAGE_BYTES <= sizeof(smem) && 64 * EF * 4 <= STAGE_BYTES, "staged blocks fit");
    void *blk = (char *)smem + ew * STAGE_BYTES;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            stage4(P, acc[i][j], wm + i * 16 + (el >> 4) * 4, wn + j * 16 + (el & 15),
                   i * 16 + (el >> 4) * 4, j * 16 + (el & 15), blk);
    __syncthreads();
    store_staged<WAVE>(P, blk, wm, wn, el);
}

// fp32: 16x16 threads, each a 4x4 block of the 64x64 tile; k-slices of 16
// staged in LDS, k-major, so the inner loop reads broadcast-free rows.
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmBatch gb)
{
    __shared__ float As[16][GT + 4];
    __shared__ float Bs[16][GT + 4];
    int agent, t;
    if (!gemm_slot(gb, agent, t)) return;
    const int pi = find_prob(gb, t);
    const GemmProb P = agent_prob(gb, pi, agent);
    t -= P.tile0;
    const int tn = __builtin_amdgcn_readfirstlane(t % P.tiles_n);
    const int tm = __builtin_amdgcn_readfirstlane(t / P.tiles_n);
    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
    const float *A = (const float *)P.A, *B = (const float *)P.B;
    // loader: row lr = tid / 4 of the tile, k-quad lq = tid % 4
    const int lr = tid >> 2, lq = tid & 3;
    const float *la = A + (size_t)min(tm * GT + lr, P.M - 1) * P.lda + lq * 4;
    const float *lb = B + (size_t)min(tn * GT + lr, P.N - 1) * P.ldb + lq * 4;
    float acc[4][4] = {};
    for (int k = 0; k < P.K; k += 16) {
        const floatx4 va = *(const floatx4 *)(la + k);
        const floatx4 vb = *(const floatx4 *)(lb + k);
        __syncthreads();
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            As[lq * 4 + e][lr] = va[e];
            Bs[lq * 4 + e][lr] = vb[e];
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < 16; ++kk) {
            const floatx4 a = *(const floatx4 *)&As[kk][ty * 4];
            const floatx4 b = *(const floatx4 *)&Bs[kk][tx * 4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const float v[4] = {acc[0][j], acc[1][j], acc[2][j], acc[3][j]};
        epi4<false>(P, tm * GT + ty * 4, tn * GT + tx * 4 + j, v);
    }
}

// Minibatch indices outside [0, rows) are clamped into it (never read out
// of bounds).
__device__ __forceinline__ int64_t clamp_row(int64_t r, int64_t rows)
{
    return r < 0 ? 0 : (r >= rows ? rows - 1 : r);
}

// ---------------------------------------------------------------------------
// Minibatch gather: X [B][Kp] and X^T [Kp][B] from the trajectory's
// observation rows idx[i] (columns >= S zeroed), plus the per-row
// transition data.  Tiles of 64 rows x 64 columns through LDS.
// ---------------------------------------------------------------------------
// One update's minibatch gather, as a workgroup body: block (bx, by) of a
// cdiv(B, 64) x cdiv(Kp, 64) grid, agent `agent`.
template <bool BF>
struct GatherArgs {
    const Elem<BF> *obs;
    int64_t ld_obs;
    int vec_obs;
    const float *action, *logp, *adv, *ret;
    const int64_t *idx;   // this update's rows of agent 0; agents aidx apart
    int64_t rows;
    int B, S, Kp, n;
    Elem<BF> *X, *Xt;
    float *Ag, *row_in;
    int64_t aws, aidx;
    int gx, gy;           // the grid: cdiv(B, 64) x cdiv(Kp, 64)
};

template <bool BF>
struct GatherSmem {
    int64_t s_idx[64];
    Elem<BF> tile[64][64 + 16 / sizeof(Elem<BF>)];
};

template <bool BF>
__device__ __forceinline__ void gather_block(const GatherArgs<BF> &ga, int bx, int by, int agent,
                                             GatherSmem<BF> &sm)
{
    typedef uint32_t v4u __attribute__((ext_vector_type(4)));
    const size_t w = (size_t)agent * (size_t)ga.aws;
    const Elem<BF> *__restrict__ obs = ga.obs;
    const float *__restrict__ action = ga.action;
    const int64_t *__restrict__ idx = shifted(ga.idx, (size_t)agent * (size_t)ga.aidx * 8);
    Elem<BF> *__restrict__ X = shifted(ga.X, w);
    Elem<BF> *__restrict__ Xt = shifted(ga.Xt, w);
    float *__restrict__ Ag = shifted(ga.Ag, w);
    float *__restrict__ row_in = shifted(ga.row_in, w);
    const int64_t ld_obs = ga.ld_obs, rows = ga.rows;
    const int B = ga.B, S = ga.S, Kp = ga.Kp, n = ga.n, vec_obs = ga.vec_obs;
    constexpr int VE = 16 / sizeof(Elem<BF>);   // elements per 16-byte vector
    constexpr int VPR = 64 / VE;                 // vectors per tile row
    int64_t *s_idx = sm.s_idx;
    auto &tile = sm.tile;
    const int i0 = bx * 64, c0 = by * 64;
    const int tid = threadIdx.x;
    if (tid < 64) s_idx[tid] = i0 + tid < B ? clamp_row(idx[i0 + tid], rows) : 0;
    __syncthreads();
    // rows of X (16-byte loads and stores), staged in LDS
#pragma unroll
    for (int q = tid; q < 64 * VPR; q += 256) {
        const int r = q / VPR, cv = q % VPR;
        const int i = i0 + r, col = c0 + cv * VE;
        union {
            v4u v;
            Elem<BF> e[VE];
        } u;
        u.v = v4u{0u, 0u, 0u, 0u};
        if (i < B && col < S) {
            const Elem<BF> *src = obs + (size_t)s_idx[r] * ld_obs + col;
            if (vec_obs && col + VE <= S) {
                u.v = *(const v4u *)src;
            } else {
#pragma unroll
                for (int e = 0; e < VE; ++e)
                    if (col + e < S) u.e[e] = src[e];
            }
        }
        if (i < B && col < Kp) *(v4u *)(X + (size_t)i * Kp + col) = u.v;
#pragma unroll
        for (int e = 0; e < VE; ++e) tile[r][cv * VE + e] = u.e[e];
    }
    __syncthreads();
    // columns of X^T: VE consecutive rows of one column per 16-byte store
#pragma unroll
    for (int q = tid; q < 64 * VPR; q += 256) {
        const int c = q / VPR, rv = q % VPR;
        const int col = c0 + c, i = i0 + rv * VE;
        if (col >= Kp || i >= B) continue;
        union {
            v4u v;
            Elem<BF> e[VE];
        } u;
#pragma unroll
        for (int e = 0; e < VE; ++e) u.e[e] = tile[rv * VE + e][c];
        *(v4u *)(Xt + (size_t)col * B + i) = u.v;
    }
    // actions, spread over the column blocks; per-row scalars in the first
    const int per = (n + ga.gy - 1) / ga.gy;
    const int k0 = by * per, k1 = min(n, k0 + per);
    for (int q = tid; q < 64 * (k1 - k0); q += 256) {
        const int r = q / (k1 - k0), k = k0 + q % (k1 - k0);
        if (i0 + r < B) Ag[(size_t)(i0 + r) * n + k] = action[(size_t)s_idx[r] * n + k];
    }
    if (by == 0 && tid < 64 && i0 + tid < B) {
        const int i = i0 + tid;
        const int64_t g = s_idx[tid];
        row_in[i] = ga.logp[g];
        row_in[B + i] = ga.adv[g];
        row_in[2 * B + i] = ga.ret[g];
    }
}

// ---------------------------------------------------------------------------
// Loss and its gradient, one launch over [B] x [vsplit + C2] virtual
// columns in 64 x 64 tiles (vsplit = n_pad rounded up to a whole tile).
// Each workgroup first takes its 64 rows' terms: four threads per row,
// partial sums in fp64 combined in a fixed order, so every column tile of
// the same rows gets the same values:
//   actor tiles: log-probability, ratio, clip decision, g_i = dL/dlogp_i
//     (zero on the clipped branch);
//   critic tiles: V_i and dL/dV_i = 2 (V_i - R_i) / B.
// The first actor tile of a row block writes row_out[0], [2], [4]
// (g, surrogate, |rho - 1| > clip), the first critic tile row_out[1], [3]
// (dL/dV, squared error); the first actor tile of all writes
// row_out[5 B] = sum_k log sigma_k.  Then the tile: columns < vsplit give dmu
// (row-major and transposed, zero for n <= col < n_pad) and the log-std
// terms (transposed), the rest the critic's second pre-activation gradient
// dV wc3 (1 - hc2^2) (row-major and transposed).  Every global load of a
// phase is issued before the first use, with clamped addresses.
// ---------------------------------------------------------------------------
template <bool BF>
__global__ __launch_bounds__(256) void loss_kernel(
    const float *__restrict__ mu, const float *__restrict__ Ag, const float *__restrict__ row_in,
    const Elem<BF> *__restrict__ Hc2, const float *__restrict__ params, int64_t ols,
    int64_t owc3, int64_t obc3, int B, int n, int n_pad, int vsplit, int C2, float clip,
    float *__restrict__ row_out, Elem<BF> *__restrict__ dMU, Elem<BF> *__restrict__ dMUt,
    float *__restrict__ LSt, Elem<BF> *__restrict__ dZc2, Elem<BF> *__restrict__ dZc2t,
    int64_t aws, int64_t aprm)
{
    {   // agent blockIdx.z: its workspace and its parameters
        const size_t w = (size_t)blockIdx.z * (size_t)aws;
        mu = shifted(mu, w);
        Ag = shifted(Ag, w);
        row_in = shifted(row_in, w);
        Hc2 = shifted(Hc2, w);
        row_out = shifted(row_out, w);
        dMU = shifted(dMU, w);
        dMUt = shifted(dMUt, w);
        LSt = shifted(LSt, w);
        dZc2 = shifted(dZc2, w);
        dZc2t = shifted(dZc2t, w);
        params = shifted(params, (size_t)blockIdx.z * (size_t)aprm);
    }
    __shared__ float t1[64][65];
    __shared__ float t2[64][65];
    __shared__ float s_row[64];    // g (actor tiles) or dL/dV (critic tiles)
    __shared__ float s_col[64];    // 1/sigma^2 (actor) or the critic head's weight
    __shared__ float s_inv[128];   // 1/sigma_k^2, k < n (actor tiles)
    __shared__ float s_ls[128];    // log sigma_k, k < n
    const int i0 = blockIdx.x * 64, c0 = blockIdx.y * 64;
    const bool actor = c0 < vsplit;
    const int tid = threadIdx.x;
    const float *ls = params + ols, *wc3 = params + owc3;
    {
        // every load of the set-up at once (clamped), then the role's values
        const int col = c0 + (tid & 63);
        const float l_k = ls[min(tid & 127, n - 1)];
        const float l_c = ls[min(col, n - 1)];
        const float w_c = wc3[min(max(col - vsplit, 0), C2 - 1)];
        if (actor) {
            if (tid < 128) {
                if (tid < n) s_inv[tid] = expf(-2.0f * l_k);
            } else if (tid - 128 < n) {
                s_ls[tid - 128] = l_k;
            }
        }
        if (tid < 64)
            s_col[tid] = actor ? (col < n ? expf(-2.0f * l_c) : 0.f)
                               : (col - vsplit < C2 ? (float)to_elem<BF>(w_c) : 0.f);
    }
    __syncthreads();
    if (actor && blockIdx.x == 0 && blockIdx.y == 0 && tid == 0) {
        // sum_k log sigma_k before this update's Adam step (the entropy)
        double sl = 0.0;
        for (int k = 0; k < n; ++k) sl += (double)s_ls[k];
        row_out[5 * B] = (float)sl;
    }

    // row terms: thread (r = tid / 4, sub = tid % 4)
    {
        const int r = tid >> 2, sub = tid & 3;
        const int i = min(i0 + r, B - 1);
        const float lp_old = row_in[i], A_i = row_in[B + i], R_i = row_in[2 * B + i];
        double part = 0.0;
        if (actor) {
            // log N(a; mu, sigma) over k = sub + 4 j (n <= 128)
            float x[32], y[32];
#pragma unroll
            for (int j = 0; j < 32; ++j) {
                const int k = min(sub + 4 * j, n - 1);
                x[j] = Ag[(size_t)i * n + k];
                y[j] = mu[(size_t)i * n + k];
            }
#pragma unroll
            for (int j = 0; j < 32; ++j) {
                const int k = sub + 4 * j;
                if (k < n) {
                    const float d = x[j] - y[j];
                    part += (double)(-0.5f * (d * d * s_inv[k]) - s_ls[k]);
                }
            }
        } else {
            // V = wc3 . hc2 over 8-element pieces q = sub + 4 j (C2 % 32 == 0)
            const Elem<BF> *h = Hc2 + (size_t)i * C2;
            const int nq = C2 / 32;
#pragma unroll 4
            for (int j = 0; j < nq; ++j) {
                const int k0 = (sub + 4 * j) * 8;
                float hv[8];
                if constexpr (BF) {
                    const bf16x8 v = *(const bf16x8 *)(h + k0);
#pragma unroll
                    for (int e = 0; e < 8; ++e) hv[e] = (float)v[e];
                } else {
                    const floatx4 v0 = *(const floatx4 *)(h + k0);
                    const floatx4 v1 = *(const floatx4 *)(h + k0 + 4);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        hv[e] = v0[e];
                        hv[4 + e] = v1[e];
                    }
                }
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    part += (double)((float)to_elem<BF>(wc3[k0 + e]) * hv[e]);
            }
        }
        // ((s0 + s1) + (s2 + s3)): the same sum in all four lanes
        part += __shfl_xor(part, 1);
        part += __shfl_xor(part, 2);
        if (sub == 0) {
            const bool live = i0 + r < B;
            const int ii = i0 + r;
            if (actor) {
                const double lp = part - 0.5 * (double)n * (double)LN_2PI_F;
                const double A = A_i;
                const double rho = exp(lp - (double)lp_old);
                const double rc = fmin(fmax(rho, 1.0 - clip), 1.0 + clip);
                const bool unclipped = rho * A <= rc * A;
                const float g = unclipped ? (float)(-A * rho / (double)B) : 0.0f;
                s_row[r] = live ? g : 0.f;
                if (live && blockIdx.y == 0) {
                    row_out[ii] = g;
                    row_out[2 * B + ii] = (float)(unclipped ? rho * A : rc * A);
                    row_out[4 * B + ii] = fabs(rho - 1.0) > (double)clip ? 1.0f : 0.0f;
                }
            } else {
                const float V = (float)(part + (double)params[obc3]);
                const double e = (double)V - (double)R_i;
                const float dV = (float)(2.0 * e / (double)B);
                s_row[r] = live ? dV : 0.f;
                if (live && c0 == vsplit) {
                    row_out[B + ii] = dV;
                    row_out[3 * B + ii] = (float)(e * e);
                }
            }
        }
    }
    __syncthreads();

    // the tile, row-major: loads first, then values and stores
    if (actor) {
        float va[16], vb[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int q = tid + 256 * j;
            const int i = min(i0 + (q >> 6), B - 1), k = min(c0 + (q & 63), n - 1);
            va[j] = Ag[(size_t)i * n + k];
            vb[j] = mu[(size_t)i * n + k];
        }
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int q = tid + 256 * j;
            const int r = q >> 6, c = q & 63;
            const int i = i0 + r, col = c0 + c;
            float a = 0.f, b = 0.f;
            if (col < n) {
                const float d = va[j] - vb[j];
                const float inv = s_col[c];
                const float g = s_row[r];
                a = g * (d * inv);
                b = g * (d * d * inv - 1.0f);
            }
            if (i < B && col < n_pad) dMU[(size_t)i * n_pad + col] = to_elem<BF>(a);
            t1[r][c] = a;
            t2[r][c] = b;
        }
    } else {
        Elem<BF> vh[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int q = tid + 256 * j;
            const int i = min(i0 + (q >> 6), B - 1), k = min(c0 - vsplit + (q & 63), C2 - 1);
            vh[j] = Hc2[(size_t)i * C2 + k];
        }
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int q = tid + 256 * j;
            const int r = q >> 6, c = q & 63;
            const int i = i0 + r, k = c0 - vsplit + c;
            float a = 0.f;
            if (k < C2) {
                const float h = (float)vh[j];
                a = s_row[r] * s_col[c] * (1.0f - h * h);
                if (i < B) dZc2[(size_t)i * C2 + k] = to_elem<BF>(a);
            }
            t1[r][c] = a;
        }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        const int q = tid + 256 * j;
        const int c = q >> 6, r = q & 63;
        const int i = i0 + r, col = c0 + c;
        if (i >= B) continue;
        if (actor) {
            if (col < n_pad) dMUt[(size_t)col * B + i] = to_elem<BF>(t1[r][c]);
            if (col < n) LSt[(size_t)col * B + i] = t2[r][c];
        } else if (col - vsplit < C2) {
            dZc2t[(size_t)(col - vsplit) * B + i] = to_elem<BF>(t1[r][c]);
        }
    }
}

// ---------------------------------------------------------------------------
// The tail of an update, one launch of two kinds of workgroups:
//  - blocks [0, mtiles): Adam over 64 x 64 tiles of the weight matrices
//    (when do_adam), each updated weight written back and rounded into its
//    row-major operand copy and, through LDS, its transposed copy;
//  - the rest: row sums, one wave per row (fp64 partials, fixed order),
//    dst[r] = scale * sum_b src[r][b] (* w[b]) + add; a row that is the
//    gradient of a bias, log-std or critic-head element (pidx >= 0) also
//    takes that element's Adam step.  The statistics are rows too.
// The two kinds touch disjoint memory.
// ---------------------------------------------------------------------------
struct RedSeg {
    const void *src;
    int64_t ld;
    int rows, len;
    int bf;             // source elements are bf16
    const float *w;     // optional weights [len]
    float *dst;         // fp32 destination, or
    double *dst64;      // fp64 destination (stats)
    double scale, add;
    int row0;           // first global row of this segment
    int vec;            // rows 16-byte aligned and len a multiple of 16 bytes
    int64_t pidx;       // flat index of row 0's parameter, or -1
};
constexpr int MAX_SEGS = 12;
struct RedBatch {
    RedSeg s[MAX_SEGS];
    int ns, total_rows;
};

struct AdamSeg {
    int64_t off;        // flat offset of the master
    int rows, cols;     // master shape
    int rows_pad, cols_pad;   // copy shape (zero outside the master)
    void *copy;         // row-major copy [.][ld_copy] at row copy_row0
    int64_t ld_copy;
    int copy_row0;
    void *copyT;        // transposed copy [cols_pad][ld_copyT], or null
    int64_t ld_copyT;
    int tiles_c, tile0;
};
constexpr int MAX_ASEGS = 5;
constexpr int AT = 64;              // Adam tile edge
struct AdamBatch {
    AdamSeg s[MAX_ASEGS];
    int ns;
    float *params, *m, *v;
    const float *grad;
    float lr, b1, b2, eps, bc1, bc2;
    int do_adam;
    int64_t aws, aprm, ast;   // bytes between agents: workspace, parameters, statistics
};

// One agent's parameters, moments and gradient
struct AdamPtrs {
    float *params, *m, *v;
    const float *grad;
};

// One Adam step of one element (the moments and the master written back).
__device__ __forceinline__ float adam_step(const AdamBatch &ab, const AdamPtrs &q, int64_t p,
                                           float th, float g, float m0, float v0)
{
    const float m = ab.b1 * m0 + (1.0f - ab.b1) * g;
    const float v = ab.b2 * v0 + (1.0f - ab.b2) * (g * g);
    q.m[p] = m;
    q.v[p] = v;
    const float mh = m / ab.bc1, vh = v / ab.bc2;
    th = th - ab.lr * (mh / (sqrtf(vh) + ab.eps));
    q.params[p] = th;
    return th;
}

template <bool BF>
__device__ __forceinline__ void adam_tile(const AdamBatch &ab, const AdamPtrs &ap, int t,
                                          Elem<BF> (*tile)[AT + 1])
{
    int si = 0;
#pragma unroll
    for (int q = 1; q < MAX_ASEGS; ++q)
        if (q < ab.ns && t >= ab.s[q].tile0) si = q;
    AdamSeg S = ab.s[si];
    S.copy = shifted(S.copy, (size_t)blockIdx.y * (size_t)ab.aws);
    S.copyT = shifted(S.copyT, (size_t)blockIdx.y * (size_t)ab.aws);
    t -= S.tile0;
    const int tid = threadIdx.x;
    const int r0 = (t / S.tiles_c) * AT, c0 = (t % S.tiles_c) * AT;
    // element j of a thread: row r0 + q / 64, column c0 + q % 64, q = tid + 256 j
    constexpr int NJ = AT * AT / 256;
    float th[NJ], gg[NJ], mm[NJ], vv[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int q = tid + 256 * j;
        const int r = min(r0 + q / AT, S.rows - 1), c = min(c0 + q % AT, S.cols - 1);
        const int64_t p = S.off + (int64_t)r * S.cols + c;
        th[j] = ap.params[p];
        if (ab.do_adam) {
            gg[j] = ap.grad[p];
            mm[j] = ap.m[p];
            vv[j] = ap.v[p];
        }
    }
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int q = tid + 256 * j;
        const int r = r0 + q / AT, c = c0 + q % AT;
        float w = 0.0f;
        if (r < S.rows && c < S.cols) {
            w = th[j];
            if (ab.do_adam)
                w = adam_step(ab, ap, S.off + (int64_t)r * S.cols + c, w, gg[j], mm[j], vv[j]);
        }
        const Elem<BF> e = to_elem<BF>(w);
        if (r < S.rows_pad && c < S.cols_pad)
            ((Elem<BF> *)S.copy)[(size_t)(S.copy_row0 + r) * S.ld_copy + c] = e;
        tile[q / AT][q % AT] = e;
    }
    if (!S.copyT) return;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int q = tid + 256 * j;
        const int c = c0 + q / AT, r = r0 + q % AT;
        if (r < S.rows_pad && c < S.cols_pad)
            ((Elem<BF> *)S.copyT)[(size_t)c * S.ld_copyT + r] = tile[q % AT][q / AT];
    }
}

__device__ __forceinline__ void reduce_row(const RedBatch &rb, const AdamBatch &ab,
                                           const AdamPtrs &ap, int g)
{
    const int lane = threadIdx.x % WAVE;
    int si = 0;
#pragma unroll
    for (int q = 1; q < MAX_SEGS; ++q)
        if (q < rb.ns && g >= rb.s[q].row0) si = q;
    RedSeg S = rb.s[si];
    {   // agent blockIdx.y: sources, weights and gradient in its workspace
        const size_t w = (size_t)blockIdx.y * (size_t)ab.aws;
        S.src = shifted(S.src, w);
        S.w = shifted(S.w, w);
        S.dst = shifted(S.dst, w);
        S.dst64 = shifted(S.dst64, (size_t)blockIdx.y * (size_t)ab.ast);
    }
    const int r = g - S.row0;
    double acc = 0.0;
    if (S.vec && S.bf) {   // 8 bf16 per lane per step
        const __bf16 *p = (const __bf16 *)S.src + (size_t)r * S.ld;
        for (int b = lane * 8; b < S.len; b += WAVE * 8) {
            const bf16x8 x = *(const bf16x8 *)(p + b);
            float part = 0.f;
#pragma unroll
            for (int e = 0; e < 8; ++e) part += (float)x[e] * (S.w ? S.w[b + e] : 1.0f);
            acc += (double)part;
        }
    } else if (S.vec) {    // 4 floats per lane per step
        const float *p = (const float *)S.src + (size_t)r * S.ld;
        for (int b = lane * 4; b < S.len; b += WAVE * 4) {
            const floatx4 x = *(const floatx4 *)(p + b);
            float part = 0.f;
#pragma unroll
            for (int e = 0; e < 4; ++e) part += x[e] * (S.w ? S.w[b + e] : 1.0f);
            acc += (double)part;
        }
    } else if (S.bf) {
        const __bf16 *p = (const __bf16 *)S.src + (size_t)r * S.ld;
        for (int b = lane; b < S.len; b += WAVE)
            acc += (double)((float)p[b] * (S.w ? S.w[b] : 1.0f));
    } else {
        const float *p = (const float *)S.src + (size_t)r * S.ld;
        for (int b = lane; b < S.len; b += WAVE)
            acc += (double)(p[b] * (S.w ? S.w[b] : 1.0f));
    }
    acc = wave_sum(acc);
    if (lane == 0) {
        const double v = S.scale * acc + S.add;
        if (S.dst64) {
            S.dst64[r] = v;
        } else {
            S.dst[r] = (float)v;
            if (S.pidx >= 0 && ab.do_adam) {
                const int64_t p = S.pidx + r;
                adam_step(ab, ap, p, ap.params[p], (float)v, ap.m[p], ap.v[p]);
            }
        }
    }
}

// blockIdx.y is the agent.  Blocks [0, 8 per) take the matrix tiles,
// XCD-aware: workgroups are dealt round-robin over the 8 XCDs, so block b
// takes tile (b % 8) per + b / 8 and each XCD walks a contiguous run of
// tiles (rows of W1 and Wc1 are not line-aligned: neighbouring tiles share
// lines, now in one L2).  For agent y the XCD of block b is that of b + y
// gridDim.x, so blocks with equal b % 8 still share one.  The next
// cdiv(rows, 4) blocks take the row sums; the last gblocks blocks gather the
// next update's minibatch (its X, X^T, actions and row data are read by
// nothing in this launch, and by nothing of this update after it).
template <bool BF>
__global__ __launch_bounds__(256) void adam_tail_kernel(AdamBatch ab, RedBatch rb, int mtiles,
                                                        GatherArgs<BF> ga, int gblocks)
{
    __shared__ Elem<BF> tile[AT][AT + 1];
    __shared__ GatherSmem<BF> gsm;
    // agent blockIdx.y
    const size_t q = (size_t)blockIdx.y * (size_t)ab.aprm;
    const AdamPtrs ap{shifted(ab.params, q), shifted(ab.m, q), shifted(ab.v, q),
                      shifted(ab.grad, (size_t)blockIdx.y * (size_t)ab.aws)};
    const int per = (mtiles + 7) / 8, rblocks = (rb.total_rows + 3) / 4;
    const int b = blockIdx.x;
    if (b < 8 * per) {
        const int t = (b % 8) * per + b / 8;
        if (t < mtiles) adam_tile<BF>(ab, ap, t, tile);
        return;
    }
    if (b < 8 * per + rblocks) {
        const int g = (b - 8 * per) * 4 + threadIdx.x / WAVE;
        if (g < rb.total_rows) reduce_row(rb, ab, ap, g);
        return;
    }
    const int g = b - 8 * per - rblocks;
    if (g < gblocks) gather_block<BF>(ga, g % ga.gx, g / ga.gx, blockIdx.y, gsm);
}

// Minibatch rows: draw i of update counter c for agent g is word i % 4 of
// Philox4x32-10(ctr = (i/4, c, g, 0x4D42), key = seed), mapped to one of the
// agent's R = L epa stored transitions by the high half of w R, then to the
// row j E + e of the time-major arrays.  One thread per draw.
__global__ __launch_bounds__(256) void minibatch_rows_kernel(uint32_t k0, uint32_t k1,
                                                             uint64_t counter, int n_updates,
                                                             int B, int E, int agent, int epa,
                                                             uint64_t R, int64_t *idx)
{
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= (int64_t)n_updates * B) return;
    const int u = (int)(t / B), i = (int)(t % B);
    const U4 w = philox4x32_10(U4{(uint32_t)(i / 4), (uint32_t)(counter + (uint64_t)u),
                                  (uint32_t)agent, 0x4D42u},
                               k0, k1);
    const uint32_t word = (i & 3) == 0 ? w.x : (i & 3) == 1 ? w.y : (i & 3) == 2 ? w.z : w.w;
    const uint64_t draw = ((uint64_t)word * R) >> 32;
    const int64_t j = (int64_t)(draw / (uint64_t)epa);
    const int64_t e = (int64_t)agent * epa + (int64_t)(draw % (uint64_t)epa);
    idx[t] = j * E + e;
}

int cdiv(int a, int b) { return (a + b - 1) / b; }

}  // namespace

hipError_t launch_minibatch_rows(uint64_t seed, uint64_t counter, int n_updates, int B, int L,
                                 int E, int agent, int epa, int64_t *idx, hipStream_t s)
{
    const int64_t total = (int64_t)n_updates * B;
    hipLaunchKernelGGL(minibatch_rows_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256),
                       0, s, (uint32_t)seed, (uint32_t)(seed >> 32), counter, n_updates, B, E,
                       agent, epa, (uint64_t)L * (uint64_t)epa, idx);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Layout
// ---------------------------------------------------------------------------
bool ppo_layout(const tp_ppo *c, PpoLayout *L)
{
    L->dtype = c->dtype;
    L->S = c->dims[0];
    L->H1 = c->dims[1];
    L->H2 = c->dims[2];
    L->n = c->dims[3];
    L->C1 = c->dims[4];
    L->C2 = c->dims[5];
    L->B = c->batch;
    L->Kp = (L->S + 31) / 32 * 32;
    L->n_pad = (L->n + 31) / 32 * 32;
    L->HC1 = L->H1 + L->C1;
    int64_t o = 0;
    auto seg = [&](int64_t count) {
        const int64_t at = o;
        o += count;
        return at;
    };
    L->oW1 = seg((int64_t)L->H1 * L->S);
    L->ob1 = seg(L->H1);
    L->oW2 = seg((int64_t)L->H2 * L->H1);
    L->ob2 = seg(L->H2);
    L->oW3 = seg((int64_t)L->n * L->H2);
    L->ob3 = seg(L->n);
    L->ols = seg(L->n);
    L->oWc1 = seg((int64_t)L->C1 * L->S);
    L->obc1 = seg(L->C1);
    L->oWc2 = seg((int64_t)L->C2 * L->C1);
    L->obc2 = seg(L->C2);
    L->owc3 = seg(L->C2);
    L->obc3 = seg(1);
    L->P = o;

    const size_t es = c->dtype == TP_BF16 ? 2 : 4;
    size_t w = 0;
    auto area = [&](size_t bytes) {
        const size_t at = w;
        w += (bytes + 255) / 256 * 256;
        return at;
    };
    const size_t B = L->B;
    L->wWcat1 = area(es * L->HC1 * L->Kp);
    L->wW2 = area(es * L->H2 * L->H1);
    L->wW2t = area(es * L->H1 * L->H2);
    L->wWc2 = area(es * L->C2 * L->C1);
    L->wWc2t = area(es * L->C1 * L->C2);
    L->wW3 = area(es * L->n_pad * L->H2);
    L->wW3t = area(es * L->H2 * L->n_pad);
    L->wX = area(es * B * L->Kp);
    L->wXt = area(es * L->Kp * B);
    L->wH1 = area(es * B * L->HC1);
    L->wH1t = area(es * L->HC1 * B);
    L->wH2 = area(es * B * L->H2);
    L->wH2t = area(es * L->H2 * B);
    L->wHc2 = area(es * B * L->C2);
    L->wHc2t = area(es * L->C2 * B);
    L->wMU = area(4 * B * L->n);
    L->wAg = area(4 * B * L->n);
    L->wRowIn = area(4 * 3 * B);
    L->wRowOut = area(4 * (5 * B + 1));
    L->wdMU = area(es * B * L->n_pad);
    L->wdMUt = area(es * L->n_pad * B);
    L->wLSt = area(4 * L->n * B);
    L->wdZc2 = area(es * B * L->C2);
    L->wdZc2t = area(es * L->C2 * B);
    L->wdZ2 = area(es * B * L->H2);
    L->wdZ2t = area(es * L->H2 * B);
    L->wdZ1t = area(es * L->HC1 * B);
    L->wG = area(4 * (size_t)L->P);
    L->total = w;
    return true;
}

// ---------------------------------------------------------------------------
// One call: refresh the operand copies, then n_updates minibatch updates
// ---------------------------------------------------------------------------
namespace {

GemmProb prob(const void *A, int64_t lda, const void *B, int64_t ldb, int M, int N, int K,
              int mode)
{
    GemmProb p{};
    p.A = A;
    p.B = B;
    p.lda = lda;
    p.ldb = ldb;
    p.M = M;
    p.N = N;
    p.K = K;
    p.mode = mode;
    p.bsplit = 1 << 30;
    p.gsplit = 1 << 30;
    p.gcols = 1 << 30;
    return p;
}

// Agents of one call: count and byte strides between their workspaces and
// parameter vectors.
struct Agents {
    int n;
    int64_t aws, aprm;
};

hipError_t run_gemms(bool bf, const Agents &ag, std::initializer_list<GemmProb> ps, hipStream_t s)
{
    GemmBatch gb{};
    gb.aws = ag.aws;
    gb.aprm = ag.aprm;
    // kernel choice: bf16 products with K in {128, 512, 1024} go through
    // LDS, in 256 x 128 tiles when the launch has at least BIG_MIN_TILES
    // tiles' worth of 128 x 128
    bool staged = bf, big = bf;
    int tiles_big = 0;
    for (const GemmProb &p : ps) {
        const int nc = p.K / LBK, nb = p.K / BBK;
        const bool ld_ok = p.lda % 8 == 0 && p.ldb % 8 == 0;
        staged = staged && p.K % LBK == 0 && (nc == 1 || nc == 4 || nc == 8) && ld_ok;
        big = big && p.K % BBK == 0 && (nb == 2 || nb == 8 || nb == 16) && ld_ok;
        tiles_big += cdiv(p.M, BT) * cdiv(p.N, BT);
    }
    big = big && tiles_big * ag.n >= BIG_MIN_TILES;
    const int TN = big ? BT : GT, TM = big ? BM : GT;
    int tiles = 0;
    for (const GemmProb &p : ps) {
        GemmProb q = p;
        q.tiles_n = cdiv(q.N, TN);
        q.tile0 = tiles;
        tiles += q.tiles_n * cdiv(q.M, TM);
        gb.p[gb.np++] = q;
    }
    gb.tiles = tiles;
    gb.na = ag.n;
    const dim3 grid(8 * cdiv(tiles * ag.n, 8));
    if (big) hipLaunchKernelGGL(gemm_big_kernel, grid, dim3(BTHREADS), 0, s, gb);
    else if (staged) hipLaunchKernelGGL(gemm_lds_kernel, grid, dim3(LTHREADS), 0, s, gb);
    else if (bf) hipLaunchKernelGGL(gemm_bf16_kernel, grid, dim3(256), 0, s, gb);
    else hipLaunchKernelGGL(gemm_f32_kernel, grid, dim3(256), 0, s, gb);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_ppo_update(const PpoArgs &a, hipStream_t s)
{
    const PpoLayout &L = a.lay;
    const bool bf = L.dtype == TP_BF16;
    const size_t es = bf ? 2 : 4;
    uint8_t *ws = (uint8_t *)a.workspace;
    auto W = [&](size_t off) { return (void *)(ws + off); };
    const int B = L.B;
    float *prm = a.params;
    float *grad = (float *)W(L.wG);
    // agents: workspaces a.ws_stride bytes apart, parameter vectors (and
    // moments) a.agent_stride floats apart; minibatch indices [A][U][B],
    // statistics [A][U][4]
    const int NA = a.n_agents;
    const Agents ag{NA, a.ws_stride, a.agent_stride * (int64_t)sizeof(float)};

    // Adam / refresh segments
    AdamBatch ab{};
    ab.params = prm;
    ab.m = a.adam_m;
    ab.v = a.adam_v;
    ab.grad = grad;
    ab.lr = a.lr;
    ab.b1 = a.beta1;
    ab.b2 = a.beta2;
    ab.eps = a.eps;
    ab.aws = ag.aws;
    ab.aprm = ag.aprm;
    ab.ast = (int64_t)a.n_updates * 4 * (int64_t)sizeof(double);
    int atiles = 0;
    auto mseg = [&](int64_t off, int rows, int cols, int rows_pad, int cols_pad, void *copy,
                    int64_t ldc, int row0, void *copyT, int64_t ldt) {
        AdamSeg g{};
        g.off = off;
        g.rows = rows;
        g.cols = cols;
        g.rows_pad = rows_pad;
        g.cols_pad = cols_pad;
        g.copy = copy;
        g.ld_copy = ldc;
        g.copy_row0 = row0;
        g.copyT = copyT;
        g.ld_copyT = ldt;
        g.tile0 = atiles;
        g.tiles_c = cdiv(cols_pad, AT);
        atiles += g.tiles_c * cdiv(rows_pad, AT);
        ab.s[ab.ns++] = g;
    };
    mseg(L.oW1, L.H1, L.S, L.H1, L.Kp, W(L.wWcat1), L.Kp, 0, nullptr, 0);
    mseg(L.oWc1, L.C1, L.S, L.C1, L.Kp, W(L.wWcat1), L.Kp, L.H1, nullptr, 0);
    mseg(L.oW2, L.H2, L.H1, L.H2, L.H1, W(L.wW2), L.H1, 0, W(L.wW2t), L.H2);
    mseg(L.oWc2, L.C2, L.C1, L.C2, L.C1, W(L.wWc2), L.C1, 0, W(L.wWc2t), L.C2);
    mseg(L.oW3, L.n, L.H2, L.n_pad, L.H2, W(L.wW3), L.H2, 0, W(L.wW3t), L.n_pad);
    // The vectors (b1, b2, b3, log-std, bc1, bc2, wc3, bc3) take their Adam
    // steps in the row sums that produce their gradients.
    const int mtiles = atiles;

    // the minibatch gather of update u (it rides in the launch before that
    // update: the initial refresh, or update u - 1's tail)
    const int vec_obs = ((uintptr_t)a.obs % 16 == 0 && (a.ld_obs * (int64_t)es) % 16 == 0) ? 1 : 0;
    GatherArgs<true> gab{};
    GatherArgs<false> gaf{};
    auto gather_args = [&](auto &g, int u) {
        typedef std::remove_const_t<std::remove_reference_t<decltype(*g.obs)>> E;
        g.obs = (const E *)a.obs;
        g.ld_obs = a.ld_obs;
        g.vec_obs = vec_obs;
        g.action = a.action;
        g.logp = a.logp;
        g.adv = a.adv;
        g.ret = a.ret;
        g.idx = a.idx + (size_t)u * B;
        g.rows = a.rows;
        g.B = B;
        g.S = L.S;
        g.Kp = L.Kp;
        g.n = L.n;
        g.X = (E *)W(L.wX);
        g.Xt = (E *)W(L.wXt);
        g.Ag = (float *)W(L.wAg);
        g.row_in = (float *)W(L.wRowIn);
        g.aws = ag.aws;
        g.aidx = (int64_t)a.n_updates * B;
        g.gx = cdiv(B, 64);
        g.gy = cdiv(L.Kp, 64);
    };

    // Adam (or, with do_adam = 0, only the operand-copy refresh), the row
    // sums and the gather of update gu (none if gu < 0), one launch
    auto tail = [&](int do_adam, int64_t step, const RedBatch &rb, int gu) -> hipError_t {
        ab.do_adam = do_adam;
        ab.bc1 = (float)(1.0 - pow((double)a.beta1, (double)step));
        ab.bc2 = (float)(1.0 - pow((double)a.beta2, (double)step));
        const int gblocks = gu >= 0 ? cdiv(B, 64) * cdiv(L.Kp, 64) : 0;
        const dim3 grid(8 * cdiv(mtiles, 8) + cdiv(rb.total_rows, 4) + gblocks, NA);
        if (bf) {
            gather_args(gab, gu >= 0 ? gu : 0);
            hipLaunchKernelGGL(adam_tail_kernel<true>, grid, dim3(256), 0, s, ab, rb, mtiles, gab,
                               gblocks);
        } else {
            gather_args(gaf, gu >= 0 ? gu : 0);
            hipLaunchKernelGGL(adam_tail_kernel<false>, grid, dim3(256), 0, s, ab, rb, mtiles, gaf,
                               gblocks);
        }
        return hipGetLastError();
    };
    hipError_t e = tail(0, 1, RedBatch{}, 0);
    if (e != hipSuccess) return e;

    void *X = W(L.wX), *Xt = W(L.wXt), *H1 = W(L.wH1), *H1t = W(L.wH1t);
    void *H2 = W(L.wH2), *H2t = W(L.wH2t), *Hc2 = W(L.wHc2), *Hc2t = W(L.wHc2t);
    float *MU = (float *)W(L.wMU), *Ag = (float *)W(L.wAg);
    float *row_in = (float *)W(L.wRowIn), *row_out = (float *)W(L.wRowOut);
    void *dMU = W(L.wdMU), *dMUt = W(L.wdMUt);
    float *LSt = (float *)W(L.wLSt);
    void *dZc2 = W(L.wdZc2), *dZc2t = W(L.wdZc2t), *dZ2 = W(L.wdZ2), *dZ2t = W(L.wdZ2t);
    void *dZ1t = W(L.wdZ1t);
    auto at = [&](void *base, size_t elems) { return (void *)((uint8_t *)base + elems * es); };

    for (int u = 0; u < a.n_updates; ++u) {
        // forward 1: [h1 | hc1] = tanh(X [W1; Wc1]^T + [b1 | bc1])
        {
            GemmProb p = prob(X, L.Kp, W(L.wWcat1), L.Kp, B, L.HC1, L.Kp, EPI_TANH);
            p.bias0 = prm + L.ob1;
            p.bias1 = prm + L.obc1;
            p.bsplit = L.H1;
            p.out = H1;
            p.ldo = L.HC1;
            p.outT = H1t;
            p.ldt = B;
            if ((e = run_gemms(bf, ag, {p}, s)) != hipSuccess) return e;
        }
        // forward 2: h2 and hc2
        {
            GemmProb pa = prob(H1, L.HC1, W(L.wW2), L.H1, B, L.H2, L.H1, EPI_TANH);
            pa.bias0 = prm + L.ob2;
            pa.out = H2;
            pa.ldo = L.H2;
            pa.outT = H2t;
            pa.ldt = B;
            GemmProb pc = prob(at(H1, L.H1), L.HC1, W(L.wWc2), L.C1, B, L.C2, L.C1, EPI_TANH);
            pc.bias0 = prm + L.obc2;
            pc.out = Hc2;
            pc.ldo = L.C2;
            pc.outT = Hc2t;
            pc.ldt = B;
            if ((e = run_gemms(bf, ag, {pa, pc}, s)) != hipSuccess) return e;
        }
        // forward 3: mu = h2 W3^T + b3
        {
            GemmProb p = prob(H2, L.H2, W(L.wW3), L.H2, B, L.n, L.H2, EPI_BIAS);
            p.bias0 = prm + L.ob3;
            p.out = MU;
            p.ldo = L.n;
            if ((e = run_gemms(bf, ag, {p}, s)) != hipSuccess) return e;
        }
        // loss and its gradient tiles: actor columns [0, n_pad) in whole
        // tiles, then the critic's C2 columns
        {
            const int ntA = cdiv(L.n_pad, 64);
            const dim3 grid(cdiv(B, 64), ntA + cdiv(L.C2, 64), NA);
            if (bf)
                hipLaunchKernelGGL(loss_kernel<true>, grid, dim3(256), 0, s, MU, Ag, row_in,
                                   (const __bf16 *)Hc2, prm, L.ols, L.owc3, L.obc3, B, L.n,
                                   L.n_pad, ntA * 64, L.C2, a.clip, row_out, (__bf16 *)dMU,
                                   (__bf16 *)dMUt, LSt, (__bf16 *)dZc2, (__bf16 *)dZc2t, ag.aws,
                                   ag.aprm);
            else
                hipLaunchKernelGGL(loss_kernel<false>, grid, dim3(256), 0, s, MU, Ag, row_in,
                                   (const float *)Hc2, prm, L.ols, L.owc3, L.obc3, B, L.n,
                                   L.n_pad, ntA * 64, L.C2, a.clip, row_out, (float *)dMU,
                                   (float *)dMUt, LSt, (float *)dZc2, (float *)dZc2t, ag.aws,
                                   ag.aprm);
        }
        // backward stage A: dW3, dZ2 (actor); dWc2, dZc1 (critic)
        {
            GemmProb g3 = prob(dMUt, B, H2t, B, L.n, L.H2, B, EPI_GRAD);
            g3.g0 = grad + L.oW3;
            g3.ldg = L.H2;
            GemmProb b3 = prob(dMU, L.n_pad, W(L.wW3t), L.n_pad, B, L.H2, L.n_pad, EPI_DTANH);
            b3.hsrc = H2t;
            b3.ldh = B;
            b3.out = dZ2;
            b3.ldo = L.H2;
            b3.outT = dZ2t;
            b3.ldt = B;
            GemmProb gc2 = prob(dZc2t, B, at(H1t, (size_t)L.H1 * B), B, L.C2, L.C1, B, EPI_GRAD);
            gc2.g0 = grad + L.oWc2;
            gc2.ldg = L.C1;
            GemmProb bc2 = prob(dZc2, L.C2, W(L.wWc2t), L.C2, B, L.C1, L.C2, EPI_DTANH);
            bc2.hsrc = at(H1t, (size_t)L.H1 * B);
            bc2.ldh = B;
            bc2.outT = at(dZ1t, (size_t)L.H1 * B);
            bc2.ldt = B;
            if ((e = run_gemms(bf, ag, {g3, b3, gc2, bc2}, s)) != hipSuccess) return e;
        }
        // backward stage B: dW2, dZ1 (actor)
        {
            GemmProb g2 = prob(dZ2t, B, H1t, B, L.H2, L.H1, B, EPI_GRAD);
            g2.g0 = grad + L.oW2;
            g2.ldg = L.H1;
            GemmProb b2 = prob(dZ2, L.H2, W(L.wW2t), L.H2, B, L.H1, L.H2, EPI_DTANH);
            b2.hsrc = H1t;
            b2.ldh = B;
            b2.outT = dZ1t;
            b2.ldt = B;
            if ((e = run_gemms(bf, ag, {g2, b2}, s)) != hipSuccess) return e;
        }
        // backward stage C: [dW1; dWc1] = [dZ1; dZc1]^T X
        {
            GemmProb g1 = prob(dZ1t, B, Xt, B, L.HC1, L.S, B, EPI_GRAD);
            g1.g0 = grad + L.oW1;
            g1.g1 = grad + L.oWc1;
            g1.gsplit = L.H1;
            g1.ldg = L.S;
            g1.gcols = L.S;
            if ((e = run_gemms(bf, ag, {g1}, s)) != hipSuccess) return e;
        }
        // the tail: Adam over the matrices; row sums of the bias, log-std
        // and critic-head gradients (each with its element's Adam step) and
        // of the statistics
        {
            RedBatch rb{};
            int rows = 0;
            auto add = [&](const void *src, int64_t ld, int nrows, int len, int isbf,
                           const float *w, int64_t pidx, double *dst64, double scale,
                           double addc) {
                RedSeg g{};
                g.pidx = pidx;
                float *dst = pidx >= 0 ? grad + pidx : nullptr;
                g.src = src;
                g.ld = ld;
                g.rows = nrows;
                g.len = len;
                g.bf = isbf;
                g.w = w;
                g.dst = dst;
                g.dst64 = dst64;
                g.scale = scale;
                g.add = addc;
                g.row0 = rows;
                const size_t esz = isbf ? 2 : 4;
                g.vec = (uintptr_t)src % 16 == 0 && (ld * (int64_t)esz) % 16 == 0 &&
                        ((int64_t)len * (int64_t)esz) % 16 == 0 && (!w || (uintptr_t)w % 16 == 0);
                rows += nrows;
                rb.s[rb.ns++] = g;
            };
            add(dZ1t, B, L.H1, B, bf, nullptr, L.ob1, nullptr, 1.0, 0.0);
            add(at(dZ1t, (size_t)L.H1 * B), B, L.C1, B, bf, nullptr, L.obc1, nullptr, 1.0, 0.0);
            add(dZ2t, B, L.H2, B, bf, nullptr, L.ob2, nullptr, 1.0, 0.0);
            add(dZc2t, B, L.C2, B, bf, nullptr, L.obc2, nullptr, 1.0, 0.0);
            add(dMUt, B, L.n, B, bf, nullptr, L.ob3, nullptr, 1.0, 0.0);
            add(LSt, B, L.n, B, 0, nullptr, L.ols, nullptr, 1.0, -(double)a.ent_coef);
            add(Hc2t, B, L.C2, B, bf, row_out + B, L.owc3, nullptr, 1.0, 0.0);
            add(row_out + B, B, 1, B, 0, nullptr, L.obc3, nullptr, 1.0, 0.0);
            if (a.stats) {
                double *st = a.stats + (size_t)u * 4;
                add(row_out + 2 * B, B, 1, B, 0, nullptr, -1, st + 0, -1.0 / B, 0.0);
                // the entropy from the log-std before this update's step
                add(row_out + 5 * B, 1, 1, 1, 0, nullptr, -1, st + 1, 1.0,
                    0.5 * (1.0 + (double)LN_2PI_F) * L.n);
                add(row_out + 3 * B, B, 1, B, 0, nullptr, -1, st + 2, 1.0 / B, 0.0);
                add(row_out + 4 * B, B, 1, B, 0, nullptr, -1, st + 3, 1.0 / B, 0.0);
            }
            rb.total_rows = rows;
            if ((e = tail(1, a.step0 + u, rb, u + 1 < a.n_updates ? u + 1 : -1)) != hipSuccess)
                return e;
        }
    }
    if (a.grad_out)   // [A][P] from the agents' workspaces
        return hipMemcpy2DAsync(a.grad_out, sizeof(float) * (size_t)L.P, grad,
                                (size_t)a.ws_stride, sizeof(float) * (size_t)L.P, (size_t)NA,
                                hipMemcpyDeviceToDevice, s);
    return hipSuccess;
}

}  // namespace tpk
