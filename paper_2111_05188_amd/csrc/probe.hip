// Hardware probes for the roofline ceilings the design notes quote
// (measurement tooling, built as libtpprobe.so; not part of the method):
//   * tpp_mfma_sweep: the same issue rates over accumulators per wave
//     (1-8), operands shared or one pair per accumulator, and waves per
//     workgroup, with the shader clock the loop ran at;
//   * tpp_mfma_issue / tpp_mfma32_issue: waves issuing
//     v_mfma_f32_16x16x32_bf16 (eight independent accumulators per wave) or
//     v_mfma_f32_32x32x16_bf16 (four) back to back on register operands:
//     the achievable dense bf16 MFMA rate of each instruction;
//   * tpp_l2_stream: every workgroup streams the same L2-resident buffer in
//     the pattern of the rollout's weight stream (a wave instruction reads
//     1 KiB: lane l the 16 bytes at 16 l), 16 loads in flight per wave: the
//     L2 -> CU bandwidth one CU can pull.
//   * tpp_copy: a plain device copy, 16 bytes per lane, four loads in flight
//     per lane, non-temporal: the HBM rate a streaming kernel can reach.
// The first two write to `out` only under a condition the data never meets,
// so the results stay live without memory traffic.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tp_probe.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int NACC = 8;

__global__ __launch_bounds__(256) void mfma_issue_kernel(int iters, float *out)
{
    const int lane = threadIdx.x % 64;
    bf16x8 a, b;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        a[e] = (__bf16)(0.001f * (float)(lane + e));
        b[e] = (__bf16)(0.002f * (float)(lane - e));
    }
    floatx4 acc[NACC];
#pragma unroll
    for (int j = 0; j < NACC; ++j) acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int j = 0; j < NACC; ++j)
            acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[j], 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < NACC; ++j) s += acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
    if (s == 1234567.0f) out[blockIdx.x * 256 + threadIdx.x] = s;
}

typedef float floatx16 __attribute__((ext_vector_type(16)));

// the same with v_mfma_f32_32x32x16_bf16 (four independent accumulators)
__global__ __launch_bounds__(256) void mfma32_issue_kernel(int iters, float *out)
{
    const int lane = threadIdx.x % 64;
    bf16x8 a, b;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        a[e] = (__bf16)(0.001f * (float)(lane + e));
        b[e] = (__bf16)(0.002f * (float)(lane - e));
    }
    floatx16 acc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[j][q] = 0.f;
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int q = 0; q < 16; ++q) s += acc[j][q];
    if (s == 1234567.0f) out[blockIdx.x * 256 + threadIdx.x] = s;
}

// The issue-rate sweep: NACC independent accumulators per wave, each with
// its own A and B operand registers (DISTINCT) or all sharing one pair, on
// v_mfma_f32_16x16x32_bf16 (M = 16) or v_mfma_f32_32x32x16_bf16 (M = 32).
// Wave 0 of workgroup 0 also records the shader clock (s_memtime) and the
// constant 100 MHz clock (s_memrealtime) around its loop, so the host can
// tell the clock the MFMAs ran at.
template <int M, int NACC, bool DISTINCT>
__global__ __launch_bounds__(256) void mfma_sweep_kernel(int iters, float *out,
                                                          unsigned long long *clk)
{
    constexpr int NA = DISTINCT ? NACC : 1;
    constexpr int NV = M == 16 ? 4 : 16;
    typedef float accv __attribute__((ext_vector_type(NV)));
    const int lane = threadIdx.x % 64;
    bf16x8 a[NA], b[NA];
#pragma unroll
    for (int j = 0; j < NA; ++j)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            a[j][e] = (__bf16)(0.001f * (float)(lane + e + j));
            b[j][e] = (__bf16)(0.002f * (float)(lane - e - j));
        }
    accv acc[NACC];
#pragma unroll
    for (int j = 0; j < NACC; ++j)
#pragma unroll
        for (int q = 0; q < NV; ++q) acc[j][q] = 0.f;
    const unsigned long long c0 = clock64(), w0 = wall_clock64();
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int j = 0; j < NACC; ++j) {
            if constexpr (M == 16)
                acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[DISTINCT ? j : 0],
                                                                 b[DISTINCT ? j : 0], acc[j], 0, 0, 0);
            else
                acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[DISTINCT ? j : 0],
                                                                 b[DISTINCT ? j : 0], acc[j], 0, 0, 0);
        }
    }
    const unsigned long long c1 = clock64(), w1 = wall_clock64();
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < NACC; ++j)
#pragma unroll
        for (int q = 0; q < NV; ++q) s += acc[j][q];
    if (s == 1234567.0f) out[blockIdx.x * blockDim.x + threadIdx.x] = s;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        clk[0] = c1 - c0;
        clk[1] = w1 - w0;
    }
}

template <int M, int NACC, bool D>
hipError_t launch_sweep(int blocks, int waves, int iters, float *out, unsigned long long *clk,
                        hipStream_t st)
{
    hipLaunchKernelGGL((mfma_sweep_kernel<M, NACC, D>), dim3(blocks), dim3(64 * waves), 0, st,
                       iters, out, clk);
    return hipGetLastError();
}

template <int M, bool D>
hipError_t sweep_nacc(int nacc, int blocks, int waves, int iters, float *out,
                      unsigned long long *clk, hipStream_t st)
{
    switch (nacc) {
    case 1: return launch_sweep<M, 1, D>(blocks, waves, iters, out, clk, st);
    case 2: return launch_sweep<M, 2, D>(blocks, waves, iters, out, clk, st);
    case 4: return launch_sweep<M, 4, D>(blocks, waves, iters, out, clk, st);
    case 8: return launch_sweep<M, 8, D>(blocks, waves, iters, out, clk, st);
    default: return hipErrorInvalidValue;
    }
}

// Workgroup-to-workgroup handoff: workgroup b (of 2 * pairs, one wave
// each) and its partner b ^ stride pass a counter back and forth `rounds`
// times through one flag word, with agent-scope release stores and acquire
// loads (mode 0) or relaxed agent-scope atomics (mode 1).  Every wait is
// bounded by spin_limit polls; a wait that runs out sets out[b].timeouts and
// the workgroup leaves its loop, so every wave exits.  out[b]: the XCD the
// workgroup ran on (hardware register XCC_ID), the 100 MHz ticks of its
// loop, the timeouts.
struct PingOut {
    unsigned int xcc, timeouts;
    unsigned long long ticks;
};

__device__ __forceinline__ unsigned int xcc_id()
{
    // HW_REG_XCC_ID (20), bits [3:0]
    return __builtin_amdgcn_s_getreg((20) | (0 << 6) | ((4 - 1) << 11));
}

__global__ __launch_bounds__(64) void pingpong_kernel(int mode, int stride, int rounds,
                                                      int spin_limit, int *flags, PingOut *out)
{
    const int b = blockIdx.x;
    const int partner = b ^ stride;
    const bool ping = b < partner;
    // pair index in [0, pairs): b = q (2 stride) + r, r < 2 stride
    const int pair = (b / (2 * stride)) * stride + (b % stride);
    int *flag = flags + pair * 32;   // one 128-byte line per pair
    unsigned int timeouts = 0;
    const unsigned long long w0 = wall_clock64();
    if (threadIdx.x == 0) {
        for (int r = 0; r < rounds && timeouts == 0; ++r) {
            const int want = ping ? 2 * r : 2 * r + 1;   // value that lets this side go
            int spins = 0;
            for (;;) {
                const int v = mode == 0
                                  ? __hip_atomic_load(flag, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT)
                                  : __hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (v >= want) break;
                if (++spins >= spin_limit) {
                    ++timeouts;
                    break;
                }
            }
            if (timeouts) break;
            if (mode == 0)
                __hip_atomic_store(flag, want + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
            else
                __hip_atomic_store(flag, want + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        const unsigned long long w1 = wall_clock64();
        out[b].xcc = xcc_id();
        out[b].timeouts = timeouts;
        out[b].ticks = w1 - w0;
    }
}

// The same handoff carrying a payload: each side, on its turn, writes
// PW 16-byte words (round-dependent values) to its half of the pair's data
// block, then raises the flag (relaxed agent-scope atomic store, after all
// its stores have completed); the other side, once it sees the flag, reads
// the payload and counts words that differ from what was written (stale
// data).  Cache policy of the payload accesses: mode 0 plain stores and
// loads that bypass the CU's L1 (sc0; the L2 of one XCD is shared by its
// CUs), mode 1 stores and loads at device scope (sc1).  data: pairs * 2 *
// PW 16-byte words.  out as for pingpong_kernel, plus the mismatch count.
constexpr int PW = 1024;

struct PingDataOut {
    unsigned int xcc, timeouts;
    unsigned long long ticks;
    unsigned int mismatches, pad;
};

__global__ __launch_bounds__(64) void pingpong_data_kernel(int mode, int stride, int rounds,
                                                           int spin_limit, int *flags,
                                                           uint32_t *data, PingDataOut *out)
{
    typedef uint32_t v4 __attribute__((ext_vector_type(4)));
    const int b = blockIdx.x, lane = threadIdx.x;
    const int partner = b ^ stride;
    const bool ping = b < partner;
    const int pair = (b / (2 * stride)) * stride + (b % stride);
    int *flag = flags + pair * 32;
    // this side writes its own half, reads the partner's
    uint32_t *base = data + (size_t)pair * 2 * PW * 4;
    const __amdgpu_buffer_rsrc_t mine = __builtin_amdgcn_make_buffer_rsrc(
        base + (ping ? 0 : PW * 4), (short)0, PW * 16, 0x00020000);
    const __amdgpu_buffer_rsrc_t theirs = __builtin_amdgcn_make_buffer_rsrc(
        base + (ping ? PW * 4 : 0), (short)0, PW * 16, 0x00020000);
    unsigned int timeouts = 0, bad = 0;
    const unsigned long long w0 = wall_clock64();
    for (int r = 0; r < rounds && timeouts == 0; ++r) {
        const int want = ping ? 2 * r : 2 * r + 1;
        if (want > 0) {
            // wait for the partner's turn, then read its payload of value want - 1
            int spins = 0, v = 0;
            for (;;) {
                if (lane == 0) v = __hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                v = __shfl(v, 0);
                if (v >= want) break;
                if (++spins >= spin_limit) {
                    ++timeouts;
                    break;
                }
            }
            if (timeouts) break;
            const uint32_t expect = (uint32_t)(want - 1);
#pragma unroll 4
            for (int k = 0; k < PW / 64; ++k) {
                const int w = lane + 64 * k;
                const v4 x = mode == 0 ? __builtin_amdgcn_raw_buffer_load_b128(theirs, w * 16, 0, 1)
                                       : __builtin_amdgcn_raw_buffer_load_b128(theirs, w * 16, 0, 16);
                bad += (x.x != expect * 4096u + (uint32_t)w) + (x.w != expect);
            }
        }
        // this side's payload for value `want`
#pragma unroll 4
        for (int k = 0; k < PW / 64; ++k) {
            const int w = lane + 64 * k;
            const v4 x = {(uint32_t)want * 4096u + (uint32_t)w, 1u, 2u, (uint32_t)want};
            if (mode == 0)
                __builtin_amdgcn_raw_buffer_store_b128(x, mine, w * 16, 0, 0);
            else
                __builtin_amdgcn_raw_buffer_store_b128(x, mine, w * 16, 0, 16);
        }
        __builtin_amdgcn_s_waitcnt(0);   // every store of this wave has completed
        if (lane == 0) __hip_atomic_store(flag, want + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    const unsigned long long w1 = wall_clock64();
    // lane totals of stale words
    for (int o = 32; o >= 1; o >>= 1) bad += __shfl_xor(bad, o);
    if (lane == 0) {
        out[b].xcc = __builtin_amdgcn_s_getreg((20) | (0 << 6) | ((4 - 1) << 11));
        out[b].timeouts = timeouts;
        out[b].ticks = w1 - w0;
        out[b].mismatches = bad;
    }
}

// The rollout's weight stream (1 KiB per wave instruction, 16 loads in
// flight) from an L2-resident buffer, with an agent-scope acquire fence
// (mode 1) or release fence (mode 2) every `every` fragments, or none
// (mode 0): what such fences cost a concurrent weight stream.
__global__ __launch_bounds__(512) void l2_stream_fence_kernel(const uint32_t *__restrict__ buf,
                                                              int frags_per_wave, int reps,
                                                              int mode, int every, uint32_t *out)
{
    typedef uint32_t v4 __attribute__((ext_vector_type(4)));
    const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
    const v4 *p = (const v4 *)buf + (size_t)wave * frags_per_wave * 64 + lane;
    v4 acc = {0u, 0u, 0u, 0u};
    constexpr int D = 16;
    for (int r = 0; r < reps; ++r) {
        v4 b[D];
#pragma unroll
        for (int d = 0; d < D; ++d) b[d] = p[(size_t)(d % frags_per_wave) * 64];
        for (int f0 = 0; f0 < frags_per_wave; f0 += D) {
#pragma unroll
            for (int d = 0; d < D; ++d) {
                acc ^= b[d];
                int nf = f0 + d + D;
                while (nf >= frags_per_wave) nf -= frags_per_wave;
                b[d] = p[(size_t)nf * 64];
                if ((f0 + d) % every == 0) {
                    if (mode == 1) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
                    if (mode == 2) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
#pragma unroll
        for (int d = 0; d < D; ++d) acc ^= b[d];
    }
    if (acc.x == 0x12345678u && acc.y == 0x9abcdef0u) ((v4 *)out)[blockIdx.x * 512 + threadIdx.x] = acc;
}

constexpr int SD = 16;   // loads in flight per wave

__global__ __launch_bounds__(512) void l2_stream_kernel(const u32x4 *__restrict__ buf,
                                                        int frags_per_wave, int reps,
                                                        u32x4 *out)
{
    const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
    const u32x4 *p = buf + (size_t)wave * frags_per_wave * 64 + lane;
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (int r = 0; r < reps; ++r) {
        u32x4 b[SD];
#pragma unroll
        for (int d = 0; d < SD; ++d) b[d] = p[(size_t)(d % frags_per_wave) * 64];
        for (int f0 = 0; f0 < frags_per_wave; f0 += SD) {
#pragma unroll
            for (int d = 0; d < SD; ++d) {
                acc ^= b[d];
                int nf = f0 + d + SD;
                while (nf >= frags_per_wave) nf -= frags_per_wave;
                b[d] = p[(size_t)nf * 64];
                __builtin_amdgcn_sched_barrier(0);
            }
        }
#pragma unroll
        for (int d = 0; d < SD; ++d) acc ^= b[d];
    }
    if (acc.x == 0x12345678u && acc.y == 0x9abcdef0u) out[blockIdx.x * 512 + threadIdx.x] = acc;
}


__global__ __launch_bounds__(256) void copy_kernel(const u32x4 *__restrict__ src,
                                                   u32x4 *__restrict__ dst, size_t n)
{
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (; i + 3 * stride < n; i += 4 * stride) {
        u32x4 v[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) v[k] = __builtin_nontemporal_load(src + i + k * stride);
#pragma unroll
        for (int k = 0; k < 4; ++k) __builtin_nontemporal_store(v[k], dst + i + k * stride);
    }
    for (; i < n; i += stride) __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

}  // namespace

extern "C" {

int tpp_mfma_issue(int blocks, int iters, float *out, void *stream)
{
    if (blocks < 1 || iters < 1 || !out) return -1;
    hipLaunchKernelGGL(mfma_issue_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream, iters,
                       out);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

double tpp_mfma_issue_flops(int blocks, int iters)
{
    return (double)blocks * 4.0 * iters * NACC * (2.0 * 16 * 16 * 32);
}

int tpp_mfma32_issue(int blocks, int iters, float *out, void *stream)
{
    if (blocks < 1 || iters < 1 || !out) return -1;
    hipLaunchKernelGGL(mfma32_issue_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream,
                       iters, out);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

double tpp_mfma32_issue_flops(int blocks, int iters)
{
    return (double)blocks * 4.0 * iters * 4 * (2.0 * 32 * 32 * 16);
}

int tpp_mfma_sweep(int m, int nacc, int distinct, int blocks, int waves, int iters, float *out,
                   unsigned long long *clk, void *stream)
{
    if ((m != 16 && m != 32) || !(nacc == 1 || nacc == 2 || nacc == 4 || nacc == 8) ||
        blocks < 1 || waves < 1 || waves > 4 || iters < 1 || !out || !clk)
        return -1;
    const hipStream_t st = (hipStream_t)stream;
    hipError_t e;
    if (m == 16)
        e = distinct ? sweep_nacc<16, true>(nacc, blocks, waves, iters, out, clk, st)
                     : sweep_nacc<16, false>(nacc, blocks, waves, iters, out, clk, st);
    else
        e = distinct ? sweep_nacc<32, true>(nacc, blocks, waves, iters, out, clk, st)
                     : sweep_nacc<32, false>(nacc, blocks, waves, iters, out, clk, st);
    return e == hipSuccess ? 0 : -4;
}

double tpp_mfma_sweep_flops(int m, int nacc, int blocks, int waves, int iters)
{
    const double per = m == 16 ? 2.0 * 16 * 16 * 32 : 2.0 * 32 * 32 * 16;
    return (double)blocks * waves * iters * nacc * per;
}

int tpp_l2_stream(const void *buf, size_t buf_bytes, int frags_per_wave, int reps, int blocks,
                  void *out, void *stream)
{
    if (!buf || !out || frags_per_wave < 1 || reps < 1 || blocks < 1) return -1;
    if ((size_t)8 * frags_per_wave * 1024 > buf_bytes) return -1;
    hipLaunchKernelGGL(l2_stream_kernel, dim3(blocks), dim3(512), 0, (hipStream_t)stream,
                       (const u32x4 *)buf, frags_per_wave, reps, (u32x4 *)out);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

int tpp_pingpong(int mode, int pairs, int stride, int rounds, int spin_limit, int *flags,
                 void *out, void *stream)
{
    // 2 * pairs workgroups; partners b and b ^ stride (stride a power of two
    // below 2 * pairs); flags: pairs * 32 ints, zeroed by the caller
    if ((mode != 0 && mode != 1) || pairs < 1 || stride < 1 || (stride & (stride - 1)) ||
        stride >= 2 * pairs || (2 * pairs) % (2 * stride) || rounds < 1 || spin_limit < 1 ||
        !flags || !out)
        return -1;
    hipLaunchKernelGGL(pingpong_kernel, dim3(2 * pairs), dim3(64), 0, (hipStream_t)stream, mode,
                       stride, rounds, spin_limit, flags, (PingOut *)out);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

int tpp_pingpong_data(int mode, int pairs, int stride, int rounds, int spin_limit, int *flags,
                      void *data, void *out, void *stream)
{
    // flags: pairs * 32 ints (zeroed); data: pairs * 2 * 1024 16-byte words;
    // out: 2 * pairs records of 24 bytes
    if ((mode != 0 && mode != 1) || pairs < 1 || stride < 1 || (stride & (stride - 1)) ||
        stride >= 2 * pairs || (2 * pairs) % (2 * stride) || rounds < 1 || spin_limit < 1 ||
        !flags || !data || !out)
        return -1;
    hipLaunchKernelGGL(pingpong_data_kernel, dim3(2 * pairs), dim3(64), 0, (hipStream_t)stream,
                       mode, stride, rounds, spin_limit, flags, (uint32_t *)data,
                       (PingDataOut *)out);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

int tpp_l2_stream_fence(const void *buf, size_t buf_bytes, int frags_per_wave, int reps,
                        int blocks, int mode, int every, void *out, void *stream)
{
    if (!buf || !out || frags_per_wave < 1 || reps < 1 || blocks < 1 || mode < 0 || mode > 2 ||
        every < 1)
        return -1;
    if ((size_t)8 * frags_per_wave * 1024 > buf_bytes) return -1;
    hipLaunchKernelGGL(l2_stream_fence_kernel, dim3(blocks), dim3(512), 0, (hipStream_t)stream,
                       (const uint32_t *)buf, frags_per_wave, reps, mode, every, (uint32_t *)out);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

int tpp_copy(const void *src, void *dst, size_t bytes, int blocks, void *stream)
{
    if (!src || !dst || bytes % 16 || blocks < 1 || (uintptr_t)src % 16 || (uintptr_t)dst % 16)
        return -1;
    hipLaunchKernelGGL(copy_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream,
                       (const u32x4 *)src, (u32x4 *)dst, bytes / 16);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // extern "C"
