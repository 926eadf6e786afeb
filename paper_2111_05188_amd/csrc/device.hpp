// Device helpers for gfx950: Philox4x32-10, Box-Muller, bf16 rounding,
// 64-lane wavefront reductions and scans.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tpk {

constexpr int WAVE = 64;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11).  Ten rounds; each round
// multiplies counter words 0 and 2 by the two Philox multipliers, and the new
// counter is (hi(M1*c2)^c1^k0, lo(M1*c2), hi(M0*c0)^c3^k1, lo(M0*c0)).  The
// key is bumped by the two Weyl increments before every round but the first.
// ---------------------------------------------------------------------------
struct U4 {
    uint32_t x, y, z, w;
};

__device__ __forceinline__ U4 philox4x32_10(U4 c, uint32_t k0, uint32_t k1)
{
    constexpr uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
    constexpr uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r > 0) {
            k0 += W0;
            k1 += W1;
        }
        const uint32_t hi0 = __umulhi(M0, c.x), lo0 = M0 * c.x;
        const uint32_t hi1 = __umulhi(M1, c.z), lo1 = M1 * c.z;
        c = U4{hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0};
    }
    return c;
}

// Top 23 bits, centred in their cell: exact in fp32, strictly inside (0,1).
__device__ __forceinline__ float uniform_open01(uint32_t w)
{
    return ((float)(w >> 9) + 0.5f) * (1.0f / 8388608.0f);
}

// Box & Muller (1958): two independent N(0,1) draws from two uniforms.
__device__ __forceinline__ void box_muller(float u0, float u1, float &z0,
                                           float &z1)
{
    const float rad = sqrtf(-2.0f * logf(u0));
    const float ang = 6.28318530717958647692f * u1;
    z0 = rad * cosf(ang);
    z1 = rad * sinf(ang);
}

// ---------------------------------------------------------------------------
// Wavefront collectives (all 64 lanes active).
// ---------------------------------------------------------------------------
__device__ __forceinline__ double wave_sum(double v)
{
#pragma unroll
    for (int o = WAVE / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
    return v;
}

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int o = WAVE / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
    return v;
}

// Inclusive prefix sum across lanes in lane order.
__device__ __forceinline__ double wave_inclusive_scan(double v, int lane)
{
#pragma unroll
    for (int o = 1; o < WAVE; o <<= 1) {
        const double t = __shfl_up(v, o, WAVE);
        if (lane >= o) v += t;
    }
    return v;
}

// fp32 -> bf16, IEEE round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ __bf16 to_bf16(float x) { return (__bf16)x; }

}  // namespace tpk
