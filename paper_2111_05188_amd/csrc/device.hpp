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

// The same with the hardware transcendentals: v_log_f32 (log2), v_sqrt_f32,
// and v_sin_f32 / v_cos_f32, whose argument is in revolutions, so the
// uniform u1 is the angle / 2 pi as it stands.  Close to fp32 precision, not
// correctly rounded: used where the draws feed a bf16 actor, whose
// tolerance is far wider.
__device__ __forceinline__ void box_muller_hw(float u0, float u1, float &z0, float &z1)
{
    // -2 ln u0 = -2 ln(2) log2(u0)
    const float rad = __builtin_amdgcn_sqrtf(-1.38629436111989061f * __builtin_amdgcn_logf(u0));
    z0 = rad * __builtin_amdgcn_cosf(u1);
    z1 = rad * __builtin_amdgcn_sinf(u1);
}

// ---------------------------------------------------------------------------
// Wavefront collectives (all 64 lanes active), built on DPP lane moves:
// row_shr:k shifts within 16-lane rows, row_bcast:15 / row_bcast:31 carry
// row totals into the following rows.  A lane whose DPP source does not
// exist (or whose row is masked off) receives 0.
// ---------------------------------------------------------------------------
enum : int { DPP_ROW_SHR = 0x110, DPP_ROW_BCAST15 = 0x142, DPP_ROW_BCAST31 = 0x143 };

template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ double dpp_f64(double x)
{
    const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(x), CTRL, ROWS, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(x), CTRL, ROWS, 0xF, false);
    return __hiloint2double(hi, lo);
}

// Inclusive prefix sum across the 64 lanes in lane order (Hillis-Steele in
// rows of 16, then row totals carried forward).
__device__ __forceinline__ double wave_inclusive_scan(double v)
{
    v += dpp_f64<DPP_ROW_SHR + 1>(v);
    v += dpp_f64<DPP_ROW_SHR + 2>(v);
    v += dpp_f64<DPP_ROW_SHR + 4>(v);
    v += dpp_f64<DPP_ROW_SHR + 8>(v);
    v += dpp_f64<DPP_ROW_BCAST15, 0xA>(v);
    v += dpp_f64<DPP_ROW_BCAST31, 0xC>(v);
    return v;
}

__device__ __forceinline__ double lane_value(double v, int lane)
{
    const int lo = __builtin_amdgcn_readlane(__double2loint(v), lane);
    const int hi = __builtin_amdgcn_readlane(__double2hiint(v), lane);
    return __hiloint2double(hi, lo);
}

__device__ __forceinline__ int lane_value(int v, int lane)
{
    return __builtin_amdgcn_readlane(v, lane);
}

__device__ __forceinline__ float lane_value(float v, int lane)
{
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// Sum over the 64 lanes (same value returned to every lane).
__device__ __forceinline__ double wave_sum(double v)
{
    return lane_value(wave_inclusive_scan(v), WAVE - 1);
}

// fp32 -> bf16, IEEE round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ __bf16 to_bf16(float x) { return (__bf16)x; }

// tanh(x) = 2 / (1 + exp(-2x)) - 1 with the hardware exp2 and reciprocal;
// the argument comes in as e2 = -2 log2(e) x (one fma with a pre-scaled
// bias).  Absolute error of a few 1e-7 (cancellation near 0 leaves the fp32
// rounding of 1), far below the bf16 rounding the result goes through.
constexpr float NEG_2LOG2E = -2.8853900817779268f;

__device__ __forceinline__ float tanh_from_e2(float e2)
{
    return fmaf(2.0f, __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(e2)), -1.0f);
}

}  // namespace tpk
