// Actor parameter packing: fp32 masters -> the rollout kernel's layouts.
#include "device.hpp"
#include "internal.hpp"

namespace tpk {

// bf16 MFMA A-fragments: element (t, s, lane, e) of [NT][KS][64][8] is
// W[16t + lane%16][32s + 8(lane/16) + e], zero outside [out][in].
__global__ void pack_bf16_kernel(const float *__restrict__ W, int out, int in,
                                 int NT, int KS, __bf16 *__restrict__ dst)
{
    const size_t total = (size_t)NT * KS * WAVE * 8;
    for (size_t p = blockIdx.x * (size_t)blockDim.x + threadIdx.x; p < total;
         p += (size_t)gridDim.x * blockDim.x) {
        const int e = (int)(p % 8);
        const int lane = (int)((p / 8) % WAVE);
        const size_t ts = p / (8 * WAVE);
        const int s = (int)(ts % KS), t = (int)(ts / KS);
        const int o = 16 * t + (lane % 16), k = 32 * s + 8 * (lane / 16) + e;
        const float w = (o < out && k < in) ? W[(size_t)o * in + k] : 0.0f;
        dst[p] = to_bf16(w);
    }
}

// fp32 k-blocked transpose: element (k4, o, e) of [K4][out][4] is
// W[o][4 k4 + e], zero for k >= in.
__global__ void pack_f32_kernel(const float *__restrict__ W, int out, int in,
                                int K4, float *__restrict__ dst)
{
    const size_t total = (size_t)K4 * out * 4;
    for (size_t p = blockIdx.x * (size_t)blockDim.x + threadIdx.x; p < total;
         p += (size_t)gridDim.x * blockDim.x) {
        const int e = (int)(p % 4);
        const int o = (int)((p / 4) % out);
        const int k = (int)(p / (4 * (size_t)out)) * 4 + e;
        dst[p] = k < in ? W[(size_t)o * in + k] : 0.0f;
    }
}

// Copy `cnt` floats and zero-fill up to `padded`.
__global__ void pack_vec_kernel(const float *__restrict__ src, int cnt,
                                int padded, float *__restrict__ dst)
{
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < padded;
         i += gridDim.x * blockDim.x)
        dst[i] = i < cnt ? src[i] : 0.0f;
}

hipError_t launch_pack(const tp_actor *a, const PackedLayout &L, void *dst,
                       hipStream_t s)
{
    const int outs[3] = {L.H1, L.H2, L.n};
    const int ins[3] = {L.S, L.H1, L.H2};
    uint8_t *base = (uint8_t *)dst;
    for (int ag = 0; ag < a->n_agents; ++ag) {
        uint8_t *pa = base + (size_t)ag * L.agent_stride;
        for (int l = 0; l < 3; ++l) {
            const float *W = a->W[l] + (size_t)ag * outs[l] * ins[l];
            if (L.dtype == TP_BF16) {
                const size_t tot = (size_t)L.NT[l] * L.KS[l] * WAVE * 8;
                const int grid = (int)((tot + 255) / 256 < 4096 ? (tot + 255) / 256 : 4096);
                hipLaunchKernelGGL(pack_bf16_kernel, dim3(grid), dim3(256), 0, s, W, outs[l],
                                   ins[l], L.NT[l], L.KS[l], (__bf16 *)(pa + L.off_W[l]));
            } else {
                const size_t tot = (size_t)L.KS[l] * outs[l] * 4;
                const int grid = (int)((tot + 255) / 256 < 4096 ? (tot + 255) / 256 : 4096);
                hipLaunchKernelGGL(pack_f32_kernel, dim3(grid), dim3(256), 0, s, W, outs[l],
                                   ins[l], L.KS[l], (float *)(pa + L.off_W[l]));
            }
            const int padded = L.dtype == TP_BF16 ? L.NT[l] * 16 : outs[l];
            hipLaunchKernelGGL(pack_vec_kernel, dim3((padded + 255) / 256), dim3(256), 0, s,
                               a->b[l] + (size_t)ag * outs[l], outs[l], padded,
                               (float *)(pa + L.off_b[l]));
        }
        const int lpad = L.dtype == TP_BF16 ? L.NT[2] * 16 : L.n;
        hipLaunchKernelGGL(pack_vec_kernel, dim3((lpad + 255) / 256), dim3(256), 0, s,
                           a->log_std + (size_t)ag * L.n, L.n, lpad,
                           (float *)(pa + L.off_ls));
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace tpk
