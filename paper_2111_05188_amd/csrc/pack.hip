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

// The same, with every value rounded to bf16 (kept in fp32 storage).
__global__ void pack_vec_bf16_kernel(const float *__restrict__ src, int cnt,
                                     int padded, float *__restrict__ dst)
{
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < padded;
         i += gridDim.x * blockDim.x)
        dst[i] = i < cnt ? (float)to_bf16(src[i]) : 0.0f;
}

// Transpose: element (k, o) of [K][out] is W[o][k] (rounded to bf16 if
// `bf16`), zero for k >= in.
__global__ void pack_transpose_kernel(const float *__restrict__ W, int out, int in,
                                      int K, int bf16, float *__restrict__ dst)
{
    const size_t total = (size_t)K * out;
    for (size_t p = blockIdx.x * (size_t)blockDim.x + threadIdx.x; p < total;
         p += (size_t)gridDim.x * blockDim.x) {
        const int o = (int)(p % out), k = (int)(p / out);
        const float w = k < in ? W[(size_t)o * in + k] : 0.0f;
        dst[p] = bf16 ? (float)to_bf16(w) : w;
    }
}

static int grid_for(size_t total)
{
    const size_t g = (total + 255) / 256;
    return (int)(g < 4096 ? (g > 0 ? g : 1) : 4096);
}

hipError_t launch_critic_pack(const tp_critic *c, const CriticLayout &L, void *dst,
                              hipStream_t s)
{
    const int outs[2] = {L.H1, L.H2}, ins[2] = {L.S, L.H1}, Ks[2] = {L.K_pad, L.H1};
    uint8_t *base = (uint8_t *)dst;
    for (int ag = 0; ag < c->n_agents; ++ag) {
        uint8_t *pa = base + (size_t)ag * L.agent_stride;
        for (int l = 0; l < 2; ++l) {
            const float *W = c->W[l] + (size_t)ag * (c->agent_stride ? (size_t)c->agent_stride
                                                                     : (size_t)outs[l] * ins[l]);
            if (L.mfma) {
                const size_t tot = (size_t)L.NT[l] * L.KS[l] * WAVE * 8;
                hipLaunchKernelGGL(pack_bf16_kernel, dim3(grid_for(tot)), dim3(256), 0, s, W,
                                   outs[l], ins[l], L.NT[l], L.KS[l], (__bf16 *)(pa + L.off_W[l]));
            } else {
                const size_t tot = (size_t)Ks[l] * outs[l];
                hipLaunchKernelGGL(pack_transpose_kernel, dim3(grid_for(tot)), dim3(256), 0, s, W,
                                   outs[l], ins[l], Ks[l], (int)(L.dtype == TP_BF16),
                                   (float *)(pa + L.off_W[l]));
            }
            hipLaunchKernelGGL(pack_vec_kernel, dim3(grid_for(outs[l])), dim3(256), 0, s,
                               c->b[l] + (size_t)ag * (c->agent_stride ? (size_t)c->agent_stride
                                                                       : (size_t)outs[l]),
                               outs[l], outs[l],
                               (float *)(pa + L.off_b[l]));
        }
        const float *w3 = c->W[2] + (size_t)ag * (c->agent_stride ? (size_t)c->agent_stride
                                                                  : (size_t)L.H2);
        if (L.dtype == TP_BF16)
            hipLaunchKernelGGL(pack_vec_bf16_kernel, dim3(grid_for(L.H2)), dim3(256), 0, s, w3,
                               L.H2, L.H2, (float *)(pa + L.off_W[2]));
        else
            hipLaunchKernelGGL(pack_vec_kernel, dim3(grid_for(L.H2)), dim3(256), 0, s, w3, L.H2,
                               L.H2, (float *)(pa + L.off_W[2]));
        hipLaunchKernelGGL(pack_vec_kernel, dim3(1), dim3(64), 0, s,
                           c->b[2] + (size_t)ag * (c->agent_stride ? (size_t)c->agent_stride : 1), 1, 1,
                           (float *)(pa + L.off_b[2]));
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
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
            const float *W = a->W[l] + (size_t)ag * (a->agent_stride ? (size_t)a->agent_stride
                                                                     : (size_t)outs[l] * ins[l]);
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
                               a->b[l] + (size_t)ag * (a->agent_stride ? (size_t)a->agent_stride
                                                                       : (size_t)outs[l]),
                               outs[l], padded,
                               (float *)(pa + L.off_b[l]));
        }
        const int lpad = L.dtype == TP_BF16 ? L.NT[2] * 16 : L.n;
        hipLaunchKernelGGL(pack_vec_kernel, dim3((lpad + 255) / 256), dim3(256), 0, s,
                           a->log_std + (size_t)ag * (a->agent_stride ? (size_t)a->agent_stride
                                                                      : (size_t)L.n),
                           L.n, lpad,
                           (float *)(pa + L.off_ls));
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace tpk
