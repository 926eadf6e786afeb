// Internal interface between the C-ABI layer (api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "tp.h"

namespace tpk {

// MDP constants as the kernels use them (fees folded into the two factors
// f_s = 1 - fee and f_b = 1 + fee, each rounded once to fp64).
struct EnvConst {
    const float *price;   // [T1][n]
    const float *ind;     // [T1][nI]
    int64_t T1;
    int n;
    int nI;               // n * n_ind
    int K_pad;            // observation row length (multiple of 32)
    int hmax;
    int horizon;
    double f_s, f_b;
    double reward_scale;
    double cash0;
    float cash_scale, price_scale, share_scale;
};

// Byte layout of one agent's packed parameters inside the packed buffer.
//  bf16: W_l as MFMA A-fragments, [NT][KS][64 lanes][8 bf16]; lane l of the
//        block (tile t, k-step s) holds W[16t + l%16][32s + 8(l/16) + 0..7].
//  f32 : W_l as k-blocked transposes, [in_pad/4][out][4]: entry
//        (k4, o, e) = W[o][4 k4 + e].
//  Biases fp32 [out padded to whole tiles]; log_std fp32 [NT3 * 16].
struct PackedLayout {
    int dtype;
    int S, H1, H2, n;
    int K_pad;
    int NT[3];            // output tiles of 16 (bf16)
    int KS[3];            // k-steps of 32 (bf16) / k-blocks of 4 (f32)
    size_t off_W[3], off_b[3], off_ls;
    size_t agent_stride;
    size_t total;
};

bool packed_layout(const tp_actor *a, PackedLayout *out);

struct RolloutArgs {
    EnvConst env;
    double *cash;
    int32_t *shares;
    int64_t *t;
    int E;
    const uint8_t *packed;
    PackedLayout lay;
    int n_agents, envs_per_agent, blocks_per_agent;
    uint32_t key_lo, key_hi;
    uint64_t step0;
    int L;
    void *obs;
    int64_t ld_obs;
    float *action;
    float *logp;
    float *reward;
    uint8_t *done;
    double *cash_tap;
    int32_t *shares_tap;
    void *obs_last;
    double *asset_tap;
    float *mu_tap;
    int32_t *n_invalid;   // count of envs not stepped (zeroed before the launch), or NULL
    // LDS carve-up (bytes / elements), filled by the launcher
    int ldx, ldh, ldmu, ldz, ldh2;
    size_t lds_X, lds_H, lds_MU, lds_OS, lds_PT, lds_scal, lds_Z, lds_B, lds_bytes;
};

hipError_t launch_rollout(RolloutArgs &a, hipStream_t s);
hipError_t launch_rollout_rs(RolloutArgs &a, hipStream_t s);
// the role-split kernel's shapes (it also needs 16-byte aligned market,
// action and holdings-tap buffers)
bool rollout_rs_shape(const PackedLayout &P, int nI);
hipError_t launch_env_reset(const EnvConst &c, double *cash, int32_t *shares,
                            int64_t *t, const int64_t *t0, int E, void *obs,
                            int64_t ld_obs, int obs_bf16, int32_t *n_invalid,
                            hipStream_t s);
hipError_t launch_env_step(const EnvConst &c, double *cash, int32_t *shares,
                           int64_t *t, const float *action, float *reward,
                           int E, void *obs, int64_t ld_obs, int obs_bf16,
                           int32_t *n_invalid, hipStream_t s);
// *p = 0 by a one-thread kernel (a fill kernel rather than a memset node, so
// the call sequence stays safe to capture in a graph)
hipError_t launch_zero_i32(int32_t *p, hipStream_t s);
// the env step's LDS observation rows for this market fit the device
bool env_rows_fit(const EnvConst &c, int obs_bf16);
size_t backtest_metrics_work_bytes(int T, int E);
// the no-allocation variant: bytes of scratch the call needs (0 on the
// one-launch path), the static scratch's size, and its device address on
// the current device
size_t backtest_metrics_scratch_needed(int T, int E);
size_t backtest_metrics_scratch_capacity();
hipError_t backtest_metrics_scratch(void **ptr);
hipError_t launch_backtest_metrics(const double *v0, const double *v, int T, int E,
                                   double periods_per_year, double risk_free, double *out,
                                   void *work, hipStream_t s);
hipError_t launch_ensemble_fuse(float *params, int N, int K, int64_t P, hipStream_t s);
hipError_t launch_fitness(const float *r, int L, int E, int A, double gamma, double *fit,
                          double *env_return, hipStream_t s);
hipError_t launch_keep_best(const double *fit, double *best, int32_t *stall, const float *params,
                            float *best_params, int A, int64_t P, hipStream_t s);
hipError_t launch_select(const double *fit, float *params, int N, int64_t P, int keep,
                         int32_t *rank, hipStream_t s);
hipError_t launch_gae(const float *r, const float *v, const uint8_t *d, int L,
                      int E, double g, double gl, float *adv, float *ret,
                      hipStream_t s);
hipError_t launch_pack(const tp_actor *a, const PackedLayout &lay, void *dst,
                       hipStream_t s);

// Byte layout of one agent's packed critic inside the packed buffer.
//  mfma (bf16, H1 == H2 in {512, 1024}, K_pad % 128 == 0): W1, W2 as MFMA
//       A-fragments [NT][KS][64 lanes][8 bf16] (as the actor's);
//  otherwise: W1T [K_pad][H1] and W2T [H1][H2] fp32 transposes (values
//       rounded to bf16 for a bf16 critic), zero rows for k >= S.
//  Then w3 [H2] fp32 (rounded to bf16 for a bf16 critic), b1 [H1],
//  b2 [H2], b3 [1] fp32.
struct CriticLayout {
    int dtype;
    int S, H1, H2, K_pad;
    bool mfma;
    int NT[2], KS[2];     // fragment tiles and k-steps of layers 1 and 2
    size_t off_W[3], off_b[3];
    size_t agent_stride;
    size_t total;
};

bool critic_mfma_shape(const CriticLayout &L);
bool critic_layout(const tp_critic *c, CriticLayout *out);

struct CriticArgs {
    const uint8_t *packed;
    CriticLayout lay;
    const void *obs;
    int64_t ld_obs;
    int64_t T;
    int E, n_agents, envs_per_agent;
    float *value;
};

hipError_t launch_critic_value(const CriticArgs &a, hipStream_t s);
hipError_t launch_critic_pack(const tp_critic *c, const CriticLayout &lay, void *dst,
                              hipStream_t s);

// PPO learner: flat parameter offsets (floats) and workspace carve-up
// (bytes, 256-byte aligned areas).  Kp = S rounded up to 32, n_pad = n
// rounded up to 32, HC1 = H1 + C1 (the concatenated first layers).
struct PpoLayout {
    int dtype;
    int S, H1, H2, n, C1, C2, B;
    int Kp, n_pad, HC1;
    int64_t oW1, ob1, oW2, ob2, oW3, ob3, ols, oWc1, obc1, oWc2, obc2, owc3, obc3, P;
    size_t wWcat1, wW2, wW2t, wWc2, wWc2t, wW3, wW3t;
    size_t wX, wXt, wH1, wH1t, wH2, wH2t, wHc2, wHc2t;
    size_t wMU, wAg, wRowIn, wRowOut, wdMU, wdMUt, wLSt, wdZc2, wdZc2t, wdZ2, wdZ2t, wdZ1t;
    size_t wG;
    size_t total;
};

bool ppo_layout(const tp_ppo *c, PpoLayout *out);

struct PpoArgs {
    PpoLayout lay;
    int n_agents;              // independent learners in one call
    int64_t agent_stride;      // floats between agents' parameters (and moments)
    int64_t ws_stride;         // bytes between agents' workspaces
    float *params, *adam_m, *adam_v;
    int64_t step0;
    int n_updates;
    const void *obs;
    int64_t ld_obs;
    const float *action, *logp, *adv, *ret;
    int64_t rows;
    const int64_t *idx;
    float *grad_out;
    double *stats;
    void *workspace;
    float clip, ent_coef, lr, beta1, beta2, eps;
};

hipError_t launch_ppo_update(const PpoArgs &a, hipStream_t s);
hipError_t launch_minibatch_rows(uint64_t seed, uint64_t counter, int n_updates, int B, int L,
                                 int E, int agent, int epa, int64_t *idx, hipStream_t s);

// Maximum LDS per workgroup on gfx950.
constexpr size_t LDS_LIMIT = 160 * 1024;

}  // namespace tpk
