/*
 * tp.h -- C ABI of the MI355X (gfx950) rollout library for the
 * FinRL-Podracer stock-trading hot path (arXiv 2111.05188).
 *
 * The library steps thousands of copies of the paper's stock-trading MDP in
 * lockstep on one GPU (the batched environment of Section 4.4, "Market
 * simulation with GPU-acceleration"), runs the actor MLP that picks every
 * env's action, samples Gaussian actions from a counter-based Philox
 * stream, records the trajectories in GPU memory (Section 4.4, "Replay
 * buffer on GPU") and computes GAE advantages and returns over them.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every pointer is a DEVICE pointer owned by the caller, unless its
 *    comment says "host".  The library never frees or retains caller
 *    memory past the call.
 *  - Every call only enqueues work on `stream` (a hipStream_t passed as
 *    void*; NULL = the null stream) and returns without synchronising.
 *  - Return value: TP_OK (0) or a negative tp_status.  On a negative return
 *    nothing was enqueued, and tp_last_error() returns a message for the
 *    calling thread.  Argument checks run on the host before any launch;
 *    a launch failure reported by the HIP runtime gives TP_EHIP.  Faults
 *    inside a kernel surface at the caller's next synchronisation.
 *  - Pointers must be aligned to their element size; observation buffers
 *    to 16 bytes with a row pitch ld_obs that is a multiple of 8 elements,
 *    the packed actor buffer to 256 bytes.  Misalignment gives TP_EINVAL.
 *    Input and output buffers must not overlap, except the env state,
 *    which is read and updated in place.
 *  - Calls on different streams with disjoint buffers are independent.
 *    Results are deterministic: the same inputs give bitwise identical
 *    outputs (no floating-point atomics).
 *
 * Layout of the market (Section 3, "State space"; row = one bar)
 * --------------------------------------------------------------
 *  price [T1][n]      fp32 closing prices, row-major, one row per timestep
 *  ind   [T1][n][I]   fp32 technical indicators, stock-major within a row
 *  Prices must lie in [2^-2, 2^13): inside that range every traded value
 *  p*q (q <= 128) and every sum of up to 128 such values is exact in fp64,
 *  so share counts and balances are reproducible bit for bit.
 *
 * Observation row (Section 3, "State space"), K_pad = S rounded up to 32,
 * S = 1 + 2n + n*I:
 *  [ b*cash_scale, p_t*price_scale (n), h_t*share_scale (n), ind_t (n*I),
 *    zeros up to K_pad ]
 *  stored as fp32 (TP_F32) or bf16 round-to-nearest-even (TP_BF16).
 */
#ifndef TP_H
#define TP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TP_VERSION 2

typedef enum {
    TP_OK = 0,
    TP_EINVAL = -1,        /* bad pointer, size, alignment or value        */
    TP_ERANGE = -2,        /* a time index would leave the market / episode */
    TP_EUNSUPPORTED = -3,  /* valid request outside what the kernels handle */
    TP_EHIP = -4           /* HIP runtime error (launch, device query)      */
} tp_status;

typedef enum { TP_F32 = 0, TP_BF16 = 1 } tp_dtype;

/* Market tensor resident in device memory (see layout above). */
typedef struct tp_market {
    const float *price;    /* [T1][n]                                       */
    const float *ind;      /* [T1][n][n_ind]                                */
    int64_t T1;            /* rows                                          */
    int32_t n;             /* stocks, 1..128                                */
    int32_t n_ind;         /* indicators per stock, 0..; n*n_ind <= 1024    */
} tp_market;

/* MDP constants (Section 3; fee and initial capital: Figs. 4-5 captions). */
typedef struct tp_env_cfg {
    int32_t hmax;          /* max shares per stock and step (Section 3,
                              "Action space"), 1..128                       */
    int32_t horizon;       /* episode length in steps; done is raised on the
                              step whose index (step0 + j) equals horizon-1 */
    double fee;            /* proportional cost, 0 <= fee < 1: a sale
                              credits p*s*(1-fee), a purchase debits
                              p*q*(1+fee) (the c_t of eq. (2))              */
    double cash0;          /* initial balance b_0 >= 0                       */
    double reward_scale;   /* r = reward_scale * (V' - V), V = b + p^T h    */
    float cash_scale;      /* observation scales                             */
    float price_scale;
    float share_scale;
} tp_env_cfg;

/* Batched env state, read and updated in place (structure of arrays). */
typedef struct tp_env_state {
    double *cash;          /* [E] balance b                                 */
    int32_t *shares;       /* [E][n] holdings h (>= 0)                       */
    int64_t *t;            /* [E] current market row                         */
    int32_t E;             /* envs, >= 1                                     */
    int32_t *n_invalid;    /* optional device int32 [1], or NULL: every call
                              that takes the state sets it to the number of
                              envs it could not start (tp_env_reset: t0
                              outside [0, T1-1)) or step (tp_env_step,
                              tp_rollout: not enough market rows left).  The
                              host cannot read device-side time indices;
                              this count is how such envs are reported.     */
} tp_env_state;

/* Actor: the PPO Gaussian policy (PPO is named in Section 5.2):
 *   mu = W3 tanh(W2 tanh(W1 x + b1) + b2) + b3,  a = mu + exp(log_std) z.
 * Parameters are fp32 masters stacked per agent; env e belongs to agent
 * e / envs_per_agent (population of agents, Section 4.2).
 *   W[0] [A][H1][S], W[1] [A][H2][H1], W[2] [A][n][H2]  row-major [out][in]
 *   b[0] [A][H1],    b[1] [A][H2],     b[2] [A][n];     log_std [A][n]
 * dtype TP_BF16 computes with bf16 (round-to-nearest-even) copies of the
 * weights, bf16 observations and bf16 hidden activations, fp32
 * accumulation; TP_F32 computes in fp32 throughout. */
typedef struct tp_actor {
    int32_t n_agents;      /* A >= 1                                         */
    int32_t envs_per_agent;/* A * envs_per_agent == E                        */
    int32_t dims[4];       /* {S, H1, H2, n}                                 */
    int32_t dtype;         /* tp_dtype                                       */
    const float *W[3];
    const float *b[3];
    const float *log_std;
    int64_t agent_stride;  /* floats from one agent's parameters to the next
                              in every W / b / log_std array; 0 = the stacked
                              layouts above.  With the learner's flat vectors
                              [A][P] (tp_ppo_update) agent_stride = P and the
                              pointers address agent 0's segments.          */
} tp_actor;

/* Trajectory store, time-major (Section 4.4, "Replay buffer on GPU").
 * Row j holds (obs_j, a_j, logp_j, r_j, done_j): the observation before
 * action j, the raw sampled action, its log-probability, the reward and
 * the episode-end flag.  Every pointer except action/logp/reward/done may
 * be NULL to skip that output. */
typedef struct tp_traj {
    void *obs;             /* [L][E][ld_obs], dtype = actor dtype, or NULL   */
    int64_t ld_obs;        /* row stride in elements: >= K_pad, % 8 == 0     */
    float *action;         /* [L][E][n] raw actions a (before clipping)      */
    float *logp;           /* [L][E] log pi(a_j | obs_j)                     */
    float *reward;         /* [L][E]                                         */
    uint8_t *done;         /* [L][E] 1 on the last step of an episode       */
    double *cash_tap;      /* [L][E] balance after step j, or NULL          */
    int32_t *shares_tap;   /* [L][E][n] holdings after step j, or NULL      */
    void *obs_last;        /* [E][ld_obs] observation after the last step
                              (the bootstrap state), or NULL                 */
    double *asset_tap;     /* [L][E] total asset b + p^T h after step j, at
                              the prices of the new row (the account value
                              of eq. (2)), or NULL; NaN for an env that is
                              not stepped                                    */
    float *mu_tap;         /* [L][E][n] the actor's output mu_j (the mean of
                              the Gaussian policy) that a_j was drawn
                              around, or NULL; NaN for an env that is not
                              stepped                                        */
} tp_traj;

/*
 * tp_env_reset -- start an episode in every env (Section 3: the state is
 * balance, shares, prices, indicators).
 *   Sets cash[e] = cash0, shares[e][:] = 0, t[e] = t0[e] and, if obs0 is
 *   not NULL, writes the observation at row t0[e] to obs0[e][0:K_pad) (pad
 *   columns zero).  t0 is a device int64 [E].  The host cannot read t0, so
 *   the kernel checks it: an env with t0[e] outside [0, T1-1) gets
 *   t[e] = -1 (an invalid env: every later step or rollout leaves it
 *   untouched and reports NaN for it) and a zero observation row; the
 *   number of such envs goes to st->n_invalid when that is not NULL.
 *   Callers that hold t0 on the host check it first with tp_check_starts,
 *   which returns TP_ERANGE for a start without enough market rows.
 *   obs_dtype: tp_dtype of obs0.
 */
int tp_env_reset(const tp_market *mkt, const tp_env_cfg *cfg,
                 const tp_env_state *st, const int64_t *t0, void *obs0,
                 int64_t ld_obs, int32_t obs_dtype, void *stream);

/*
 * tp_env_step -- one transition of every env with caller-supplied raw
 * actions (Section 3, eqs. (2)-(4); teacher forcing).
 *   action [E][n] fp32 raw actions; u = clip(a, -1, 1) (NaN -> 0),
 *   k = trunc(u * hmax) shares (fp32 product, toward zero).  All sells
 *   (s = min(-k, h)) execute first at p_t, then buys in ascending stock
 *   index, each the largest q <= k the balance still covers with fees.
 *   reward [E] = reward_scale * (V(t+1) - V(t)); the state advances one
 *   row; if obs_next is not NULL the new observation is written there
 *   ([E][ld_obs], obs_dtype).
 *   Every t[e] + 1 must be < T1: the host cannot read device t, so the
 *   kernel checks it; an env with t[e] < 0 or t[e] + 1 >= T1 is left
 *   unchanged, gets reward NaN and (if requested) a NaN observation row,
 *   and is counted in st->n_invalid when that is not NULL.
 */
int tp_env_step(const tp_market *mkt, const tp_env_cfg *cfg,
                const tp_env_state *st, const float *action, float *reward,
                void *obs_next, int64_t ld_obs, int32_t obs_dtype,
                void *stream);

/*
 * tp_actor_packed_bytes / tp_actor_pack -- convert the actor's fp32 masters
 * into the kernel's tiled layout (bf16 round-to-nearest-even copies for
 * TP_BF16) in a caller-owned device buffer of tp_actor_packed_bytes()
 * bytes.  Call again after every parameter update: tp_rollout reads only
 * the packed copy.  tp_actor_packed_bytes returns 0 for an invalid actor.
 */
size_t tp_actor_packed_bytes(const tp_actor *actor);
int tp_actor_pack(const tp_actor *actor, void *packed, size_t packed_bytes,
                  void *stream);

/*
 * tp_actor_release / tp_critic_release -- forget a packed buffer (host
 * only; nothing is freed).  The library records, per packed buffer, the
 * shape it was filled with, and tp_rollout / tp_critic_value accept only
 * buffers so recorded.  Call this before freeing a packed buffer, so that
 * a later allocation at the same address is not taken for it.  Packing
 * into a buffer also forgets every recorded buffer it overlaps.  Returns
 * TP_EINVAL for a pointer that is not recorded.
 */
int tp_actor_release(const void *packed);
int tp_critic_release(const void *packed);

/*
 * tp_check_starts -- host-side check of episode start rows (Section 3: the
 * MDP steps through consecutive bars of the market).  t0_host [E] is a
 * HOST array; every env must have L market rows after its start:
 * 0 <= t0[e] and t0[e] + L <= T1 - 1.  Returns TP_OK, or TP_ERANGE with
 * the first offending env in tp_last_error(); TP_EINVAL for bad sizes.
 */
int tp_check_starts(const int64_t *t0_host, int32_t E, int64_t T1, int32_t L);

/*
 * tp_rollout -- L lockstep steps of the batched env driven by the actor
 * (the worker's exploration pass, Section 4.3; batch mode, Section 4.4).
 *   For j = 0..L-1 and every env e (agent g = e / envs_per_agent):
 *     obs_j  from the current state and market row t;
 *     mu     = actor_g(obs_j);
 *     z_i    = Box-Muller normals from Philox4x32-10 with counter
 *              (i/4, e, step0+j, g) and key (seed low 32, seed high 32);
 *              the 4 uniforms u = ((w >> 9) + 0.5) 2^-23 of one counter
 *              give two pairs (u0,u1), (u2,u3); stock i takes z_{i mod 4};
 *     a      = mu + exp(log_std) z;  logp = sum(-z^2/2 - log_std)
 *              - (n/2) ln(2 pi);
 *     the env step of tp_env_step with a;  done = (step0+j+1 == horizon).
 *   One kernel launch runs all L steps.  step0 is the episode step of the
 *   state on entry (it selects the random stream), so a rollout split into
 *   pieces with matching step0 reproduces the unsplit one bit for bit.
 *   Requires step0 + L <= horizon.  Device-side t is not visible to the
 *   host: an env with t < 0 or t + L > T1 - 1 is not stepped: its state is
 *   left unchanged, its action / logp / reward / mu rows are NaN, done is
 *   0, the taps hold the unchanged state, its observation rows are not
 *   written, and it is counted in st->n_invalid when that is not NULL.
 *   `packed` must come from tp_actor_pack with the same actor shape and
 *   must not have been released (tp_actor_release) since.
 */
int tp_rollout(const tp_market *mkt, const tp_env_cfg *cfg,
               const tp_env_state *st, const tp_actor *actor,
               const void *packed, size_t packed_bytes, uint64_t seed,
               uint64_t step0, int32_t L, const tp_traj *traj, void *stream);

/*
 * tp_rollout_path -- which rollout kernel tp_rollout launches for this
 * market and actor shape: 1 = the role-split kernel (bf16, 100 stocks x 4,
 * 8 or 10 indicators, S-H-H-100 with H = 256, 512, 768 or 1024, given
 * 16-byte aligned market, action and holdings-tap buffers), 0 = the generic
 * kernel, or a negative tp_status for an invalid market or actor.  Host
 * only.
 */
int tp_rollout_path(const tp_market *market, const tp_actor *actor);

/*
 * tp_gae -- generalized advantage estimation over a rollout (PPO's
 * estimator; discounting as in eq. (1), gamma from Table 2).
 *   reward, done, adv, ret [L][E]; value [L+1][E] (row L = bootstrap).
 *   delta_j = r_j + gamma (1-d_j) V_{j+1} - V_j;
 *   A_j = delta_j + gamma lambda (1-d_j) A_{j+1} (A_L = 0);  ret_j = A_j + V_j.
 *   Accumulates in fp64, stores fp32.  0 < gamma <= 1, 0 <= lambda <= 1.
 */
int tp_gae(const float *reward, const float *value, const uint8_t *done,
           int32_t L, int32_t E, float gamma, float lambda, float *adv,
           float *ret, void *stream);

/* Critic: the value network of the PPO learner (PPO, Section 5.2; the
 * learner trains the networks, Section 4.3):
 *   V(x) = w3 . tanh(W2 tanh(W1 x + b1) + b2) + b3   (a scalar per state).
 * fp32 masters stacked per agent, env e belongs to agent e / envs_per_agent:
 *   W[0] [A][H1][S], W[1] [A][H2][H1], W[2] [A][H2] (w3);
 *   b[0] [A][H1], b[1] [A][H2], b[2] [A].
 * dtype as for the actor (TP_BF16: bf16 copies of weights, observations and
 * hidden activations, fp32 accumulation; TP_F32: fp32 throughout). */
typedef struct tp_critic {
    int32_t n_agents;      /* A >= 1                                         */
    int32_t envs_per_agent;/* A * envs_per_agent == E of the observations    */
    int32_t dims[3];       /* {S, H1, H2}                                    */
    int32_t dtype;         /* tp_dtype                                       */
    const float *W[3];
    const float *b[3];
    int64_t agent_stride;  /* as tp_actor.agent_stride                       */
} tp_critic;

/*
 * tp_critic_packed_bytes / tp_critic_pack -- the critic's fp32 masters in
 * the kernels' layout (as tp_actor_pack), in a caller-owned device buffer
 * of tp_critic_packed_bytes() bytes (256-byte aligned).  Returns 0 / an
 * error for an invalid critic.
 */
size_t tp_critic_packed_bytes(const tp_critic *critic);
int tp_critic_pack(const tp_critic *critic, void *packed, size_t packed_bytes,
                   void *stream);

/*
 * tp_critic_value -- V of every observation row of a time-major block of
 * observations (a trajectory's obs, or its bootstrap row obs_last).
 *   obs   [T][E][ld_obs] rows in the layout tp_rollout writes (dtype =
 *         critic dtype; the first S = dims[0] columns are the state, the
 *         rest up to K_pad are ignored);
 *   value [T][E] fp32 out; row (t, e) uses agent e / envs_per_agent.
 *   T >= 1, E = n_agents * envs_per_agent; obs 16-byte aligned, ld_obs >=
 *   K_pad and a multiple of 8; `packed` from tp_critic_pack with the same
 *   shape.  Rows are independent; results are deterministic.
 */
int tp_critic_value(const tp_critic *critic, const void *packed,
                    size_t packed_bytes, const void *obs, int64_t ld_obs,
                    int64_t T, int32_t E, float *value, void *stream);

/*
 * tp_backtest_metrics -- the evaluator's measurements of a backtest
 * (Section 5.2, "Evaluation metrics"), per env, from its total-asset series
 * V_0 = v0[e] and V_t = v[t-1][e], t = 1..T (e.g. a rollout's asset_tap):
 *   r_t = V_t / V_{t-1} - 1, s = sample standard deviation of r;
 *   out[e][0] cumulative return  V_T / V_0 - 1
 *   out[e][1] annual return      (V_T / V_0)^(P / T) - 1
 *   out[e][2] annual volatility  s sqrt(P)
 *   out[e][3] Sharpe ratio       (mean(r) - risk_free / P) / s * sqrt(P),
 *                                0 when s = 0
 *   out[e][4] max drawdown       max_t (peak_t - V_t) / peak_t, peak_t =
 *                                max_{u <= t} V_u
 *   with P = periods_per_year (252 for daily bars, 252 * 390 for minute
 *   bars) and risk_free the annual rate.  v0 [E], v [T][E], out [E][5] fp64
 *   device arrays; T, E >= 1, periods_per_year > 0; work: a device buffer of
 *   at least tp_backtest_metrics_work_bytes(T, E) bytes (contents are
 *   scratch; calls that share one workspace must not overlap).
 * The sums behind the volatility and the Sharpe ratio are taken over time
 * segments in a fixed order (deterministic); the drawdown is exact.
 */
int tp_backtest_metrics(const double *v0, const double *v, int32_t T, int32_t E,
                        double periods_per_year, double risk_free, double *out,
                        void *work, size_t work_bytes, void *stream);

/*
 * tp_backtest_metrics_noalloc -- tp_backtest_metrics for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the same kernels and the same results,
 * bit for bit, with the segment partials in a static device scratch array
 * of 4.5 MiB that the library holds on each GPU it runs on until the
 * process ends, instead of a caller workspace.  Nothing is allocated.
 * Every shape within the limits of tp_backtest_metrics fits (the largest
 * needs about 4.1 MiB); a request that would not fit returns
 * TP_EUNSUPPORTED.  All calls on one GPU share its scratch, which keeps the
 * last call's contents (nothing in it needs clearing): calls that may
 * overlap on one GPU (different streams, or different host threads) race
 * and must be serialised by the caller.  The stream must belong to the
 * current device.  Arguments otherwise as tp_backtest_metrics.
 */
int tp_backtest_metrics_noalloc(const double *v0, const double *v, int32_t T, int32_t E,
                                double periods_per_year, double risk_free, double *out,
                                void *stream);

/* Bytes of the caller-owned device workspace tp_backtest_metrics needs for
 * T steps of E series (8-byte aligned; segment partial sums and maxima), or
 * 0 for T < 1 or E outside 1 .. 64 * 65535.  Host only. */
size_t tp_backtest_metrics_work_bytes(int32_t T, int32_t E);

/*
 * PPO learner (PPO, Section 5.2; hyper-parameters of Table 2: Adam,
 * learning rate 2^-14, batch 2^10, repeat 2^3, ratio clip 0.25, entropy
 * coefficient 0.02; the learner trains the networks on the transitions the
 * workers stored, Section 4.3): minibatch updates of one agent's actor and
 * critic, both read from and written to one flat fp32 vector.
 *
 * Flat parameters of one agent, fp32 [P] (P = tp_ppo_param_count), in order:
 *   W1 [H1][S], b1 [H1], W2 [H2][H1], b2 [H2], W3 [n][H2], b3 [n],
 *   log_std [n], Wc1 [C1][S], bc1 [C1], Wc2 [C2][C1], bc2 [C2], wc3 [C2],
 *   bc3 [1]
 * (a tp_actor / tp_critic with agent_stride = P points into [A][P]).
 *
 * One update on the minibatch rows idx[0..B-1] of a time-major trajectory
 * (row r = j E + e of its [L][E] arrays) takes the gradient of
 *   L = L_clip - ent_coef H + L_critic, where
 *   logp_i = sum_k [-(a_ik - mu_ik)^2 / (2 sigma_k^2) - log_std_k] - (n/2) ln 2pi,
 *   rho_i  = exp(logp_i - logp_old_i),
 *   L_clip = -(1/B) sum_i min(rho_i A_i, clip(rho_i, 1 - clip, 1 + clip) A_i),
 *   H      = sum_k (log_std_k + (1 + ln 2pi) / 2)   (Gaussian entropy),
 *   L_critic = (1/B) sum_i (V_i - R_i)^2,
 * with mu and V the actor and critic of this vector on observation row x_i
 * (tanh hidden layers as in tp_rollout / tp_critic_value), then one Adam
 * step (Kingma and Ba) at step number t:
 *   m = b1 m + (1 - b1) g;  v = b2 v + (1 - b2) g^2;
 *   theta -= lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps).
 */
typedef struct tp_ppo {
    int32_t dims[6];       /* S, H1, H2, n (actor), C1, C2 (critic)           */
    int32_t dtype;         /* TP_BF16: bf16 operands (weights rounded from the
                              masters, observations as stored, activations and
                              backpropagated gradients rounded), fp32 sums;
                              TP_F32: fp32 throughout                        */
    int32_t batch;         /* B, rows per minibatch: a multiple of 32        */
    float clip;            /* ratio clip, 0 < clip < 1 (0.25)                */
    float ent_coef;        /* entropy coefficient >= 0 (0.02)                */
    float lr;              /* learning rate > 0 (2^-14)                      */
    float beta1, beta2;    /* Adam decay rates in [0, 1) (0.9, 0.999)        */
    float eps;             /* Adam epsilon > 0 (1e-8)                        */
} tp_ppo;

/* P for this configuration, or 0 (tp_last_error says why) when the
 * configuration is invalid: S >= 1, 1 <= n <= 128, H1, H2, C1, C2 positive
 * multiples of 32, batch a positive multiple of 32. */
int64_t tp_ppo_param_count(const tp_ppo *cfg);

/* Bytes of the caller-owned device workspace tp_ppo_update needs (operand
 * copies of the weights, minibatch activations and gradients), or 0. */
size_t tp_ppo_workspace_bytes(const tp_ppo *cfg);

/*
 * tp_ppo_update -- n_updates minibatch updates in sequence on `stream`.
 *   params, adam_m, adam_v  [P] fp32 device, updated in place (m and v start
 *                           at zero before step 1);
 *   step0                   Adam step number of the first update (>= 1);
 *                           update u uses step0 + u;
 *   obs [rows][ld_obs]      observation rows (bf16 for TP_BF16, fp32 for
 *                           TP_F32) as tp_rollout writes them; columns >= S
 *                           are ignored; ld_obs >= S;
 *   action [rows][n], logp, adv, ret [rows]  fp32: the stored raw actions,
 *                           their log-probabilities under the policy that
 *                           acted, the GAE advantages and returns;
 *   idx [n_updates][B]      int64 device row indices (values outside
 *                           [0, rows) are clamped into it; rows of envs that
 *                           were not stepped hold NaN and must not be drawn);
 *   grad [P]                optional (NULL): the last update's gradient;
 *   stats [n_updates][4]    optional fp64: L_clip, H, L_critic and the
 *                           fraction of rows with |rho - 1| > clip, at the
 *                           parameters each update starts from;
 *   workspace               >= tp_ppo_workspace_bytes, 256-byte aligned.
 * Nothing is allocated.  Returns TP_EINVAL for a bad configuration, NULL or
 * misaligned pointers, or a short workspace.
 */
int tp_ppo_update(const tp_ppo *cfg, float *params, float *adam_m, float *adam_v,
                  int64_t step0, int32_t n_updates, const void *obs, int64_t ld_obs,
                  const float *action, const float *logp, const float *adv,
                  const float *ret, int64_t rows, const int64_t *idx, float *grad,
                  double *stats, void *workspace, size_t workspace_bytes, void *stream);

/*
 * tp_ppo_update_agents -- tp_ppo_update for n_agents independent learners
 * in one call (the population's agents, and the pods of an agent, train
 * separately between fusions: Section 4.4).  Every launch of an update
 * covers all agents, so small minibatches still fill the device.
 *   n_agents       1 .. 1024;
 *   agent_stride   floats from one agent's params / adam_m / adam_v to the
 *                  next (>= P; ignored for one agent): the flat [A][P]
 *                  layout has agent_stride = P;
 *   idx            [n_agents][n_updates][B] int64 device row indices into
 *                  the shared trajectory arrays (each agent draws its own
 *                  rows, e.g. from its envs with tp_minibatch_rows);
 *   grad           optional [n_agents][P]; stats optional
 *                  [n_agents][n_updates][4];
 *   workspace      >= n_agents * tp_ppo_workspace_bytes(cfg), 256-byte
 *                  aligned; agent a uses the a-th slice.
 * Agent a's results equal those of tp_ppo_update on its own arrays, bit
 * for bit.  Returns TP_EINVAL as tp_ppo_update does, and for n_agents out
 * of range or agent_stride < P.
 */
int tp_ppo_update_agents(const tp_ppo *cfg, int32_t n_agents, int64_t agent_stride,
                         float *params, float *adam_m, float *adam_v, int64_t step0,
                         int32_t n_updates, const void *obs, int64_t ld_obs,
                         const float *action, const float *logp, const float *adv,
                         const float *ret, int64_t rows, const int64_t *idx, float *grad,
                         double *stats, void *workspace, size_t workspace_bytes,
                         void *stream);

/*
 * tp_minibatch_rows -- the learner's minibatch draws (the learner samples
 * the stored transitions, Section 4.3; batch size from Table 2), with
 * replacement, from agent `agent`'s R = L * envs_per_agent transitions:
 * draw i of update u is word i % 4 of Philox4x32-10 with counter
 * (i / 4, counter + u, agent, 0x4D42) and key (seed low, seed high) -- a
 * stream of its own beside the action noise -- mapped to
 * x = floor(w R / 2^32), step j = x / envs_per_agent, env
 * e = agent * envs_per_agent + x % envs_per_agent, row j * E + e.
 *   idx [n_updates][B] int64 device out (tp_ppo_update's idx).
 * Returns TP_EINVAL for bad sizes or an agent outside 0 .. E/envs_per_agent-1.
 */
int tp_minibatch_rows(uint64_t seed, uint64_t counter, int32_t n_updates, int32_t B,
                      int32_t L, int32_t E, int32_t agent, int32_t envs_per_agent,
                      int64_t *idx, void *stream);

/*
 * Evolution layer (Section 4.2): model ensemble, evaluator and selector
 * over a population of agents whose parameters are flat fp32 vectors of P
 * values each (e.g. the actor's W and b masters laid end to end).
 */

/*
 * tp_ensemble_fuse -- every pod of agent g (K pods trained with different
 * seeds) takes the mean of the agent's K parameter vectors.
 *   params [N][K][P] fp32, in place; each mean is summed in fp64 over
 *   k = 0..K-1 and rounded once.  N, K >= 1, P >= 1.
 */
int tp_ensemble_fuse(float *params, int32_t N, int32_t K, int64_t P,
                     void *stream);

/*
 * tp_fitness -- the evaluator's fitness score, the objective J of eq. (1)
 * on an evaluation rollout: env_return[e] = sum_j gamma^j reward[j][e]
 * (fp64; NaN if any of the env's rewards is NaN, i.e. it was not stepped),
 * and fitness[g] = the mean of env_return over the envs of agent g that
 * were stepped (NaN if none), in env order.  Env e belongs to agent
 * e / (E / n_agents).
 *   reward [L][E] fp32; env_return [E], fitness [n_agents] fp64 out;
 *   E % n_agents == 0.
 */
int tp_fitness(const float *reward, int32_t L, int32_t E, int32_t n_agents,
               double gamma, double *env_return, double *fitness, void *stream);

/*
 * tp_keep_best -- the evaluator's keep-best bookkeeping: for every agent g
 * whose fitness[g] beats best[g] (a NaN best is always beaten, a NaN
 * fitness never beats), best[g] = fitness[g], best_params[g] = params[g]
 * and stall[g] = 0; otherwise stall[g] += 1.  A training loop stops the
 * agent (early stopping) once stall[g] reaches its patience and keeps
 * best_params[g] as the final agent.
 *   fitness, best [A] fp64; stall [A] int32; params, best_params [A][P].
 */
int tp_keep_best(const double *fitness, double *best, int32_t *stall,
                 const float *params, float *best_params, int32_t A, int64_t P,
                 void *stream);

/*
 * tp_select -- the selector's step (Section 4.2, the selection of a genetic
 * algorithm): rank the N agents by fitness, descending, NaN last, ties to
 * the lower index; the `keep` best survive and the agent of rank r >= keep
 * becomes a copy of the survivor of rank (r - keep) mod keep.
 *   fitness [N] fp64; params [N][P] fp32, in place; rank [N] int32 out
 *   (the rank of each agent).  1 <= keep <= N <= 1024.
 */
int tp_select(const double *fitness, float *params, int32_t N, int64_t P,
              int32_t keep, int32_t *rank, void *stream);

/* Message for the last non-OK return on the calling thread ("" if none). */
const char *tp_last_error(void);

/* TP_VERSION of the built library. */
int tp_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TP_H */
