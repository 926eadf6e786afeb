/*
 * Oracle for the FinRL-Podracer rollout hot path (arXiv 2111.05188).
 *
 * TEST INFRASTRUCTURE ONLY.  This is a plain, slow, sequential CPU
 * implementation of what the GPU library computes.  It exists to check the
 * HIP kernels.  Only the test suite, the package smoke check and the
 * benchmark's CPU-baseline leg may load it.  It shares no code, header,
 * table or helper with the HIP path.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fPIC -shared (no fast-math).
 * Every floating-point fma below is written out as fma(); nothing else is
 * contracted.
 *
 * What each part follows (paper = FinRL-Podracer, arXiv 2111.05188):
 *   - state s_t = [balance b_t, shares h_t, close prices p_t, indicators]
 *     : Section 3, "State space".
 *   - action: per stock an integer number of shares in {-k..k}, |k| <= h_max
 *     : Section 3, "Action space".
 *   - reward = change of total asset (balance + p^T h) minus transaction
 *     cost : Section 3, eq. (2).
 *   - transition: sell set / buy set, balance and holdings update, holdings
 *     stay >= 0 : Section 3, eqs. (3)-(4).
 *   - objective / discounting: eq. (1); gamma = 0.99 from Table 2.
 *   - the policy is PPO's Gaussian actor (PPO is named in Section 5.2), GAE is
 *     PPO's advantage estimator.  Neither detail is printed in the paper;
 *     the readings used are listed beside each function.
 *
 * Parity pins (tests that tie this file to the paper and to mathematics
 * rather than to itself) live in tests/test_oracle_*.py.  orc_philox4x32_10
 * is pinned against ROCm's rocRAND host implementation of the same
 * generator.  orc_obs has its layout and its power-of-two block scaling
 * pinned; the two scale constants are a reading (parity unpinned).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_VERSION 1

/* ------------------------------------------------------------------------ */
/* Inputs                                                                    */
/* ------------------------------------------------------------------------ */

/* Market: price fp32 [rows][n], ind fp32 [rows][n][n_ind]; row t of the
 * full tensor lives at index (t - row0). */
typedef struct {
    const float *price;
    const float *ind;
    int64_t row0;
    int64_t rows;
    int32_t n;
    int32_t n_ind;
} orc_market;

/* MDP constants. */
typedef struct {
    int32_t hmax;          /* max shares traded per stock and step          */
    int32_t horizon;       /* episode length in steps (done flag)           */
    double fee;            /* proportional transaction cost                 */
    double cash0;          /* initial balance                               */
    double reward_scale;   /* r = reward_scale * (V' - V)                   */
    float cash_scale;      /* observation scales                            */
    float price_scale;
    float share_scale;
} orc_env_cfg;

/* Actor: fp32 master weights, stacked per agent.
 * W[l] : [n_agents][out_l][in_l] row-major, b[l] : [n_agents][out_l],
 * log_std : [n_agents][n].  dims = {S, H1, H2, n}.  bf16 != 0 selects the
 * bf16 configuration (weights, observations and hidden activations rounded
 * to bf16). */
typedef struct {
    int32_t n_agents;
    int32_t envs_per_agent;
    int32_t dims[4];
    int32_t bf16;
    const float *W[3];
    const float *b[3];
    const float *log_std;
} orc_actor;

int orc_version(void) { return ORC_VERSION; }

/* Threads the rollout's envs are split over: 1 for the plain build, the
 * OpenMP team size for the OpenMP build. */
#ifdef _OPENMP
#include <omp.h>
int orc_threads(void) { return omp_get_max_threads(); }
#else
int orc_threads(void) { return 1; }
#endif

/* ------------------------------------------------------------------------ */
/* bf16 rounding (IEEE round-to-nearest-even on the upper 16 bits)           */
/* ------------------------------------------------------------------------ */

static uint32_t f2u(float x) { uint32_t u; memcpy(&u, &x, 4); return u; }
static float u2f(uint32_t u) { float x; memcpy(&x, &u, 4); return x; }

/* fp32 -> bf16 bit pattern.  The kept part is the upper half of the fp32
 * bit pattern; the discarded lower half is compared with the halfway point
 * 0x8000 and ties go to the even kept value.  NaN stays a quiet NaN. */
uint16_t orc_bf16_bits(float x)
{
    uint32_t u = f2u(x);
    if (isnan(x)) return (uint16_t)((u >> 16) | 0x0040u);
    uint32_t hi = u >> 16, lo = u & 0xFFFFu;
    if (lo > 0x8000u || (lo == 0x8000u && (hi & 1u))) hi += 1u;
    return (uint16_t)hi;
}

float orc_bf16_value(uint16_t h) { return u2f((uint32_t)h << 16); }

static float round_bf16(float x) { return orc_bf16_value(orc_bf16_bits(x)); }

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11, "Parallel random       */
/* numbers: as easy as 1, 2, 3"): a 4-word counter is enciphered by ten      */
/* rounds of a multiply-based bijection keyed by a 2-word key; the key is    */
/* advanced by the Weyl constants between rounds.                            */
/* ------------------------------------------------------------------------ */

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

void orc_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2],
                       uint32_t out[4])
{
    uint32_t x0 = ctr_in[0], x1 = ctr_in[1], x2 = ctr_in[2], x3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) { k0 += PHILOX_W0; k1 += PHILOX_W1; }
        uint64_t p0 = (uint64_t)PHILOX_M0 * (uint64_t)x0;
        uint64_t p1 = (uint64_t)PHILOX_M1 * (uint64_t)x2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t y0 = hi1 ^ x1 ^ k0;
        uint32_t y1 = lo1;
        uint32_t y2 = hi0 ^ x3 ^ k1;
        uint32_t y3 = lo0;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* 32 random bits -> uniform in (0,1): keep the top 23 bits, centre them in
 * their cell.  ((w >> 9) + 0.5) * 2^-23 is exact in fp32 and never 0 or 1. */
float orc_uniform(uint32_t w)
{
    return ((float)(w >> 9) + 0.5f) * (1.0f / 8388608.0f);
}

/* Standard normals for one (env, step): z_i for i = 0..n-1.  Counter
 * (i/4, env, step, agent), key (seed low word, seed high word).  The four
 * uniforms of one counter give two Box-Muller pairs (Box & Muller 1958):
 *   z0 = sqrt(-2 ln u0) cos(2 pi u1),  z1 = sqrt(-2 ln u0) sin(2 pi u1),
 * and likewise (u2, u3) -> z2, z3.  Stock i takes z_{i mod 4} of counter
 * i/4.  Computed in fp32 with the C library's logf/sqrtf/cosf/sinf. */
void orc_normals(uint64_t seed, uint32_t step, uint32_t env, uint32_t agent,
                 int32_t n, float *z)
{
    const uint32_t key[2] = { (uint32_t)seed, (uint32_t)(seed >> 32) };
    for (int32_t c = 0; 4 * c < n; ++c) {
        const uint32_t ctr[4] = { (uint32_t)c, env, step, agent };
        uint32_t w[4];
        orc_philox4x32_10(ctr, key, w);
        float zz[4];
        for (int pair = 0; pair < 2; ++pair) {
            float u0 = orc_uniform(w[2 * pair]);
            float u1 = orc_uniform(w[2 * pair + 1]);
            float rad = sqrtf(-2.0f * logf(u0));
            float ang = 6.28318530717958647692f * u1;
            zz[2 * pair] = rad * cosf(ang);
            zz[2 * pair + 1] = rad * sinf(ang);
        }
        for (int m = 0; m < 4 && 4 * c + m < n; ++m) z[4 * c + m] = zz[m];
    }
}

/* ------------------------------------------------------------------------ */
/* Observation (Section 3, "State space"): [b, p_t, h_t, indicators_t].     */
/* Scales are a reading (power-of-two, exact): b*cash_scale, p*price_scale,  */
/* h*share_scale, indicators raw.  Pad positions S..K_pad-1 are zero.        */
/* Layout and power-of-two scaling pinned; the two constants: parity        */
/* unpinned (no value in the paper fixes them).                              */
/* ------------------------------------------------------------------------ */

static const float *price_row(const orc_market *m, int64_t t)
{
    return m->price + (size_t)(t - m->row0) * (size_t)m->n;
}

static const float *ind_row(const orc_market *m, int64_t t)
{
    return m->ind + (size_t)(t - m->row0) * (size_t)m->n * (size_t)m->n_ind;
}

/* Writes K_pad values of one observation as fp32 (obs_f32 != NULL) or as
 * bf16 bit patterns (obs_bf16 != NULL). */
void orc_obs(const orc_market *m, const orc_env_cfg *cfg, int64_t t,
             double cash, const int32_t *shares, int32_t K_pad,
             float *obs_f32, uint16_t *obs_bf16)
{
    const int32_t n = m->n, nI = m->n * m->n_ind;
    const float *p = price_row(m, t), *ind = ind_row(m, t);
    for (int32_t k = 0; k < K_pad; ++k) {
        float x;
        if (k == 0) x = (float)(cash * (double)cfg->cash_scale);
        else if (k <= n) x = p[k - 1] * cfg->price_scale;
        else if (k <= 2 * n) x = (float)shares[k - 1 - n] * cfg->share_scale;
        else if (k <= 2 * n + nI) x = ind[k - 1 - 2 * n];
        else x = 0.0f;
        if (obs_f32) obs_f32[k] = x;
        if (obs_bf16) obs_bf16[k] = orc_bf16_bits(x);
    }
}

/* ------------------------------------------------------------------------ */
/* Reset: b = cash0, h = 0, t = t0 (initial capital: Figs. 4-5 captions).          */
/* ------------------------------------------------------------------------ */

void orc_env_reset(const orc_env_cfg *cfg, int32_t E, int32_t n,
                   const int64_t *t0, double *cash, int32_t *shares,
                   int64_t *t)
{
    for (int32_t e = 0; e < E; ++e) {
        cash[e] = cfg->cash0;
        for (int32_t i = 0; i < n; ++i) shares[(size_t)e * n + i] = 0;
        t[e] = t0[e];
    }
}

/* ------------------------------------------------------------------------ */
/* Action mapping (Section 3, "Action space"): raw Gaussian action a ->      */
/* u = clip(a, -1, 1) (NaN -> 0, i.e. hold) -> k = trunc(u * h_max) shares,  */
/* the product taken in fp32, truncated toward zero.                         */
/* ------------------------------------------------------------------------ */

float orc_clip_action(float a)
{
    if (isnan(a)) return 0.0f;
    if (a < -1.0f) return -1.0f;
    if (a > 1.0f) return 1.0f;
    return a;
}

int32_t orc_shares_from_action(float a, int32_t hmax)
{
    float u = orc_clip_action(a);
    float prod = u * (float)hmax;
    return (int32_t)truncf(prod);
}

/* ------------------------------------------------------------------------ */
/* One env step (Section 3, eqs. (2)-(4)).                                   */
/*                                                                           */
/* Readings where the paper leaves a choice open:                            */
/*  - trades execute at p_t; the new total asset is valued at p_{t+1}        */
/*    (eq. (2) values the next state at p_{t+1}, eq. (3) trades at p_t);     */
/*  - the transaction cost c_t is charged to the balance: a sale credits     */
/*    p*s*(1-fee), a purchase debits p*q*(1+fee); then eq. (2)'s            */
/*    r = V' - V - c_t with c_t counted once equals the change of the       */
/*    balance-plus-holdings value;                                          */
/*  - all sells first, then buys in ascending stock index, each buying the   */
/*    largest whole number of shares q <= k that the balance still covers    */
/*    (fees included), so b >= 0 and h >= 0 always hold (eq. (4));           */
/*  - reward r = reward_scale * (V' - V) rounded to fp32.                    */
/*                                                                           */
/* Sums of p*s and p*q are exact in fp64 for prices in [2^-2, 2^13) and      */
/* trades of at most 128 shares over at most 128 stocks.                     */
/*                                                                           */
/* Optional diagnostics out[5] = {V, V', S (sold value), G (bought value),   */
/* b_s (balance after sells)}.                                               */
/* ------------------------------------------------------------------------ */

/* An env whose next row is not in the market (t < row0 or t + 1 beyond the
 * last row) is not stepped: its state is left as it is and the reward is
 * NaN (the library's documented behaviour for such an env). */
static int has_rows(const orc_market *m, int64_t t, int64_t steps)
{
    return t >= m->row0 && t + steps <= m->row0 + m->rows - 1;
}

float orc_env_step_one(const orc_market *m, const orc_env_cfg *cfg,
                       double *cash, int32_t *shares, int64_t *t,
                       const float *action, double *diag)
{
    const int32_t n = m->n;
    if (!has_rows(m, *t, 1)) return NAN;
    const double f_s = 1.0 - cfg->fee, f_b = 1.0 + cfg->fee;
    const float *p = price_row(m, *t);
    const float *p1 = price_row(m, *t + 1);
    double b = *cash;

    /* V = b + p^T h: the dot product first (exact, see above), then one
       rounded addition of the balance */
    double ph = 0.0;
    for (int32_t i = 0; i < n; ++i) ph += (double)shares[i] * (double)p[i];
    const double V = b + ph;

    /* sells */
    double S = 0.0;
    for (int32_t i = 0; i < n; ++i) {
        int32_t k = orc_shares_from_action(action[i], cfg->hmax);
        if (k < 0) {
            int32_t s = -k < shares[i] ? -k : shares[i];
            shares[i] -= s;
            S += (double)p[i] * (double)s;
        }
    }
    double b_s = fma(S, f_s, b);

    /* buys, ascending stock index, largest affordable q <= k */
    double G = 0.0;
    for (int32_t i = 0; i < n; ++i) {
        int32_t k = orc_shares_from_action(action[i], cfg->hmax);
        if (k <= 0) continue;
        int32_t q = k;
        while (q > 0 && fma(f_b, G + (double)p[i] * (double)q, -b_s) > 0.0)
            --q;
        G += (double)p[i] * (double)q;
        shares[i] += q;
    }
    double nb = fma(-f_b, G, b_s);
    if (nb < 0.0) nb = 0.0;
    *cash = nb;
    *t += 1;

    double ph1 = 0.0;
    for (int32_t i = 0; i < n; ++i) ph1 += (double)shares[i] * (double)p1[i];
    const double V1 = nb + ph1;

    if (diag) { diag[0] = V; diag[1] = V1; diag[2] = S; diag[3] = G; diag[4] = b_s; }
    return (float)(cfg->reward_scale * (V1 - V));
}

/* Batched step over E envs (teacher forcing: the caller supplies the raw
 * actions [E][n]).  reward [E]; obs_next (fp32 or bf16 bits) [E][K_pad]
 * optional. */
void orc_env_step(const orc_market *m, const orc_env_cfg *cfg, int32_t E,
                  double *cash, int32_t *shares, int64_t *t,
                  const float *action, float *reward, int32_t K_pad,
                  float *obs_f32, uint16_t *obs_bf16)
{
    const int32_t n = m->n;
    for (int32_t e = 0; e < E; ++e) {
        const int ok = has_rows(m, t[e], 1);
        reward[e] = orc_env_step_one(m, cfg, &cash[e], &shares[(size_t)e * n],
                                     &t[e], &action[(size_t)e * n], NULL);
        if (ok) {
            orc_obs(m, cfg, t[e], cash[e], &shares[(size_t)e * n], K_pad,
                    obs_f32 ? obs_f32 + (size_t)e * K_pad : NULL,
                    obs_bf16 ? obs_bf16 + (size_t)e * K_pad : NULL);
        } else {
            for (int32_t k = 0; k < K_pad; ++k) {
                if (obs_f32) obs_f32[(size_t)e * K_pad + k] = NAN;
                if (obs_bf16) obs_bf16[(size_t)e * K_pad + k] = orc_bf16_bits(NAN);
            }
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Actor forward for one observation (PPO Gaussian policy mean; PPO is named in */
/* Section 5.2).  Reading: tanh hidden layers, linear output.               */
/*   y = W x + b accumulated in fp64 in input order, rounded to fp32;        */
/*   hidden: tanhf, then (bf16 configs) rounded to bf16;                     */
/*   bf16 configs use bf16-rounded copies of the fp32 master weights.        */
/* x holds the observation values as fp32 (bf16-exact for bf16 configs).    */
/* ------------------------------------------------------------------------ */

static void layer(const float *W, const float *b, int32_t out, int32_t in,
                  const float *x, float *y, int hidden, int bf16)
{
    for (int32_t o = 0; o < out; ++o) {
        double acc = 0.0;
        for (int32_t k = 0; k < in; ++k)
            acc += (double)W[(size_t)o * in + k] * (double)x[k];
        float v = (float)(acc + (double)b[o]);
        if (hidden) {
            v = tanhf(v);
            if (bf16) v = round_bf16(v);
        }
        y[o] = v;
    }
}

/* Weights already rounded (bf16 configs) by the caller. */
static void mlp_one(const float *const W[3], const float *const b[3],
                    const int32_t dims[4], int bf16, const float *x,
                    float *h1, float *h2, float *mu)
{
    layer(W[0], b[0], dims[1], dims[0], x, h1, 1, bf16);
    layer(W[1], b[1], dims[2], dims[1], h1, h2, 1, bf16);
    layer(W[2], b[2], dims[3], dims[2], h2, mu, 0, bf16);
}

static float *rounded_copy(const float *src, size_t count, int bf16)
{
    float *dst = (float *)malloc(count * sizeof(float));
    for (size_t i = 0; i < count; ++i) dst[i] = bf16 ? round_bf16(src[i]) : src[i];
    return dst;
}

/* mu [M][n] for M observations x [M][ld_x] (fp32 values) of one agent. */
void orc_mlp(const orc_actor *a, int32_t agent, int32_t M, const float *x,
             int32_t ld_x, float *mu)
{
    const int32_t *d = a->dims;
    const int32_t outs[3] = { d[1], d[2], d[3] }, ins[3] = { d[0], d[1], d[2] };
    float *W[3];
    const float *bb[3];
    for (int l = 0; l < 3; ++l) {
        size_t cnt = (size_t)outs[l] * ins[l];
        W[l] = rounded_copy(a->W[l] + (size_t)agent * cnt, cnt, a->bf16);
        bb[l] = a->b[l] + (size_t)agent * outs[l];
    }
    float *h1 = (float *)malloc(sizeof(float) * d[1]);
    float *h2 = (float *)malloc(sizeof(float) * d[2]);
    float *xin = (float *)malloc(sizeof(float) * d[0]);
    for (int32_t r = 0; r < M; ++r) {
        for (int32_t k = 0; k < d[0]; ++k) {
            float v = x[(size_t)r * ld_x + k];
            xin[k] = a->bf16 ? round_bf16(v) : v;
        }
        mlp_one((const float *const *)W, bb, d, a->bf16, xin, h1, h2,
                mu + (size_t)r * d[3]);
    }
    free(h1); free(h2); free(xin);
    for (int l = 0; l < 3; ++l) free(W[l]);
}

/* ------------------------------------------------------------------------ */
/* Rollout (one PPO worker pass over E envs for L steps; "batch mode",       */
/* Section 4.4).  For step j and env e (global id env_ids[e]):               */
/*   obs_j from the state -> mu = actor(obs_j) -> z = normals(seed,          */
/*   step0+j, env, agent) -> a = mu + exp(log_std) z,                        */
/*   logp = sum_i(-z_i^2/2 - log_std_i) - (n/2) ln(2 pi) -> env step with    */
/*   a (or, under teacher forcing, with the supplied action) -> reward,      */
/*   done = (step0 + j + 1 == horizon).                                      */
/* Outputs (each optional, time-major): obs [L][E][K_pad] (fp32 or bf16     */
/* bits), act [L][E][n], logp [L][E], reward [L][E], done [L][E],           */
/* cash_tap [L][E], shares_tap [L][E][n] (state after step j), mu [L][E][n], */
/* asset_tap [L][E] (total asset b + p^T h after step j, at the new prices;  */
/* NaN for an env that is not stepped).                                      */
/* ------------------------------------------------------------------------ */

typedef struct {
    float *obs_f32;
    uint16_t *obs_bf16;
    float *act;
    float *logp;
    float *reward;
    uint8_t *done;
    double *cash_tap;
    int32_t *shares_tap;
    float *mu;
    double *asset_tap;
} orc_traj;

void orc_rollout(const orc_market *m, const orc_env_cfg *cfg,
                 const orc_actor *a, int32_t E, const int32_t *env_ids,
                 double *cash, int32_t *shares, int64_t *t, uint64_t seed,
                 uint64_t step0, int32_t L, int32_t K_pad,
                 const float *teacher, orc_traj *tr)
{
    const int32_t n = m->n;
    const int32_t *d = a->dims;
    const int32_t outs[3] = { d[1], d[2], d[3] }, ins[3] = { d[0], d[1], d[2] };
    const double half_log_2pi_n = 0.5 * (double)n * log(2.0 * 3.14159265358979323846);

    /* bf16 copies of every agent's weights (or plain copies for fp32) */
    const int32_t A = a->n_agents;
    float **W = (float **)malloc(sizeof(float *) * 3 * (size_t)A);
    for (int32_t ag = 0; ag < A; ++ag)
        for (int l = 0; l < 3; ++l) {
            size_t cnt = (size_t)outs[l] * ins[l];
            W[3 * ag + l] = rounded_copy(a->W[l] + (size_t)ag * cnt, cnt, a->bf16);
        }

    /* an env without market rows for all L steps is not stepped: its
     * state stays, its rows hold NaN (done = 0, obs untouched) */
    uint8_t *active = (uint8_t *)malloc((size_t)E + 1);
    for (int32_t e = 0; e < E; ++e) active[e] = (uint8_t)has_rows(m, t[e], L);

    /* Envs share nothing, so each env runs its L steps on its own; the
     * OpenMP build (liboracle_omp.so, the CPU baseline over all cores) splits
     * the envs over threads, the plain build runs them one after another.
     * Either way every env sees the same operations in the same order. */
#pragma omp parallel
    {
    float *x = (float *)malloc(sizeof(float) * K_pad);
    uint16_t *xb = (uint16_t *)malloc(sizeof(uint16_t) * K_pad);
    float *h1 = (float *)malloc(sizeof(float) * d[1]);
    float *h2 = (float *)malloc(sizeof(float) * d[2]);
    float *mu = (float *)malloc(sizeof(float) * n);
    float *z = (float *)malloc(sizeof(float) * n);
    float *act = (float *)malloc(sizeof(float) * n);
#pragma omp for schedule(dynamic, 1)
    for (int32_t e = 0; e < E; ++e) {
        for (int32_t j = 0; j < L; ++j) {
            const uint32_t step = (uint32_t)(step0 + (uint64_t)j);
            const int32_t gid = env_ids ? env_ids[e] : e;
            const int32_t ag = gid / a->envs_per_agent;
            int32_t *h = &shares[(size_t)e * n];
            const size_t row = (size_t)j * E + e;
            if (!active[e]) {
                for (int32_t i = 0; i < n; ++i) {
                    if (tr->act) tr->act[row * n + i] = NAN;
                    if (tr->mu) tr->mu[row * n + i] = NAN;
                }
                if (tr->logp) tr->logp[row] = NAN;
                if (tr->reward) tr->reward[row] = NAN;
                if (tr->done) tr->done[row] = 0;
                if (tr->cash_tap) tr->cash_tap[row] = cash[e];
                if (tr->shares_tap) memcpy(tr->shares_tap + row * n, h, sizeof(int32_t) * n);
                if (tr->asset_tap) tr->asset_tap[row] = NAN;
                continue;
            }

            /* observation */
            orc_obs(m, cfg, t[e], cash[e], h, K_pad, x, a->bf16 ? xb : NULL);
            if (a->bf16)
                for (int32_t k = 0; k < K_pad; ++k) x[k] = orc_bf16_value(xb[k]);
            if (tr->obs_f32) memcpy(tr->obs_f32 + row * K_pad, x, sizeof(float) * K_pad);
            if (tr->obs_bf16) memcpy(tr->obs_bf16 + row * K_pad, xb, sizeof(uint16_t) * K_pad);

            /* actor */
            const float *Wa[3] = { W[3 * ag], W[3 * ag + 1], W[3 * ag + 2] };
            const float *ba[3] = { a->b[0] + (size_t)ag * d[1],
                                   a->b[1] + (size_t)ag * d[2],
                                   a->b[2] + (size_t)ag * d[3] };
            mlp_one(Wa, ba, d, a->bf16, x, h1, h2, mu);

            /* Gaussian sample */
            orc_normals(seed, step, (uint32_t)gid, (uint32_t)ag, n, z);
            const float *ls = a->log_std + (size_t)ag * n;
            double lp = 0.0;
            for (int32_t i = 0; i < n; ++i) {
                float sigma = expf(ls[i]);
                float sz = sigma * z[i];
                act[i] = mu[i] + sz;
                lp += -0.5 * (double)z[i] * (double)z[i] - (double)ls[i];
            }
            lp -= half_log_2pi_n;
            if (tr->act) memcpy(tr->act + row * n, act, sizeof(float) * n);
            if (tr->mu) memcpy(tr->mu + row * n, mu, sizeof(float) * n);
            if (tr->logp) tr->logp[row] = (float)lp;

            /* env step */
            const float *used = teacher ? teacher + row * n : act;
            float r = orc_env_step_one(m, cfg, &cash[e], h, &t[e], used, NULL);
            if (tr->reward) tr->reward[row] = r;
            if (tr->done)
                tr->done[row] = (uint8_t)((int64_t)(step0 + (uint64_t)j) + 1 == (int64_t)cfg->horizon);
            if (tr->cash_tap) tr->cash_tap[row] = cash[e];
            if (tr->shares_tap) memcpy(tr->shares_tap + row * n, h, sizeof(int32_t) * n);
            if (tr->asset_tap) {
                /* V = b + p_t^T h at the row the step moved to (eq. (2)'s
                   account value) */
                const float *p = price_row(m, t[e]);
                double ph = 0.0;
                for (int32_t i = 0; i < n; ++i) ph += (double)p[i] * (double)h[i];
                tr->asset_tap[row] = cash[e] + ph;
            }
        }
    }
    free(x); free(xb); free(h1); free(h2); free(mu); free(z); free(act);
    }
    free(active);
    for (int32_t i = 0; i < 3 * A; ++i) free(W[i]);
    free(W);
}

/* ------------------------------------------------------------------------ */
/* GAE / reward-to-go over one rollout (PPO's generalized advantage          */
/* estimator; gamma = 0.99 from Table 2, lambda a config value).  fp64:      */
/*   delta_j = r_j + gamma (1 - d_j) V_{j+1} - V_j                           */
/*   A_j     = delta_j + gamma lambda (1 - d_j) A_{j+1},   A_L = 0           */
/*   ret_j   = A_j + V_j                                                     */
/* r, d, adv, ret : [L][E]; V : [L+1][E] (row L is the bootstrap value).     */
/* ------------------------------------------------------------------------ */

void orc_gae(const float *r, const float *v, const uint8_t *d, int32_t L,
             int32_t E, float gamma, float lambda, float *adv, float *ret)
{
    const double g = (double)gamma, gl = (double)gamma * (double)lambda;
    for (int32_t e = 0; e < E; ++e) {
        double A = 0.0;
        for (int32_t j = L - 1; j >= 0; --j) {
            const size_t i = (size_t)j * E + e;
            const double nd = d[i] ? 0.0 : 1.0;
            const double delta = (double)r[i] + g * nd * (double)v[i + E] - (double)v[i];
            A = delta + gl * nd * A;
            adv[i] = (float)A;
            ret[i] = (float)(A + (double)v[i]);
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Backtest metrics of a total-asset series (Section 5.2, "Evaluation       */
/* metrics").  Per env e, V_0 = v0[e] and V_t = v[(t-1) E + e], t = 1..T:    */
/*   per-period returns  r_t = V_t / V_{t-1} - 1;                           */
/*   cumulative return   V_T / V_0 - 1;                                     */
/*   annual return       (V_T / V_0)^(P / T) - 1 (geometric, P periods a    */
/*                       year);                                             */
/*   annual volatility   s sqrt(P), s the sample standard deviation of r;   */
/*   Sharpe ratio        (mean(r) - rf / P) / s * sqrt(P) (0 when s = 0);   */
/*   max drawdown        max_t (max_{u<=t} V_u - V_t) / max_{u<=t} V_u.     */
/* out [E][5] = {cumulative, annual return, annual volatility, Sharpe,      */
/* max drawdown}.  T = 1 gives s = 0.                                        */
/* ------------------------------------------------------------------------ */

void orc_backtest_metrics(const double *v0, const double *v, int32_t T, int32_t E,
                          double periods_per_year, double risk_free, double *out)
{
    for (int32_t e = 0; e < E; ++e) {
        double *o = out + (size_t)e * 5;
        /* the series for this env */
        double *V = (double *)malloc(sizeof(double) * ((size_t)T + 1));
        V[0] = v0[e];
        for (int32_t t = 1; t <= T; ++t) V[t] = v[(size_t)(t - 1) * E + e];
        /* returns, their mean and sample standard deviation (two passes) */
        double mean = 0.0;
        for (int32_t t = 1; t <= T; ++t) mean += V[t] / V[t - 1] - 1.0;
        mean /= (double)T;
        double ss = 0.0;
        for (int32_t t = 1; t <= T; ++t) {
            const double d = (V[t] / V[t - 1] - 1.0) - mean;
            ss += d * d;
        }
        const double sd = T > 1 ? sqrt(ss / (double)(T - 1)) : 0.0;
        o[0] = V[T] / V[0] - 1.0;
        o[1] = pow(V[T] / V[0], periods_per_year / (double)T) - 1.0;
        o[2] = sd * sqrt(periods_per_year);
        o[3] = sd > 0.0 ? (mean - risk_free / periods_per_year) / sd * sqrt(periods_per_year) : 0.0;
        /* drawdown against the running peak */
        double peak = V[0], mdd = 0.0;
        for (int32_t t = 0; t <= T; ++t) {
            if (V[t] > peak) peak = V[t];
            const double dd = (peak - V[t]) / peak;
            if (dd > mdd) mdd = dd;
        }
        o[4] = mdd;
        free(V);
    }
}

/* ------------------------------------------------------------------------ */
/* Evolution layer (Section 4.2).                                            */
/*                                                                           */
/* Model ensemble: agent g is trained by K pods that differ only in their   */
/* random seeds; fusing gives every pod the mean of the agent's K parameter */
/* vectors.  params [N][K][P], in place; the mean is summed in fp64 over    */
/* k = 0..K-1 and rounded once.                                              */
/* ------------------------------------------------------------------------ */

void orc_ensemble_fuse(float *params, int32_t N, int32_t K, int64_t P)
{
    for (int32_t g = 0; g < N; ++g) {
        float *base = params + (size_t)g * K * P;
        for (int64_t p = 0; p < P; ++p) {
            double s = 0.0;
            for (int32_t k = 0; k < K; ++k) s += (double)base[(size_t)k * P + p];
            const float m = (float)(s / (double)K);
            for (int32_t k = 0; k < K; ++k) base[(size_t)k * P + p] = m;
        }
    }
}

/* Fitness (the objective J of eq. (1) as the evaluator's score): per agent */
/* g, the mean over its envs e of sum_j gamma^j r[j][e].  An env with a NaN */
/* reward (not stepped) is left out; an agent without stepped envs gets NaN.*/
void orc_fitness(const float *reward, int32_t L, int32_t E, int32_t A,
                 double gamma, double *fitness)
{
    const int32_t epa = E / A;
    for (int32_t g = 0; g < A; ++g) {
        double sum = 0.0;
        int32_t cnt = 0;
        for (int32_t e = g * epa; e < (g + 1) * epa; ++e) {
            double ret = 0.0, disc = 1.0;
            int ok = 1;
            for (int32_t j = 0; j < L; ++j) {
                const float r = reward[(size_t)j * E + e];
                if (isnan(r)) ok = 0;
                ret += disc * (double)r;
                disc *= gamma;
            }
            if (ok) {
                sum += ret;
                ++cnt;
            }
        }
        fitness[g] = cnt ? sum / (double)cnt : NAN;
    }
}

/* Keep-best bookkeeping of the evaluator: an agent whose fitness beats its */
/* best so far (a NaN best counts as beaten; a NaN fitness never beats)     */
/* takes it as the new best, its parameters become best_params and its     */
/* stall count resets; otherwise the stall count grows by one (a training   */
/* loop stops the agent once it reaches the patience: early stopping).      */
void orc_keep_best(const double *fitness, double *best, int32_t *stall,
                   const float *params, float *best_params, int32_t A, int64_t P)
{
    for (int32_t g = 0; g < A; ++g) {
        const int better = !isnan(fitness[g]) && (isnan(best[g]) || fitness[g] > best[g]);
        if (better) {
            best[g] = fitness[g];
            memcpy(best_params + (size_t)g * P, params + (size_t)g * P, sizeof(float) * (size_t)P);
            stall[g] = 0;
        } else {
            stall[g] += 1;
        }
    }
}

/* Selector (Section 4.2; the selection step of a genetic algorithm): rank  */
/* the N agents by fitness, descending, NaN last, ties to the lower index;  */
/* the `keep` best survive and the agent of rank r >= keep becomes a copy   */
/* of the survivor of rank (r - keep) mod keep.  rank [N] out; params       */
/* [N][P] in place.                                                          */
void orc_select(const double *fitness, float *params, int32_t N, int64_t P,
                int32_t keep, int32_t *rank)
{
    int32_t *order = (int32_t *)malloc(sizeof(int32_t) * (size_t)N);
    for (int32_t i = 0; i < N; ++i) order[i] = i;
    /* insertion sort by (fitness desc, NaN last, index asc) */
    for (int32_t a = 1; a < N; ++a) {
        const int32_t x = order[a];
        int32_t b = a - 1;
        while (b >= 0) {
            const int32_t y = order[b];
            const double fx = fitness[x], fy = fitness[y];
            int x_first;
            if (isnan(fx)) x_first = 0;
            else if (isnan(fy)) x_first = 1;
            else x_first = fx > fy;
            if (!x_first) break;
            order[b + 1] = y;
            --b;
        }
        order[b + 1] = x;
    }
    for (int32_t r = 0; r < N; ++r) rank[order[r]] = r;
    for (int32_t r = keep; r < N; ++r) {
        const int32_t dst = order[r], src = order[(r - keep) % keep];
        memcpy(params + (size_t)dst * P, params + (size_t)src * P, sizeof(float) * (size_t)P);
    }
    free(order);
}

/* Minibatch rows of the learner (the learner samples stored transitions,  */
/* Section 4.3; batch size from Table 2).  Draw i of update counter c for   */
/* agent g: w = word i%4 of Philox4x32-10(ctr = (i/4, c, g, 0x4D42),        */
/* key = seed); u = floor(w R / 2^32) is uniform over the agent's R = L epa */
/* stored transitions (steps j < L of envs g epa .. (g+1) epa - 1), and the */
/* row is j E + e with j = u / epa, e = g epa + u % epa.  With replacement.*/
void orc_minibatch_rows(uint64_t seed, uint64_t counter, int32_t n_updates, int32_t B,
                        int32_t L, int32_t E, int32_t agent, int32_t envs_per_agent,
                        int64_t *idx)
{
    const uint32_t key[2] = { (uint32_t)seed, (uint32_t)(seed >> 32) };
    const uint64_t R = (uint64_t)L * (uint64_t)envs_per_agent;
    for (int32_t u = 0; u < n_updates; ++u) {
        for (int32_t i = 0; i < B; ++i) {
            const uint32_t ctr[4] = { (uint32_t)(i / 4), (uint32_t)(counter + (uint64_t)u),
                                      (uint32_t)agent, 0x4D42u };
            uint32_t w[4];
            orc_philox4x32_10(ctr, key, w);
            const uint64_t draw = ((uint64_t)w[i % 4] * R) >> 32;
            const int64_t j = (int64_t)(draw / (uint64_t)envs_per_agent);
            const int64_t e = (int64_t)agent * envs_per_agent
                              + (int64_t)(draw % (uint64_t)envs_per_agent);
            idx[(size_t)u * B + i] = j * E + e;
        }
    }
}
