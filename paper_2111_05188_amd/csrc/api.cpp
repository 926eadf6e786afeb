// C-ABI entry points (include/tp.h): host-side argument checks, error
// reporting, parameter layout and kernel dispatch.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <map>
#include <mutex>
#include <string>

#include "internal.hpp"
#include "tp.h"

using namespace tpk;

namespace {

thread_local std::string g_err;

int fail(int code, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int ok()
{
    g_err.clear();
    return TP_OK;
}

int hip_fail(hipError_t e, const char *what)
{
    return fail(TP_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

int check_market(const tp_market *m)
{
    if (!m) return fail(TP_EINVAL, "market is NULL");
    if (!m->price) return fail(TP_EINVAL, "market.price is NULL");
    if (m->n < 1 || m->n > 128) return fail(TP_EINVAL, "market.n = %d outside 1..128", m->n);
    if (m->n_ind < 0) return fail(TP_EINVAL, "market.n_ind = %d < 0", m->n_ind);
    if ((int64_t)m->n * m->n_ind > 1024)
        return fail(TP_EUNSUPPORTED, "market.n * n_ind = %lld > 1024", (long long)m->n * m->n_ind);
    if (m->n_ind > 0 && !m->ind) return fail(TP_EINVAL, "market.ind is NULL");
    if (m->T1 < 2) return fail(TP_EINVAL, "market.T1 = %lld < 2", (long long)m->T1);
    if (!aligned(m->price, 4) || !aligned(m->ind, 4))
        return fail(TP_EINVAL, "market arrays are not 4-byte aligned");
    return TP_OK;
}

int check_cfg(const tp_env_cfg *c)
{
    if (!c) return fail(TP_EINVAL, "env cfg is NULL");
    if (c->hmax < 1 || c->hmax > 128) return fail(TP_EINVAL, "cfg.hmax = %d outside 1..128", c->hmax);
    if (c->horizon < 1) return fail(TP_EINVAL, "cfg.horizon = %d < 1", c->horizon);
    if (!(c->fee >= 0.0 && c->fee < 1.0)) return fail(TP_EINVAL, "cfg.fee = %g outside [0,1)", c->fee);
    if (!(c->cash0 >= 0.0) || !std::isfinite(c->cash0))
        return fail(TP_EINVAL, "cfg.cash0 = %g is negative or not finite", c->cash0);
    if (!std::isfinite(c->reward_scale)) return fail(TP_EINVAL, "cfg.reward_scale is not finite");
    if (!std::isfinite(c->cash_scale) || !std::isfinite(c->price_scale) ||
        !std::isfinite(c->share_scale))
        return fail(TP_EINVAL, "cfg observation scales are not finite");
    return TP_OK;
}

int check_state(const tp_env_state *s, int n)
{
    if (!s) return fail(TP_EINVAL, "state is NULL");
    if (s->E < 1) return fail(TP_EINVAL, "state.E = %d < 1", s->E);
    if (!s->cash || !s->shares || !s->t) return fail(TP_EINVAL, "state array is NULL");
    if (!aligned(s->cash, 8) || !aligned(s->t, 8) || !aligned(s->shares, 4) ||
        !aligned(s->n_invalid, 4))
        return fail(TP_EINVAL, "state arrays are not naturally aligned");
    (void)n;
    return TP_OK;
}

int K_pad_of(const tp_market *m) { return (1 + 2 * m->n + m->n * m->n_ind + 31) / 32 * 32; }

int check_obs(const void *obs, int64_t ld, int dtype, int K_pad, const char *what)
{
    if (!obs) return TP_OK;
    if (dtype != TP_F32 && dtype != TP_BF16) return fail(TP_EINVAL, "%s: bad dtype %d", what, dtype);
    if (ld < K_pad || ld % 8 != 0)
        return fail(TP_EINVAL, "%s: ld_obs = %lld must be >= K_pad = %d and a multiple of 8", what,
                    (long long)ld, K_pad);
    if (!aligned(obs, 16)) return fail(TP_EINVAL, "%s: not 16-byte aligned", what);
    return TP_OK;
}

EnvConst make_env(const tp_market *m, const tp_env_cfg *c)
{
    EnvConst e;
    e.price = m->price;
    e.ind = m->ind;
    e.T1 = m->T1;
    e.n = m->n;
    e.nI = m->n * m->n_ind;
    e.K_pad = K_pad_of(m);
    e.hmax = c->hmax;
    e.horizon = c->horizon;
    e.f_s = 1.0 - c->fee;
    e.f_b = 1.0 + c->fee;
    e.reward_scale = c->reward_scale;
    e.cash0 = c->cash0;
    e.cash_scale = c->cash_scale;
    e.price_scale = c->price_scale;
    e.share_scale = c->share_scale;
    return e;
}

struct PackSig {
    int dims[4], dtype, n_agents;
    size_t total;
};

// Packed buffers filled by tp_actor_pack / tp_critic_pack, keyed by their
// device address, with the shape they hold (guarded by g_mu).  A buffer is
// forgotten by tp_*_release, or when a later pack writes over any of its
// bytes (the caller has freed it and the allocator handed out the memory
// again).
std::mutex g_mu;
std::map<const void *, PackSig> g_packed;

int check_actor(const tp_actor *a, PackedLayout *lay)
{
    if (!a) return fail(TP_EINVAL, "actor is NULL");
    if (a->n_agents < 1 || a->envs_per_agent < 1)
        return fail(TP_EINVAL, "actor.n_agents = %d, envs_per_agent = %d must be >= 1", a->n_agents,
                    a->envs_per_agent);
    if (a->dtype != TP_F32 && a->dtype != TP_BF16)
        return fail(TP_EINVAL, "actor.dtype = %d", a->dtype);
    for (int l = 0; l < 3; ++l)
        if (!a->W[l] || !a->b[l]) return fail(TP_EINVAL, "actor W[%d] or b[%d] is NULL", l, l);
    if (!a->log_std) return fail(TP_EINVAL, "actor.log_std is NULL");
    if (a->agent_stride < 0) return fail(TP_EINVAL, "actor.agent_stride < 0");
    const int S = a->dims[0], H1 = a->dims[1], H2 = a->dims[2], n = a->dims[3];
    if (S < 1 || H1 < 1 || H2 < 1 || n < 1 || n > 128)
        return fail(TP_EINVAL, "actor dims {%d,%d,%d,%d} invalid", S, H1, H2, n);
    if (a->dtype == TP_BF16 && (H1 % 128 || H2 % 128))
        return fail(TP_EUNSUPPORTED, "bf16 actor needs H1, H2 multiples of 128 (got %d, %d)", H1, H2);
    if (a->dtype == TP_F32 && (H1 % 4 || H2 % 4))
        return fail(TP_EUNSUPPORTED, "fp32 actor needs H1, H2 multiples of 4 (got %d, %d)", H1, H2);
    if (!packed_layout(a, lay)) return fail(TP_EINVAL, "actor layout failed");
    return TP_OK;
}

struct CriticSig {
    int dims[3], dtype, n_agents;
    size_t total;
};

std::map<const void *, CriticSig> g_packed_critic;

// Forget every recorded buffer that overlaps [p, p + bytes) (g_mu held).
template <class M>
void forget_overlapping(M &m, const void *p, size_t bytes)
{
    const uintptr_t lo = (uintptr_t)p, hi = lo + bytes;
    for (auto it = m.begin(); it != m.end();) {
        const uintptr_t a = (uintptr_t)it->first, b = a + it->second.total;
        if (a < hi && lo < b)
            it = m.erase(it);
        else
            ++it;
    }
}

void forget_all_overlapping(const void *p, size_t bytes)
{
    forget_overlapping(g_packed, p, bytes);
    forget_overlapping(g_packed_critic, p, bytes);
}

int check_ppo(const tp_ppo *c, PpoLayout *lay)
{
    if (!c) return fail(TP_EINVAL, "learner configuration is NULL");
    const int32_t *d = c->dims;
    if (c->dtype != TP_BF16 && c->dtype != TP_F32)
        return fail(TP_EINVAL, "learner dtype %d", c->dtype);
    if (d[0] < 1 || d[3] < 1 || d[3] > 128)
        return fail(TP_EINVAL, "learner S = %d, n = %d (need S >= 1, 1 <= n <= 128)", d[0], d[3]);
    for (int i : {1, 2, 4, 5})
        if (d[i] < 32 || d[i] % 32)
            return fail(TP_EINVAL, "learner hidden width dims[%d] = %d: positive multiples of 32",
                        i, d[i]);
    if (c->batch < 32 || c->batch % 32)
        return fail(TP_EINVAL, "learner batch = %d: a positive multiple of 32", c->batch);
    if (!(c->clip > 0.f && c->clip < 1.f)) return fail(TP_EINVAL, "clip = %g", c->clip);
    if (!(c->ent_coef >= 0.f)) return fail(TP_EINVAL, "ent_coef = %g", c->ent_coef);
    if (!(c->lr > 0.f)) return fail(TP_EINVAL, "lr = %g", c->lr);
    if (!(c->beta1 >= 0.f && c->beta1 < 1.f) || !(c->beta2 >= 0.f && c->beta2 < 1.f))
        return fail(TP_EINVAL, "Adam betas %g, %g outside [0, 1)", c->beta1, c->beta2);
    if (!(c->eps > 0.f)) return fail(TP_EINVAL, "Adam eps = %g", c->eps);
    ppo_layout(c, lay);
    return TP_OK;
}

int check_critic(const tp_critic *c, CriticLayout *lay)
{
    if (!c) return fail(TP_EINVAL, "critic is NULL");
    if (c->n_agents < 1 || c->envs_per_agent < 1)
        return fail(TP_EINVAL, "critic.n_agents = %d, envs_per_agent = %d must be >= 1",
                    c->n_agents, c->envs_per_agent);
    if (c->dtype != TP_F32 && c->dtype != TP_BF16)
        return fail(TP_EINVAL, "critic.dtype = %d", c->dtype);
    for (int l = 0; l < 3; ++l)
        if (!c->W[l] || !c->b[l]) return fail(TP_EINVAL, "critic W[%d] or b[%d] is NULL", l, l);
    if (c->agent_stride < 0) return fail(TP_EINVAL, "critic.agent_stride < 0");
    const int S = c->dims[0], H1 = c->dims[1], H2 = c->dims[2];
    if (S < 1 || H1 < 1 || H2 < 1 || S > 65536 || H1 > 4096 || H2 > 4096)
        return fail(TP_EINVAL, "critic dims {%d,%d,%d} invalid", S, H1, H2);
    if (H1 % 4 || H2 % 4)
        return fail(TP_EUNSUPPORTED, "critic needs H1, H2 multiples of 4 (got %d, %d)", H1, H2);
    critic_layout(c, lay);
    if (!lay->mfma && (size_t)16 * (lay->K_pad + H1 + 256) * 4 > LDS_LIMIT)
        return fail(TP_EUNSUPPORTED, "critic {%d,%d,%d} exceeds the generic kernel's working set",
                    S, H1, H2);
    return TP_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// packed parameter layout
// ---------------------------------------------------------------------------
namespace tpk {

bool packed_layout(const tp_actor *a, PackedLayout *L)
{
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    L->dtype = a->dtype;
    L->S = a->dims[0];
    L->H1 = a->dims[1];
    L->H2 = a->dims[2];
    L->n = a->dims[3];
    L->K_pad = (L->S + 31) / 32 * 32;
    // bf16: layer-1 inputs padded to whole pipeline rounds (4 k-steps of 32)
    const int K1 = a->dtype == TP_BF16 ? (L->S + 127) / 128 * 128 : L->K_pad;
    const int ins[3] = {K1, L->H1, L->H2};
    const int outs[3] = {L->H1, L->H2, L->n};
    size_t off = 0;
    for (int l = 0; l < 3; ++l) {
        size_t wbytes;
        if (a->dtype == TP_BF16) {
            L->NT[l] = (outs[l] + 15) / 16;
            // action tiles in whole groups of 4 (one per matrix wave)
            if (l == 2) L->NT[l] = (L->NT[l] + 3) / 4 * 4;
            L->KS[l] = ins[l] / 32;
            wbytes = (size_t)L->NT[l] * L->KS[l] * 64 * 16;
        } else {
            L->NT[l] = outs[l];
            L->KS[l] = ins[l] / 4;
            wbytes = (size_t)L->KS[l] * outs[l] * 16;
        }
        L->off_W[l] = off;
        // guard: the MFMA pipeline reads up to 4 k-steps (4 KiB per wave
        // lane group) past a layer's last fragment
        off = al(off + wbytes + (a->dtype == TP_BF16 ? 4 * 1024 : 0));
    }
    for (int l = 0; l < 3; ++l) {
        const int padded = a->dtype == TP_BF16 ? L->NT[l] * 16 : outs[l];
        L->off_b[l] = off;
        off = al(off + (size_t)padded * 4);
    }
    L->off_ls = off;
    off = al(off + (size_t)(a->dtype == TP_BF16 ? L->NT[2] * 16 : L->n) * 4);
    L->agent_stride = off;
    L->total = off * (size_t)a->n_agents;
    return true;
}

bool critic_layout(const tp_critic *c, CriticLayout *L)
{
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    L->dtype = c->dtype;
    L->S = c->dims[0];
    L->H1 = c->dims[1];
    L->H2 = c->dims[2];
    L->K_pad = (L->S + 31) / 32 * 32;
    L->mfma = critic_mfma_shape(*L);
    size_t off = 0;
    const int outs[2] = {L->H1, L->H2}, ins[2] = {L->K_pad, L->H1};
    for (int l = 0; l < 2; ++l) {
        L->NT[l] = (outs[l] + 15) / 16;
        L->KS[l] = ins[l] / 32;
        const size_t wbytes = L->mfma ? (size_t)L->NT[l] * L->KS[l] * 64 * 16
                                      : (size_t)ins[l] * outs[l] * 4;
        L->off_W[l] = off;
        off = al(off + wbytes);
    }
    L->off_W[2] = off;
    off = al(off + (size_t)L->H2 * 4);
    L->off_b[0] = off;
    off = al(off + (size_t)L->H1 * 4);
    L->off_b[1] = off;
    off = al(off + (size_t)L->H2 * 4);
    L->off_b[2] = off;
    off = al(off + 4);
    L->agent_stride = off;
    L->total = off * (size_t)c->n_agents;
    return true;
}

}  // namespace tpk

// ---------------------------------------------------------------------------
// entry points
// ---------------------------------------------------------------------------
extern "C" {

const char *tp_last_error(void) { return g_err.c_str(); }

int tp_version(void) { return TP_VERSION; }

int tp_actor_release(const void *packed)
{
    std::lock_guard<std::mutex> g(g_mu);
    if (!g_packed.erase(packed)) return fail(TP_EINVAL, "%p is not a packed actor buffer", packed);
    return ok();
}

int tp_critic_release(const void *packed)
{
    std::lock_guard<std::mutex> g(g_mu);
    if (!g_packed_critic.erase(packed))
        return fail(TP_EINVAL, "%p is not a packed critic buffer", packed);
    return ok();
}

int tp_check_starts(const int64_t *t0_host, int32_t E, int64_t T1, int32_t L)
{
    if (!t0_host) return fail(TP_EINVAL, "t0_host is NULL");
    if (E < 1 || L < 1 || T1 < 2)
        return fail(TP_EINVAL, "E = %d, L = %d, T1 = %lld (need E, L >= 1, T1 >= 2)", E, L,
                    (long long)T1);
    for (int32_t e = 0; e < E; ++e) {
        const int64_t t0 = t0_host[e];
        if (t0 < 0 || t0 > T1 - 1 - L)
            return fail(TP_ERANGE,
                        "env %d starts at row %lld: %d steps need rows up to %lld of %lld", e,
                        (long long)t0, L, (long long)t0 + L, (long long)T1);
    }
    return ok();
}

int tp_env_reset(const tp_market *mkt, const tp_env_cfg *cfg, const tp_env_state *st,
                 const int64_t *t0, void *obs0, int64_t ld_obs, int32_t obs_dtype, void *stream)
{
    int rc;
    if ((rc = check_market(mkt)) || (rc = check_cfg(cfg)) || (rc = check_state(st, mkt->n)))
        return rc;
    if (!t0 || !aligned(t0, 8)) return fail(TP_EINVAL, "t0 is NULL or misaligned");
    if ((rc = check_obs(obs0, ld_obs, obs_dtype, K_pad_of(mkt), "obs0"))) return rc;
    const EnvConst c = make_env(mkt, cfg);
    hipError_t e = launch_env_reset(c, st->cash, st->shares, st->t, t0, st->E, obs0, ld_obs,
                                    obs_dtype == TP_BF16, st->n_invalid, (hipStream_t)stream);
    if (e == hipErrorInvalidConfiguration)
        return fail(TP_EUNSUPPORTED, "observation rows of K_pad = %d exceed the LDS limit", c.K_pad);
    if (e != hipSuccess) return hip_fail(e, "env_reset launch");
    return ok();
}

int tp_env_step(const tp_market *mkt, const tp_env_cfg *cfg, const tp_env_state *st,
                const float *action, float *reward, void *obs_next, int64_t ld_obs,
                int32_t obs_dtype, void *stream)
{
    int rc;
    if ((rc = check_market(mkt)) || (rc = check_cfg(cfg)) || (rc = check_state(st, mkt->n)))
        return rc;
    if (!action || !reward) return fail(TP_EINVAL, "action or reward is NULL");
    if (!aligned(action, 4) || !aligned(reward, 4))
        return fail(TP_EINVAL, "action or reward misaligned");
    if ((rc = check_obs(obs_next, ld_obs, obs_dtype, K_pad_of(mkt), "obs_next"))) return rc;
    const EnvConst c = make_env(mkt, cfg);
    hipError_t e = launch_env_step(c, st->cash, st->shares, st->t, action, reward, st->E, obs_next,
                                   ld_obs, obs_dtype == TP_BF16, st->n_invalid,
                                   (hipStream_t)stream);
    if (e == hipErrorInvalidConfiguration)
        return fail(TP_EUNSUPPORTED, "observation rows of K_pad = %d exceed the LDS limit", c.K_pad);
    if (e != hipSuccess) return hip_fail(e, "env_step launch");
    return ok();
}

size_t tp_actor_packed_bytes(const tp_actor *actor)
{
    PackedLayout L;
    if (check_actor(actor, &L)) return 0;
    g_err.clear();
    return L.total;
}

int tp_actor_pack(const tp_actor *actor, void *packed, size_t packed_bytes, void *stream)
{
    PackedLayout L;
    int rc;
    if ((rc = check_actor(actor, &L))) return rc;
    if (!packed || !aligned(packed, 256)) return fail(TP_EINVAL, "packed is NULL or not 256-byte aligned");
    if (packed_bytes < L.total)
        return fail(TP_EINVAL, "packed_bytes = %zu < required %zu", packed_bytes, L.total);
    hipError_t e = launch_pack(actor, L, packed, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "pack launch");
    {
        std::lock_guard<std::mutex> g(g_mu);
        PackSig sig;
        for (int i = 0; i < 4; ++i) sig.dims[i] = actor->dims[i];
        sig.dtype = actor->dtype;
        sig.n_agents = actor->n_agents;
        sig.total = L.total;
        forget_all_overlapping(packed, L.total);
        g_packed[packed] = sig;
    }
    return ok();
}

int tp_rollout_path(const tp_market *mkt, const tp_actor *actor)
{
    PackedLayout lay;
    int rc = check_market(mkt);
    if (rc != TP_OK) return rc;
    if ((rc = check_actor(actor, &lay)) != TP_OK) return rc;
    ok();
    return rollout_rs_shape(lay, mkt->n * mkt->n_ind) ? 1 : 0;
}

int tp_rollout(const tp_market *mkt, const tp_env_cfg *cfg, const tp_env_state *st,
               const tp_actor *actor, const void *packed, size_t packed_bytes, uint64_t seed,
               uint64_t step0, int32_t L, const tp_traj *traj, void *stream)
{
    int rc;
    PackedLayout lay;
    if ((rc = check_market(mkt)) || (rc = check_cfg(cfg)) || (rc = check_state(st, mkt->n)) ||
        (rc = check_actor(actor, &lay)))
        return rc;
    const int n = mkt->n, S = 1 + 2 * n + n * mkt->n_ind;
    if (actor->dims[0] != S || actor->dims[3] != n)
        return fail(TP_EINVAL, "actor dims {%d,..,%d} do not match the market (S = %d, n = %d)",
                    actor->dims[0], actor->dims[3], S, n);
    if ((int64_t)actor->n_agents * actor->envs_per_agent != st->E)
        return fail(TP_EINVAL, "n_agents * envs_per_agent = %lld != E = %d",
                    (long long)actor->n_agents * actor->envs_per_agent, st->E);
    if (L < 1) return fail(TP_EINVAL, "L = %d < 1", L);
    if (step0 + (uint64_t)L > (uint64_t)cfg->horizon)
        return fail(TP_ERANGE, "step0 + L = %llu exceeds the horizon %d",
                    (unsigned long long)(step0 + L), cfg->horizon);
    if (!traj) return fail(TP_EINVAL, "traj is NULL");
    if (!traj->action || !traj->logp || !traj->reward || !traj->done)
        return fail(TP_EINVAL, "traj.action/logp/reward/done must not be NULL");
    if (!aligned(traj->action, 4) || !aligned(traj->logp, 4) || !aligned(traj->reward, 4) ||
        !aligned(traj->cash_tap, 8) || !aligned(traj->shares_tap, 4) ||
        !aligned(traj->asset_tap, 8) || !aligned(traj->mu_tap, 4))
        return fail(TP_EINVAL, "traj arrays are not naturally aligned");
    const int K_pad = K_pad_of(mkt);
    if ((rc = check_obs(traj->obs, traj->ld_obs, actor->dtype, K_pad, "traj.obs")) ||
        (rc = check_obs(traj->obs_last, traj->ld_obs, actor->dtype, K_pad, "traj.obs_last")))
        return rc;
    if (!packed) return fail(TP_EINVAL, "packed is NULL");
    {
        std::lock_guard<std::mutex> g(g_mu);
        auto it = g_packed.find(packed);
        if (it == g_packed.end())
            return fail(TP_EINVAL, "packed buffer was not filled by tp_actor_pack");
        const PackSig &sg = it->second;
        for (int i = 0; i < 4; ++i)
            if (sg.dims[i] != actor->dims[i])
                return fail(TP_EINVAL, "packed buffer holds a different actor shape");
        if (sg.dtype != actor->dtype || sg.n_agents != actor->n_agents)
            return fail(TP_EINVAL, "packed buffer holds a different dtype / agent count");
    }
    if (packed_bytes < lay.total)
        return fail(TP_EINVAL, "packed_bytes = %zu < required %zu", packed_bytes, lay.total);

    RolloutArgs a{};
    a.env = make_env(mkt, cfg);
    a.cash = st->cash;
    a.shares = st->shares;
    a.t = st->t;
    a.E = st->E;
    a.packed = (const uint8_t *)packed;
    a.lay = lay;
    a.n_agents = actor->n_agents;
    a.envs_per_agent = actor->envs_per_agent;
    a.key_lo = (uint32_t)seed;
    a.key_hi = (uint32_t)(seed >> 32);
    a.step0 = step0;
    a.L = L;
    a.obs = traj->obs;
    a.ld_obs = traj->ld_obs;
    a.action = traj->action;
    a.logp = traj->logp;
    a.reward = traj->reward;
    a.done = traj->done;
    a.cash_tap = traj->cash_tap;
    a.shares_tap = traj->shares_tap;
    a.obs_last = traj->obs_last;
    a.asset_tap = traj->asset_tap;
    a.mu_tap = traj->mu_tap;
    a.n_invalid = st->n_invalid;
    hipError_t e = launch_rollout(a, (hipStream_t)stream);
    if (e == hipErrorInvalidConfiguration)
        return fail(TP_EUNSUPPORTED, "rollout working set (%zu bytes of LDS) exceeds the limit",
                    a.lds_bytes);
    if (e != hipSuccess) return hip_fail(e, "rollout launch");
    return ok();
}

size_t tp_critic_packed_bytes(const tp_critic *critic)
{
    CriticLayout L;
    if (check_critic(critic, &L)) return 0;
    g_err.clear();
    return L.total;
}

int tp_critic_pack(const tp_critic *critic, void *packed, size_t packed_bytes, void *stream)
{
    CriticLayout L;
    int rc;
    if ((rc = check_critic(critic, &L))) return rc;
    if (!packed || !aligned(packed, 256)) return fail(TP_EINVAL, "packed is NULL or not 256-byte aligned");
    if (packed_bytes < L.total)
        return fail(TP_EINVAL, "packed_bytes = %zu < required %zu", packed_bytes, L.total);
    hipError_t e = launch_critic_pack(critic, L, packed, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "critic pack launch");
    {
        std::lock_guard<std::mutex> g(g_mu);
        CriticSig sig;
        for (int i = 0; i < 3; ++i) sig.dims[i] = critic->dims[i];
        sig.dtype = critic->dtype;
        sig.n_agents = critic->n_agents;
        sig.total = L.total;
        forget_all_overlapping(packed, L.total);
        g_packed_critic[packed] = sig;
    }
    return ok();
}

int tp_critic_value(const tp_critic *critic, const void *packed, size_t packed_bytes,
                    const void *obs, int64_t ld_obs, int64_t T, int32_t E, float *value,
                    void *stream)
{
    CriticLayout L;
    int rc;
    if ((rc = check_critic(critic, &L))) return rc;
    if (T < 1 || E < 1) return fail(TP_EINVAL, "T = %lld, E = %d must be >= 1", (long long)T, E);
    if ((int64_t)critic->n_agents * critic->envs_per_agent != E)
        return fail(TP_EINVAL, "n_agents * envs_per_agent = %lld != E = %d",
                    (long long)critic->n_agents * critic->envs_per_agent, E);
    if (!obs || !aligned(obs, 16)) return fail(TP_EINVAL, "obs is NULL or not 16-byte aligned");
    if (ld_obs < L.K_pad || ld_obs % 8)
        return fail(TP_EINVAL, "ld_obs = %lld must be >= K_pad = %d and a multiple of 8",
                    (long long)ld_obs, L.K_pad);
    if (!value || !aligned(value, 4)) return fail(TP_EINVAL, "value is NULL or misaligned");
    if (!packed) return fail(TP_EINVAL, "packed is NULL");
    {
        std::lock_guard<std::mutex> g(g_mu);
        auto it = g_packed_critic.find(packed);
        if (it == g_packed_critic.end())
            return fail(TP_EINVAL, "packed buffer was not filled by tp_critic_pack");
        const CriticSig &sg = it->second;
        for (int i = 0; i < 3; ++i)
            if (sg.dims[i] != critic->dims[i])
                return fail(TP_EINVAL, "packed buffer holds a different critic shape");
        if (sg.dtype != critic->dtype || sg.n_agents != critic->n_agents)
            return fail(TP_EINVAL, "packed buffer holds a different dtype / agent count");
    }
    if (packed_bytes < L.total)
        return fail(TP_EINVAL, "packed_bytes = %zu < required %zu", packed_bytes, L.total);
    CriticArgs a;
    a.packed = (const uint8_t *)packed;
    a.lay = L;
    a.obs = obs;
    a.ld_obs = ld_obs;
    a.T = T;
    a.E = E;
    a.n_agents = critic->n_agents;
    a.envs_per_agent = critic->envs_per_agent;
    a.value = value;
    hipError_t e = launch_critic_value(a, (hipStream_t)stream);
    if (e == hipErrorInvalidConfiguration)
        return fail(TP_EUNSUPPORTED, "critic launch exceeds the grid or LDS limits");
    if (e != hipSuccess) return hip_fail(e, "critic launch");
    return ok();
}

size_t tp_backtest_metrics_work_bytes(int32_t T, int32_t E)
{
    if (T < 1 || E < 1 || E > 64 * 65535) {
        fail(TP_EINVAL, "T = %d, E = %d (1 <= E <= %d)", T, E, 64 * 65535);
        return 0;
    }
    ok();
    return backtest_metrics_work_bytes(T, E);
}

int tp_backtest_metrics(const double *v0, const double *v, int32_t T, int32_t E,
                        double periods_per_year, double risk_free, double *out, void *work,
                        size_t work_bytes, void *stream)
{
    if (!v0 || !v || !out || !work) return fail(TP_EINVAL, "a metrics array is NULL");
    if (!aligned(v0, 8) || !aligned(v, 8) || !aligned(out, 8) || !aligned(work, 8))
        return fail(TP_EINVAL, "metrics arrays are not 8-byte aligned");
    if (T < 1 || E < 1 || E > 64 * 65535)
        return fail(TP_EINVAL, "T = %d, E = %d (1 <= E <= %d)", T, E, 64 * 65535);
    if (work_bytes < backtest_metrics_work_bytes(T, E))
        return fail(TP_EINVAL, "metrics workspace of %zu bytes, %zu needed", work_bytes,
                    backtest_metrics_work_bytes(T, E));
    if (!(periods_per_year > 0.0))
        return fail(TP_EINVAL, "periods_per_year = %g must be > 0", periods_per_year);
    if (!std::isfinite(risk_free)) return fail(TP_EINVAL, "risk_free = %g", risk_free);
    hipError_t e = launch_backtest_metrics(v0, v, T, E, periods_per_year, risk_free, out, work,
                                           (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "metrics launch");
    return ok();
}

int tp_backtest_metrics_noalloc(const double *v0, const double *v, int32_t T, int32_t E,
                                double periods_per_year, double risk_free, double *out,
                                void *stream)
{
    if (!v0 || !v || !out) return fail(TP_EINVAL, "a metrics array is NULL");
    if (!aligned(v0, 8) || !aligned(v, 8) || !aligned(out, 8))
        return fail(TP_EINVAL, "metrics arrays are not 8-byte aligned");
    if (T < 1 || E < 1 || E > 64 * 65535)
        return fail(TP_EINVAL, "T = %d, E = %d (1 <= E <= %d)", T, E, 64 * 65535);
    if (!(periods_per_year > 0.0))
        return fail(TP_EINVAL, "periods_per_year = %g must be > 0", periods_per_year);
    if (!std::isfinite(risk_free)) return fail(TP_EINVAL, "risk_free = %g", risk_free);
    const size_t need = backtest_metrics_scratch_needed(T, E);
    if (need > backtest_metrics_scratch_capacity())
        return fail(TP_EUNSUPPORTED, "T = %d, E = %d needs %zu bytes of scratch; the static "
                    "scratch holds %zu (use tp_backtest_metrics with a workspace)", T, E, need,
                    backtest_metrics_scratch_capacity());
    void *work = nullptr;
    hipError_t e = backtest_metrics_scratch(&work);
    if (e != hipSuccess) return hip_fail(e, "metrics scratch address");
    e = launch_backtest_metrics(v0, v, T, E, periods_per_year, risk_free, out, work,
                                (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "metrics launch");
    return ok();
}

int64_t tp_ppo_param_count(const tp_ppo *cfg)
{
    PpoLayout L;
    if (check_ppo(cfg, &L) != TP_OK) return 0;
    ok();
    return L.P;
}

size_t tp_ppo_workspace_bytes(const tp_ppo *cfg)
{
    PpoLayout L;
    if (check_ppo(cfg, &L) != TP_OK) return 0;
    ok();
    return L.total;
}

int tp_ppo_update_agents(const tp_ppo *cfg, int32_t n_agents, int64_t agent_stride,
                         float *params, float *adam_m, float *adam_v, int64_t step0,
                         int32_t n_updates, const void *obs, int64_t ld_obs, const float *action,
                         const float *logp, const float *adv, const float *ret, int64_t rows,
                         const int64_t *idx, float *grad, double *stats, void *workspace,
                         size_t workspace_bytes, void *stream)
{
    PpoArgs a{};
    int rc = check_ppo(cfg, &a.lay);
    if (rc != TP_OK) return rc;
    if (n_agents < 1 || n_agents > 1024)
        return fail(TP_EINVAL, "n_agents = %d outside [1, 1024]", n_agents);
    if (n_agents > 1 && agent_stride < a.lay.P)
        return fail(TP_EINVAL, "agent_stride = %lld < P = %lld: agents would overlap",
                    (long long)agent_stride, (long long)a.lay.P);
    if (!params || !adam_m || !adam_v || !obs || !action || !logp || !adv || !ret || !idx ||
        !workspace)
        return fail(TP_EINVAL, "a learner array is NULL");
    if (!aligned(params, 4) || !aligned(adam_m, 4) || !aligned(adam_v, 4) ||
        !aligned(obs, cfg->dtype == TP_BF16 ? 2 : 4) || !aligned(action, 4) ||
        !aligned(logp, 4) || !aligned(adv, 4) || !aligned(ret, 4) || !aligned(idx, 8) ||
        (grad && !aligned(grad, 4)) || (stats && !aligned(stats, 8)))
        return fail(TP_EINVAL, "learner arrays are misaligned");
    if (!aligned(workspace, 256)) return fail(TP_EINVAL, "workspace must be 256-byte aligned");
    if (workspace_bytes / (size_t)n_agents < a.lay.total)
        return fail(TP_EINVAL, "workspace of %zu bytes, %zu needed", workspace_bytes,
                    a.lay.total * (size_t)n_agents);
    if (step0 < 1) return fail(TP_EINVAL, "step0 = %lld must be >= 1", (long long)step0);
    if (n_updates < 1) return fail(TP_EINVAL, "n_updates = %d must be >= 1", n_updates);
    if (rows < 1) return fail(TP_EINVAL, "rows = %lld must be >= 1", (long long)rows);
    if (ld_obs < cfg->dims[0])
        return fail(TP_EINVAL, "ld_obs = %lld < S = %d", (long long)ld_obs, cfg->dims[0]);
    a.n_agents = n_agents;
    a.agent_stride = n_agents > 1 ? agent_stride : a.lay.P;
    a.ws_stride = (int64_t)a.lay.total;
    a.params = params;
    a.adam_m = adam_m;
    a.adam_v = adam_v;
    a.step0 = step0;
    a.n_updates = n_updates;
    a.obs = obs;
    a.ld_obs = ld_obs;
    a.action = action;
    a.logp = logp;
    a.adv = adv;
    a.ret = ret;
    a.rows = rows;
    a.idx = idx;
    a.grad_out = grad;
    a.stats = stats;
    a.workspace = workspace;
    a.clip = cfg->clip;
    a.ent_coef = cfg->ent_coef;
    a.lr = cfg->lr;
    a.beta1 = cfg->beta1;
    a.beta2 = cfg->beta2;
    a.eps = cfg->eps;
    hipError_t e = launch_ppo_update(a, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "learner launch");
    return ok();
}

int tp_ppo_update(const tp_ppo *cfg, float *params, float *adam_m, float *adam_v, int64_t step0,
                  int32_t n_updates, const void *obs, int64_t ld_obs, const float *action,
                  const float *logp, const float *adv, const float *ret, int64_t rows,
                  const int64_t *idx, float *grad, double *stats, void *workspace,
                  size_t workspace_bytes, void *stream)
{
    return tp_ppo_update_agents(cfg, 1, 0, params, adam_m, adam_v, step0, n_updates, obs, ld_obs,
                                action, logp, adv, ret, rows, idx, grad, stats, workspace,
                                workspace_bytes, stream);
}

int tp_minibatch_rows(uint64_t seed, uint64_t counter, int32_t n_updates, int32_t B, int32_t L,
                      int32_t E, int32_t agent, int32_t envs_per_agent, int64_t *idx,
                      void *stream)
{
    if (!idx || !aligned(idx, 8)) return fail(TP_EINVAL, "idx is NULL or misaligned");
    if (n_updates < 1 || B < 1 || L < 1 || E < 1 || envs_per_agent < 1 || E % envs_per_agent)
        return fail(TP_EINVAL, "n_updates = %d, B = %d, L = %d, E = %d, envs_per_agent = %d",
                    n_updates, B, L, E, envs_per_agent);
    if (agent < 0 || agent >= E / envs_per_agent)
        return fail(TP_EINVAL, "agent = %d outside 0..%d", agent, E / envs_per_agent - 1);
    if ((int64_t)n_updates * B > ((int64_t)1 << 40))
        return fail(TP_EINVAL, "n_updates * B too large");
    hipError_t e = launch_minibatch_rows(seed, counter, n_updates, B, L, E, agent,
                                         envs_per_agent, idx, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "minibatch launch");
    return ok();
}

int tp_ensemble_fuse(float *params, int32_t N, int32_t K, int64_t P, void *stream)
{
    if (!params || !aligned(params, 4)) return fail(TP_EINVAL, "params is NULL or misaligned");
    if (N < 1 || K < 1 || P < 1)
        return fail(TP_EINVAL, "N = %d, K = %d, P = %lld must be >= 1", N, K, (long long)P);
    hipError_t e = launch_ensemble_fuse(params, N, K, P, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "fuse launch");
    return ok();
}

int tp_fitness(const float *reward, int32_t L, int32_t E, int32_t n_agents, double gamma,
               double *env_return, double *fitness, void *stream)
{
    if (!reward || !env_return || !fitness) return fail(TP_EINVAL, "a fitness array is NULL");
    if (!aligned(reward, 4) || !aligned(env_return, 8) || !aligned(fitness, 8))
        return fail(TP_EINVAL, "fitness arrays are misaligned");
    if (L < 1 || E < 1 || n_agents < 1 || E % n_agents)
        return fail(TP_EINVAL, "L = %d, E = %d, n_agents = %d (E must be a multiple)", L, E,
                    n_agents);
    if (!(gamma > 0.0 && gamma <= 1.0)) return fail(TP_EINVAL, "gamma = %g outside (0,1]", gamma);
    hipError_t e = launch_fitness(reward, L, E, n_agents, gamma, fitness, env_return,
                                  (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "fitness launch");
    return ok();
}

int tp_keep_best(const double *fitness, double *best, int32_t *stall, const float *params,
                 float *best_params, int32_t A, int64_t P, void *stream)
{
    if (!fitness || !best || !stall || !params || !best_params)
        return fail(TP_EINVAL, "a keep-best array is NULL");
    if (!aligned(fitness, 8) || !aligned(best, 8) || !aligned(stall, 4) || !aligned(params, 4) ||
        !aligned(best_params, 4))
        return fail(TP_EINVAL, "keep-best arrays are misaligned");
    if (A < 1 || P < 1) return fail(TP_EINVAL, "A = %d, P = %lld must be >= 1", A, (long long)P);
    hipError_t e = launch_keep_best(fitness, best, stall, params, best_params, A, P,
                                    (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "keep-best launch");
    return ok();
}

int tp_select(const double *fitness, float *params, int32_t N, int64_t P, int32_t keep,
              int32_t *rank, void *stream)
{
    if (!fitness || !params || !rank) return fail(TP_EINVAL, "a select array is NULL");
    if (!aligned(fitness, 8) || !aligned(params, 4) || !aligned(rank, 4))
        return fail(TP_EINVAL, "select arrays are misaligned");
    if (N < 1 || N > 1024 || P < 1)
        return fail(TP_EINVAL, "N = %d (1..1024), P = %lld", N, (long long)P);
    if (keep < 1 || keep > N) return fail(TP_EINVAL, "keep = %d outside 1..N = %d", keep, N);
    hipError_t e = launch_select(fitness, params, N, P, keep, rank, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "select launch");
    return ok();
}

int tp_gae(const float *reward, const float *value, const uint8_t *done, int32_t L, int32_t E,
           float gamma, float lambda, float *adv, float *ret, void *stream)
{
    if (!reward || !value || !done || !adv || !ret) return fail(TP_EINVAL, "a gae array is NULL");
    if (!aligned(reward, 4) || !aligned(value, 4) || !aligned(adv, 4) || !aligned(ret, 4))
        return fail(TP_EINVAL, "gae arrays are not 4-byte aligned");
    if (L < 1 || E < 1) return fail(TP_EINVAL, "L = %d, E = %d must be >= 1", L, E);
    if (!(gamma > 0.0f && gamma <= 1.0f)) return fail(TP_EINVAL, "gamma = %g outside (0,1]", gamma);
    if (!(lambda >= 0.0f && lambda <= 1.0f)) return fail(TP_EINVAL, "lambda = %g outside [0,1]", lambda);
    hipError_t e = launch_gae(reward, value, done, L, E, (double)gamma,
                              (double)gamma * (double)lambda, adv, ret, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "gae launch");
    return ok();
}

}  // extern "C"
