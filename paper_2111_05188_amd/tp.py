"""Python binding of libtp.so (include/tp.h): argument marshalling only.

Every function takes torch CUDA (HIP) tensors, passes their device pointers
and the current stream to the C ABI, and raises ``TPError`` on a negative
status.  No computation happens here; the library must be built
(``paper_2111_05188_amd.build``) -- a missing library is an error, never a
fallback.
"""

from __future__ import annotations

import ctypes as C
import os

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
# TP_LIB_PATH selects another build of the same library (the CPU sanitizer
# test loads a host-instrumented build); default: the in-tree libtp.so.
LIB_PATH = os.environ.get("TP_LIB_PATH") or os.path.join(HERE, "libtp.so")

TP_OK, TP_EINVAL, TP_ERANGE, TP_EUNSUPPORTED, TP_EHIP = 0, -1, -2, -3, -4
TP_F32, TP_BF16 = 0, 1
_NAMES = {TP_EINVAL: "TP_EINVAL", TP_ERANGE: "TP_ERANGE",
          TP_EUNSUPPORTED: "TP_EUNSUPPORTED", TP_EHIP: "TP_EHIP"}


class TPError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{_NAMES.get(code, code)}: {msg}")
        self.code = code


class Market(C.Structure):
    _fields_ = [("price", C.c_void_p), ("ind", C.c_void_p), ("T1", C.c_int64),
                ("n", C.c_int32), ("n_ind", C.c_int32)]


class EnvCfg(C.Structure):
    _fields_ = [("hmax", C.c_int32), ("horizon", C.c_int32),
                ("fee", C.c_double), ("cash0", C.c_double),
                ("reward_scale", C.c_double), ("cash_scale", C.c_float),
                ("price_scale", C.c_float), ("share_scale", C.c_float)]


class EnvState(C.Structure):
    _fields_ = [("cash", C.c_void_p), ("shares", C.c_void_p),
                ("t", C.c_void_p), ("E", C.c_int32), ("n_invalid", C.c_void_p)]


class Actor(C.Structure):
    _fields_ = [("n_agents", C.c_int32), ("envs_per_agent", C.c_int32),
                ("dims", C.c_int32 * 4), ("dtype", C.c_int32),
                ("W", C.c_void_p * 3), ("b", C.c_void_p * 3),
                ("log_std", C.c_void_p), ("agent_stride", C.c_int64)]


class Critic(C.Structure):
    _fields_ = [("n_agents", C.c_int32), ("envs_per_agent", C.c_int32),
                ("dims", C.c_int32 * 3), ("dtype", C.c_int32),
                ("W", C.c_void_p * 3), ("b", C.c_void_p * 3),
                ("agent_stride", C.c_int64)]


class Ppo(C.Structure):
    _fields_ = [("dims", C.c_int32 * 6), ("dtype", C.c_int32), ("batch", C.c_int32),
                ("clip", C.c_float), ("ent_coef", C.c_float), ("lr", C.c_float),
                ("beta1", C.c_float), ("beta2", C.c_float), ("eps", C.c_float)]


class Traj(C.Structure):
    _fields_ = [("obs", C.c_void_p), ("ld_obs", C.c_int64),
                ("action", C.c_void_p), ("logp", C.c_void_p),
                ("reward", C.c_void_p), ("done", C.c_void_p),
                ("cash_tap", C.c_void_p), ("shares_tap", C.c_void_p),
                ("obs_last", C.c_void_p), ("asset_tap", C.c_void_p),
                ("mu_tap", C.c_void_p)]


EXPORTS = ("tp_env_reset", "tp_env_step", "tp_actor_packed_bytes",
           "tp_actor_pack", "tp_rollout", "tp_gae", "tp_critic_packed_bytes",
           "tp_critic_pack", "tp_critic_value", "tp_backtest_metrics",
           "tp_backtest_metrics_work_bytes", "tp_ensemble_fuse", "tp_fitness",
           "tp_keep_best", "tp_select",
           "tp_ppo_param_count", "tp_ppo_workspace_bytes", "tp_ppo_update",
           "tp_ppo_update_agents", "tp_minibatch_rows", "tp_rollout_path",
           "tp_actor_release", "tp_critic_release", "tp_check_starts",
           "tp_backtest_metrics_noalloc",
           "tp_last_error", "tp_version")

_lib = None


def load(path: str = LIB_PATH):
    """Load libtp.so and declare its signatures (no GPU work)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built: run paper_2111_05188_amd/build.py")
    L = C.CDLL(path)
    vp, i32, i64, u64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64, C.c_size_t
    L.tp_env_reset.argtypes = [vp, vp, vp, vp, vp, i64, i32, vp]
    L.tp_env_step.argtypes = [vp, vp, vp, vp, vp, vp, i64, i32, vp]
    L.tp_actor_packed_bytes.argtypes = [vp]
    L.tp_actor_packed_bytes.restype = sz
    L.tp_actor_pack.argtypes = [vp, vp, sz, vp]
    L.tp_rollout.argtypes = [vp, vp, vp, vp, vp, sz, u64, u64, i32, vp, vp]
    L.tp_gae.argtypes = [vp, vp, vp, i32, i32, C.c_float, C.c_float, vp, vp, vp]
    L.tp_critic_packed_bytes.argtypes = [vp]
    L.tp_critic_packed_bytes.restype = sz
    L.tp_critic_pack.argtypes = [vp, vp, sz, vp]
    L.tp_critic_value.argtypes = [vp, vp, sz, vp, i64, i64, i32, vp, vp]
    L.tp_backtest_metrics.argtypes = [vp, vp, i32, i32, C.c_double, C.c_double, vp, vp,
                                      C.c_size_t, vp]
    L.tp_backtest_metrics_noalloc.argtypes = [vp, vp, i32, i32, C.c_double, C.c_double, vp,
                                              vp]
    L.tp_backtest_metrics_work_bytes.restype = C.c_size_t
    L.tp_backtest_metrics_work_bytes.argtypes = [i32, i32]
    L.tp_ensemble_fuse.argtypes = [vp, i32, i32, i64, vp]
    L.tp_fitness.argtypes = [vp, i32, i32, i32, C.c_double, vp, vp, vp]
    L.tp_keep_best.argtypes = [vp, vp, vp, vp, vp, i32, i64, vp]
    L.tp_select.argtypes = [vp, vp, i32, i64, i32, vp, vp]
    L.tp_ppo_param_count.restype = i64
    L.tp_ppo_param_count.argtypes = [vp]
    L.tp_ppo_workspace_bytes.restype = C.c_size_t
    L.tp_ppo_workspace_bytes.argtypes = [vp]
    L.tp_rollout_path.argtypes = [vp, vp]
    L.tp_minibatch_rows.argtypes = [C.c_uint64, C.c_uint64, i32, i32, i32, i32, i32, i32, vp,
                                    vp]
    L.tp_ppo_update.argtypes = [vp, vp, vp, vp, i64, i32, vp, i64, vp, vp, vp, vp, i64, vp,
                                vp, vp, vp, C.c_size_t, vp]
    L.tp_ppo_update_agents.argtypes = [vp, i32, i64, vp, vp, vp, i64, i32, vp, i64, vp, vp, vp,
                                       vp, i64, vp, vp, vp, vp, C.c_size_t, vp]
    L.tp_actor_release.argtypes = [vp]
    L.tp_critic_release.argtypes = [vp]
    L.tp_check_starts.argtypes = [vp, i32, i64, i32]
    L.tp_last_error.restype = C.c_char_p
    L.tp_version.restype = C.c_int
    for f in ("tp_env_reset", "tp_env_step", "tp_actor_pack", "tp_rollout", "tp_gae",
              "tp_critic_pack", "tp_critic_value", "tp_backtest_metrics",
              "tp_ensemble_fuse", "tp_fitness", "tp_keep_best", "tp_select",
              "tp_ppo_update", "tp_ppo_update_agents", "tp_minibatch_rows",
              "tp_actor_release", "tp_critic_release", "tp_check_starts",
              "tp_backtest_metrics_noalloc"):
        getattr(L, f).restype = C.c_int
    _lib = L
    return L


def _check(rc: int):
    if rc != TP_OK:
        raise TPError(rc, load().tp_last_error().decode())


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


# --------------------------------------------------------------------------
# structure helpers (hold references to the tensors they point at)
# --------------------------------------------------------------------------

class MarketT:
    def __init__(self, price: torch.Tensor, ind: torch.Tensor):
        assert price.dim() == 2 and ind.dim() == 3
        self.price, self.ind = price, ind
        self.s = Market(_ptr(price), _ptr(ind), price.shape[0], price.shape[1],
                        ind.shape[2])

    @property
    def n(self):
        return self.s.n

    @property
    def K_pad(self):
        S = 1 + 2 * self.s.n + self.s.n * self.s.n_ind
        return (S + 31) // 32 * 32


def env_cfg(hmax, horizon, fee, cash0, reward_scale, cash_scale, price_scale,
            share_scale) -> EnvCfg:
    return EnvCfg(hmax, horizon, fee, cash0, reward_scale, cash_scale,
                  price_scale, share_scale)


class StateT:
    """Env state arrays; ``n_invalid`` (optional int32 [1]) receives the
    number of envs each call could not start or step."""

    def __init__(self, cash: torch.Tensor, shares: torch.Tensor, t: torch.Tensor,
                 n_invalid: torch.Tensor | None = None):
        self.cash, self.shares, self.t, self.n_invalid = cash, shares, t, n_invalid
        self.s = EnvState(_ptr(cash), _ptr(shares), _ptr(t), cash.shape[0], _ptr(n_invalid))

    @staticmethod
    def empty(E: int, n: int, device="cuda", count_invalid: bool = False):
        return StateT(torch.zeros(E, dtype=torch.float64, device=device),
                      torch.zeros(E, n, dtype=torch.int32, device=device),
                      torch.zeros(E, dtype=torch.int64, device=device),
                      torch.zeros(1, dtype=torch.int32, device=device) if count_invalid else None)


class ActorT:
    """fp32 master parameters stacked per agent (see tp_actor), or views of
    flat per-agent vectors (agent_stride = P, n_agents given)."""

    def __init__(self, W, b, log_std, dims, dtype: int, envs_per_agent: int,
                 agent_stride: int = 0, n_agents: int | None = None):
        self.W, self.b, self.log_std = list(W), list(b), log_std
        s = Actor()
        s.n_agents = W[0].shape[0] if n_agents is None else n_agents
        s.agent_stride = agent_stride
        s.envs_per_agent = envs_per_agent
        for i in range(4):
            s.dims[i] = dims[i]
        s.dtype = dtype
        for l in range(3):
            s.W[l] = _ptr(self.W[l])
            s.b[l] = _ptr(self.b[l])
        s.log_std = _ptr(log_std)
        self.s = s
        self.packed = None

    def packed_bytes(self) -> int:
        nb = load().tp_actor_packed_bytes(C.byref(self.s))
        if nb == 0:
            _check(TP_EINVAL)
        return nb

    def pack(self, stream=None):
        """(Re)build the packed copy the rollout kernel reads."""
        nb = self.packed_bytes()
        if self.packed is None or self.packed.numel() < nb:
            self.release()
            self.packed = torch.empty(nb, dtype=torch.uint8, device=self.W[0].device)
        _check(load().tp_actor_pack(C.byref(self.s), _ptr(self.packed), nb,
                                    _stream(stream)))
        return self.packed

    def release(self):
        """Forget the packed copy (the library stops accepting its address)."""
        if self.packed is not None:
            load().tp_actor_release(_ptr(self.packed))
            self.packed = None

    def __del__(self):
        try:
            self.release()
        except Exception:  # interpreter shutdown
            pass


class CriticT:
    """fp32 master parameters of the critic stacked per agent (see tp_critic),
    or views of flat per-agent vectors (agent_stride = P, n_agents given)."""

    def __init__(self, W, b, dims, dtype: int, envs_per_agent: int,
                 agent_stride: int = 0, n_agents: int | None = None):
        self.W, self.b = list(W), list(b)
        s = Critic()
        s.n_agents = W[0].shape[0] if n_agents is None else n_agents
        s.agent_stride = agent_stride
        s.envs_per_agent = envs_per_agent
        for i in range(3):
            s.dims[i] = dims[i]
        s.dtype = dtype
        for l in range(3):
            s.W[l] = _ptr(self.W[l])
            s.b[l] = _ptr(self.b[l])
        self.s = s
        self.packed = None

    def packed_bytes(self) -> int:
        nb = load().tp_critic_packed_bytes(C.byref(self.s))
        if nb == 0:
            _check(TP_EINVAL)
        return nb

    def pack(self, stream=None):
        nb = self.packed_bytes()
        if self.packed is None or self.packed.numel() < nb:
            self.release()
            self.packed = torch.empty(nb, dtype=torch.uint8, device=self.W[0].device)
        _check(load().tp_critic_pack(C.byref(self.s), _ptr(self.packed), nb,
                                     _stream(stream)))
        return self.packed

    def release(self):
        if self.packed is not None:
            load().tp_critic_release(_ptr(self.packed))
            self.packed = None

    def __del__(self):
        try:
            self.release()
        except Exception:  # interpreter shutdown
            pass


class TrajT:
    def __init__(self, action, logp, reward, done, obs=None, ld_obs=0,
                 cash_tap=None, shares_tap=None, obs_last=None, asset_tap=None,
                 mu_tap=None):
        self.t = (action, logp, reward, done, obs, cash_tap, shares_tap, obs_last,
                  asset_tap, mu_tap)
        self.s = Traj(_ptr(obs), ld_obs, _ptr(action), _ptr(logp), _ptr(reward),
                      _ptr(done), _ptr(cash_tap), _ptr(shares_tap), _ptr(obs_last),
                      _ptr(asset_tap), _ptr(mu_tap))

    @staticmethod
    def alloc(L, E, n, K_pad=None, obs_dtype=None, taps=False, obs_last=False,
              device="cuda"):
        """Trajectory buffers; ``taps`` adds the parity taps (balance,
        holdings, total asset and the actor's output mu)."""
        kw = {}
        obs_all = None
        if K_pad is not None:
            ld = (K_pad + 7) // 8 * 8
            # the bootstrap row follows the L rows, so that [L+1][E] is one
            # block (the critic reads it in one call)
            obs_all = torch.empty(L + (1 if obs_last else 0), E, ld, dtype=obs_dtype,
                                  device=device)
            kw["obs"] = obs_all[:L]
            kw["ld_obs"] = ld
            if obs_last:
                kw["obs_last"] = obs_all[L]
        if taps:
            kw["cash_tap"] = torch.empty(L, E, dtype=torch.float64, device=device)
            kw["shares_tap"] = torch.empty(L, E, n, dtype=torch.int32, device=device)
            kw["asset_tap"] = torch.empty(L, E, dtype=torch.float64, device=device)
            kw["mu_tap"] = torch.empty(L, E, n, dtype=torch.float32, device=device)
        tr = TrajT(torch.empty(L, E, n, dtype=torch.float32, device=device),
                   torch.empty(L, E, dtype=torch.float32, device=device),
                   torch.empty(L, E, dtype=torch.float32, device=device),
                   torch.empty(L, E, dtype=torch.uint8, device=device), **kw)
        tr.obs_all = obs_all
        return tr

    action = property(lambda self: self.t[0])
    logp = property(lambda self: self.t[1])
    reward = property(lambda self: self.t[2])
    done = property(lambda self: self.t[3])
    obs = property(lambda self: self.t[4])
    cash_tap = property(lambda self: self.t[5])
    shares_tap = property(lambda self: self.t[6])
    obs_last = property(lambda self: self.t[7])
    asset_tap = property(lambda self: self.t[8])
    mu_tap = property(lambda self: self.t[9])


def _dtype_code(t: torch.Tensor | None, default=TP_F32) -> int:
    if t is None:
        return default
    return TP_BF16 if t.dtype == torch.bfloat16 else TP_F32


# --------------------------------------------------------------------------
# entry points (same names as the C ABI, without the tp_ prefix)
# --------------------------------------------------------------------------

def env_reset(mkt: MarketT, cfg: EnvCfg, st: StateT, t0: torch.Tensor,
              obs0: torch.Tensor | None = None, stream=None):
    ld = obs0.shape[-1] if obs0 is not None else 0
    _check(load().tp_env_reset(C.byref(mkt.s), C.byref(cfg), C.byref(st.s),
                               _ptr(t0), _ptr(obs0), ld, _dtype_code(obs0),
                               _stream(stream)))


def env_step(mkt: MarketT, cfg: EnvCfg, st: StateT, action: torch.Tensor,
             reward: torch.Tensor, obs_next: torch.Tensor | None = None,
             stream=None):
    ld = obs_next.shape[-1] if obs_next is not None else 0
    _check(load().tp_env_step(C.byref(mkt.s), C.byref(cfg), C.byref(st.s),
                              _ptr(action), _ptr(reward), _ptr(obs_next), ld,
                              _dtype_code(obs_next), _stream(stream)))


def rollout(mkt: MarketT, cfg: EnvCfg, st: StateT, actor: ActorT, seed: int,
            step0: int, L: int, traj: TrajT, stream=None):
    if actor.packed is None:
        raise TPError(TP_EINVAL, "actor is not packed: call actor.pack()")
    _check(load().tp_rollout(C.byref(mkt.s), C.byref(cfg), C.byref(st.s),
                             C.byref(actor.s), _ptr(actor.packed),
                             actor.packed.numel(), seed & (2 ** 64 - 1),
                             step0, L, C.byref(traj.s), _stream(stream)))


def gae(reward, value, done, gamma, lam, adv, ret, stream=None):
    L, E = reward.shape
    _check(load().tp_gae(_ptr(reward), _ptr(value), _ptr(done), L, E, gamma,
                         lam, _ptr(adv), _ptr(ret), _stream(stream)))


def check_starts(t0, T1: int, L: int):
    """Host-side check that every start row t0 (host int64 array) leaves L
    market rows; raises TPError(TP_ERANGE) naming the first bad env."""
    t0 = np.ascontiguousarray(t0, dtype=np.int64)
    _check(load().tp_check_starts(t0.ctypes.data, t0.shape[0], T1, L))


def last_error() -> str:
    return load().tp_last_error().decode()


def version() -> int:
    return load().tp_version()


def critic_value(critic: CriticT, obs: torch.Tensor, value: torch.Tensor, stream=None):
    """V of every row of obs [T][E][ld_obs] into value [T][E]."""
    if critic.packed is None:
        raise TPError(TP_EINVAL, "critic is not packed: call critic.pack()")
    T, E, ld = obs.shape
    assert value.shape == (T, E) and value.dtype == torch.float32
    _check(load().tp_critic_value(C.byref(critic.s), _ptr(critic.packed),
                                  critic.packed.numel(), _ptr(obs), ld, T, E,
                                  _ptr(value), _stream(stream)))


def backtest_metrics_workspace(T: int, E: int, device="cuda") -> torch.Tensor:
    nb = load().tp_backtest_metrics_work_bytes(T, E)
    if nb == 0:
        raise TPError(TP_EINVAL, load().tp_last_error().decode())
    return torch.empty(nb, dtype=torch.uint8, device=device)


def backtest_metrics(v0: torch.Tensor, v: torch.Tensor, periods_per_year: float,
                     risk_free: float = 0.0, out: torch.Tensor | None = None, work=None,
                     stream=None):
    """Per-env [cumulative, annual return, annual volatility, Sharpe, max
    drawdown] of V_0 = v0 [E], V_1..V_T = v [T][E] (fp64)."""
    T, E = v.shape
    if out is None:
        out = torch.empty(E, 5, dtype=torch.float64, device=v.device)
    if work is None:
        work = backtest_metrics_workspace(T, E, v.device)
    _check(load().tp_backtest_metrics(_ptr(v0), _ptr(v), T, E, periods_per_year,
                                      risk_free, _ptr(out), _ptr(work), work.numel(),
                                      _stream(stream)))
    return out


def backtest_metrics_noalloc(v0: torch.Tensor, v: torch.Tensor, periods_per_year: float,
                             risk_free: float = 0.0, out: torch.Tensor | None = None,
                             stream=None):
    """backtest_metrics without a workspace: the library's static device
    scratch holds the partials (calls on one GPU must not overlap)."""
    T, E = v.shape
    if out is None:
        out = torch.empty(E, 5, dtype=torch.float64, device=v.device)
    _check(load().tp_backtest_metrics_noalloc(_ptr(v0), _ptr(v), T, E, periods_per_year,
                                              risk_free, _ptr(out), _stream(stream)))
    return out


def ensemble_fuse(params: torch.Tensor, stream=None):
    """params [N][K][P] fp32: each pod takes its agent's mean, in place."""
    N, K, P = params.shape
    _check(load().tp_ensemble_fuse(_ptr(params), N, K, P, _stream(stream)))


def fitness(reward: torch.Tensor, n_agents: int, gamma: float, env_return=None,
            out=None, stream=None):
    """Per-agent fitness (fp64 [n_agents]) and per-env returns (fp64 [E])."""
    L, E = reward.shape
    if env_return is None:
        env_return = torch.empty(E, dtype=torch.float64, device=reward.device)
    if out is None:
        out = torch.empty(n_agents, dtype=torch.float64, device=reward.device)
    _check(load().tp_fitness(_ptr(reward), L, E, n_agents, gamma, _ptr(env_return),
                             _ptr(out), _stream(stream)))
    return out, env_return


def keep_best(fit, best, stall, params, best_params, stream=None):
    A, P = params.shape
    _check(load().tp_keep_best(_ptr(fit), _ptr(best), _ptr(stall), _ptr(params),
                               _ptr(best_params), A, P, _stream(stream)))


def select(fit, params, keep: int, rank=None, stream=None):
    N, P = params.shape
    if rank is None:
        rank = torch.empty(N, dtype=torch.int32, device=params.device)
    _check(load().tp_select(_ptr(fit), _ptr(params), N, P, keep, _ptr(rank),
                            _stream(stream)))
    return rank


def ppo_cfg(dims, dtype: int, batch: int, clip=0.25, ent_coef=0.02, lr=2.0 ** -14,
            beta1=0.9, beta2=0.999, eps=1e-8) -> Ppo:
    """Learner configuration; dims = (S, H1, H2, n, C1, C2)."""
    c = Ppo()
    for i in range(6):
        c.dims[i] = int(dims[i])
    c.dtype, c.batch = dtype, batch
    c.clip, c.ent_coef, c.lr = clip, ent_coef, lr
    c.beta1, c.beta2, c.eps = beta1, beta2, eps
    return c


def ppo_param_count(cfg: Ppo) -> int:
    p = load().tp_ppo_param_count(C.byref(cfg))
    if p == 0:
        raise TPError(TP_EINVAL, load().tp_last_error().decode())
    return p


def ppo_workspace(cfg: Ppo, device="cuda", n_agents: int = 1) -> torch.Tensor:
    nb = load().tp_ppo_workspace_bytes(C.byref(cfg))
    if nb == 0:
        raise TPError(TP_EINVAL, load().tp_last_error().decode())
    return torch.empty(nb * n_agents, dtype=torch.uint8, device=device)


def ppo_update(cfg: Ppo, params, adam_m, adam_v, step0: int, obs, action, logp, adv, ret,
               idx, workspace, grad=None, stats=None, stream=None):
    """n_updates = idx.shape[0] minibatch updates (idx [n_updates][B] int64);
    obs [rows][ld] (bf16 or fp32), action [rows][n], logp/adv/ret [rows]."""
    nu, B = idx.shape
    assert B == cfg.batch and idx.dtype == torch.int64
    rows, ld = obs.shape
    _check(load().tp_ppo_update(C.byref(cfg), _ptr(params), _ptr(adam_m), _ptr(adam_v),
                                step0, nu, _ptr(obs), ld, _ptr(action), _ptr(logp),
                                _ptr(adv), _ptr(ret), rows, _ptr(idx), _ptr(grad),
                                _ptr(stats), _ptr(workspace), workspace.numel(),
                                _stream(stream)))


def ppo_update_agents(cfg: Ppo, params, adam_m, adam_v, step0: int, obs, action, logp, adv,
                      ret, idx, workspace, grad=None, stats=None, stream=None):
    """ppo_update for A independent learners in one call: params, adam_m,
    adam_v [A][stride] (stride >= P), idx [A][n_updates][B] int64, grad
    [A][P] and stats [A][n_updates][4] optional, workspace from
    ppo_workspace(cfg, n_agents=A)."""
    A, nu, B = idx.shape
    assert B == cfg.batch and idx.dtype == torch.int64
    assert params.dim() == 2 and params.shape[0] == A
    assert adam_m.shape == params.shape and adam_v.shape == params.shape
    assert params.stride(1) == 1 and adam_m.stride() == params.stride()
    assert adam_v.stride() == params.stride() and idx.is_contiguous()
    P = ppo_param_count(cfg)
    assert params.shape[1] >= P
    assert grad is None or (grad.shape == (A, P) and grad.is_contiguous())
    assert stats is None or (stats.shape == (A, nu, 4) and stats.is_contiguous())
    rows, ld = obs.shape
    _check(load().tp_ppo_update_agents(C.byref(cfg), A, params.stride(0), _ptr(params),
                                       _ptr(adam_m), _ptr(adam_v), step0, nu, _ptr(obs), ld,
                                       _ptr(action), _ptr(logp), _ptr(adv), _ptr(ret), rows,
                                       _ptr(idx), _ptr(grad), _ptr(stats), _ptr(workspace),
                                       workspace.numel(), _stream(stream)))


def flat_segments(dims6):
    """(offset, shape) of each segment of one agent's flat vector, in the
    order tp_ppo_update documents (dims6 = S, H1, H2, n, C1, C2)."""
    S, H1, H2, n, C1, C2 = dims6
    shapes = [("W1", (H1, S)), ("b1", (H1,)), ("W2", (H2, H1)), ("b2", (H2,)),
              ("W3", (n, H2)), ("b3", (n,)), ("log_std", (n,)), ("Wc1", (C1, S)),
              ("bc1", (C1,)), ("Wc2", (C2, C1)), ("bc2", (C2,)), ("wc3", (C2,)),
              ("bc3", (1,))]
    out, off = {}, 0
    for name, shp in shapes:
        out[name] = (off, shp)
        off += int(np.prod(shp))
    return out, off


def flat_views(flat: torch.Tensor, dims6, dtype: int, envs_per_agent: int):
    """ActorT and CriticT reading agent a's networks from flat[a] ([A][P])."""
    seg, P = flat_segments(dims6)
    assert flat.dim() == 2 and flat.shape[1] == P and flat.is_contiguous()
    A = flat.shape[0]
    v = {k: flat[0, o:o + int(np.prod(shp))] for k, (o, shp) in seg.items()}
    S, H1, H2, n, C1, C2 = dims6
    actor = ActorT([v["W1"], v["W2"], v["W3"]], [v["b1"], v["b2"], v["b3"]], v["log_std"],
                   (S, H1, H2, n), dtype, envs_per_agent, agent_stride=P, n_agents=A)
    critic = CriticT([v["Wc1"], v["Wc2"], v["wc3"]], [v["bc1"], v["bc2"], v["bc3"]],
                     (S, C1, C2), dtype, envs_per_agent, agent_stride=P, n_agents=A)
    actor.flat = critic.flat = flat
    return actor, critic


def minibatch_rows(seed: int, counter: int, n_updates: int, B: int, L: int, E: int, agent: int,
                   envs_per_agent: int, out=None, device="cuda", stream=None):
    """Learner minibatch rows [n_updates][B] int64 of one agent."""
    if out is None:
        out = torch.empty(n_updates, B, dtype=torch.int64, device=device)
    _check(load().tp_minibatch_rows(seed, counter, n_updates, B, L, E, agent, envs_per_agent,
                                    _ptr(out), _stream(stream)))
    return out


def rollout_path(mkt: MarketT, actor: ActorT) -> int:
    """1 if tp_rollout runs the role-split kernel for this shape, else 0."""
    r = load().tp_rollout_path(C.byref(mkt.s), C.byref(actor.s))
    if r < 0:
        _check(r)
    return r
