"""ctypes wrapper around the C oracle (``oracle/oracle.c``).

TEST INFRASTRUCTURE ONLY: the oracle is the plain sequential CPU definition
the HIP path is checked against.  Only the test suite, the package smoke
check and the benchmark's CPU-baseline leg may import this module.  It shares
no code with the HIP library and never imports it.

All arrays are numpy, C-contiguous, host memory.
"""

from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
# ORACLE_LIB points the wrapper at another build of oracle.c (used to check
# that the pins fail when a mistake is planted in the oracle).
_LIB = os.environ.get("ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
# The same source built with OpenMP: the rollout's envs run on all cores
# (the CPU baseline's all-core leg); results are identical to the plain build.
_LIB_OMP = os.path.join(_HERE, "liboracle_omp.so")

CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
          "-shared", "-Wall", "-Wextra"]


def _compile(out, extra=()):
    tmp = out + ".tmp"
    subprocess.check_call(["gcc", *CFLAGS, *extra, "-o", tmp, _SRC, "-lm"])
    os.replace(tmp, out)


def build(force: bool = True) -> str:
    """Compile liboracle.so (and the OpenMP build liboracle_omp.so) with gcc
    (no fast-math, no fp contraction)."""
    if force or not os.path.exists(_LIB):
        _compile(_LIB, ["-Wno-unknown-pragmas"])
    if force or not os.path.exists(_LIB_OMP):
        _compile(_LIB_OMP, ["-fopenmp"])
    return _LIB


class Market(C.Structure):
    _fields_ = [("price", C.c_void_p), ("ind", C.c_void_p),
                ("row0", C.c_int64), ("rows", C.c_int64),
                ("n", C.c_int32), ("n_ind", C.c_int32)]


class EnvCfg(C.Structure):
    _fields_ = [("hmax", C.c_int32), ("horizon", C.c_int32),
                ("fee", C.c_double), ("cash0", C.c_double),
                ("reward_scale", C.c_double), ("cash_scale", C.c_float),
                ("price_scale", C.c_float), ("share_scale", C.c_float)]


class Actor(C.Structure):
    _fields_ = [("n_agents", C.c_int32), ("envs_per_agent", C.c_int32),
                ("dims", C.c_int32 * 4), ("bf16", C.c_int32),
                ("W", C.c_void_p * 3), ("b", C.c_void_p * 3),
                ("log_std", C.c_void_p)]


class Traj(C.Structure):
    _fields_ = [("obs_f32", C.c_void_p), ("obs_bf16", C.c_void_p),
                ("act", C.c_void_p), ("logp", C.c_void_p),
                ("reward", C.c_void_p), ("done", C.c_void_p),
                ("cash_tap", C.c_void_p), ("shares_tap", C.c_void_p),
                ("mu", C.c_void_p), ("asset_tap", C.c_void_p)]


_lib = None
_lib_omp = None


def lib(omp: bool = False):
    """The oracle library; omp=True gives the OpenMP build (the rollout's
    envs over OMP_NUM_THREADS threads, results identical)."""
    global _lib, _lib_omp
    if omp:
        if _lib_omp is None:
            if not os.path.exists(_LIB_OMP) or os.path.getmtime(_LIB_OMP) < os.path.getmtime(_SRC):
                build()
            _lib_omp = _declare(C.CDLL(_LIB_OMP))
        return _lib_omp
    if _lib is None:
        if not os.environ.get("ORACLE_LIB") and (
                not os.path.exists(_LIB)
                or os.path.getmtime(_LIB) < os.path.getmtime(_SRC)):
            build()
        _lib = _declare(C.CDLL(_LIB))
    return _lib


def _declare(L):
    """Argument and result types of the oracle's functions."""
    vp, i32, i64, u32, u64 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint32, C.c_uint64
    L.orc_bf16_bits.restype = C.c_uint16
    L.orc_bf16_bits.argtypes = [C.c_float]
    L.orc_bf16_value.restype = C.c_float
    L.orc_bf16_value.argtypes = [C.c_uint16]
    L.orc_philox4x32_10.argtypes = [vp, vp, vp]
    L.orc_uniform.restype = C.c_float
    L.orc_uniform.argtypes = [u32]
    L.orc_normals.argtypes = [u64, u32, u32, u32, i32, vp]
    L.orc_obs.argtypes = [vp, vp, i64, C.c_double, vp, i32, vp, vp]
    L.orc_env_reset.argtypes = [vp, i32, i32, vp, vp, vp, vp]
    L.orc_clip_action.restype = C.c_float
    L.orc_clip_action.argtypes = [C.c_float]
    L.orc_shares_from_action.restype = i32
    L.orc_shares_from_action.argtypes = [C.c_float, i32]
    L.orc_env_step_one.restype = C.c_float
    L.orc_env_step_one.argtypes = [vp, vp, vp, vp, vp, vp, vp]
    L.orc_env_step.argtypes = [vp, vp, i32, vp, vp, vp, vp, vp, i32, vp, vp]
    L.orc_mlp.argtypes = [vp, i32, i32, vp, i32, vp]
    L.orc_rollout.argtypes = [vp, vp, vp, i32, vp, vp, vp, vp, u64, u64,
                              i32, i32, vp, vp]
    L.orc_gae.argtypes = [vp, vp, vp, i32, i32, C.c_float, C.c_float, vp, vp]
    L.orc_backtest_metrics.argtypes = [vp, vp, i32, i32, C.c_double, C.c_double, vp]
    L.orc_ensemble_fuse.argtypes = [vp, i32, i32, C.c_int64]
    L.orc_fitness.argtypes = [vp, i32, i32, i32, C.c_double, vp]
    L.orc_keep_best.argtypes = [vp, vp, vp, vp, vp, i32, C.c_int64]
    L.orc_select.argtypes = [vp, vp, i32, C.c_int64, i32, vp]
    L.orc_minibatch_rows.argtypes = [u64, u64, i32, i32, i32, i32, i32, i32, vp]
    L.orc_version.restype = C.c_int
    L.orc_threads.restype = C.c_int
    return L


def _p(a):
    return None if a is None else a.ctypes.data


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


# --------------------------------------------------------------------------
# structure builders (keep the numpy arrays alive on the returned object)
# --------------------------------------------------------------------------

class _Keep:
    def __init__(self, struct, *arrays):
        self.s = struct
        self.keep = arrays


def market(price, ind, row0=0):
    price = _c(price, np.float32)
    ind = _c(ind, np.float32)
    s = Market(_p(price), _p(ind), row0, price.shape[0], price.shape[1],
               ind.shape[2])
    return _Keep(s, price, ind)


def env_cfg(cfg, horizon=None):
    return EnvCfg(cfg.hmax, cfg.L if horizon is None else horizon, cfg.fee,
                  cfg.cash0, cfg.reward_scale, cfg.cash_scale,
                  cfg.price_scale, cfg.share_scale)


def actor(W, b, log_std, dims, bf16, envs_per_agent):
    W = [_c(w, np.float32) for w in W]
    b = [_c(x, np.float32) for x in b]
    log_std = _c(log_std, np.float32)
    s = Actor()
    s.n_agents = W[0].shape[0]
    s.envs_per_agent = envs_per_agent
    for i in range(4):
        s.dims[i] = dims[i]
    s.bf16 = 1 if bf16 else 0
    for l in range(3):
        s.W[l] = _p(W[l])
        s.b[l] = _p(b[l])
    s.log_std = _p(log_std)
    return _Keep(s, *W, *b, log_std)


# --------------------------------------------------------------------------
# functions
# --------------------------------------------------------------------------

def bf16_bits(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.float32).ravel()
    L = lib()
    return np.array([L.orc_bf16_bits(float(v)) for v in x],
                    dtype=np.uint16)


def bf16_value(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint32) << 16).view(np.float32)


def philox(ctr, key):
    c = _c(ctr, np.uint32)
    k = _c(key, np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().orc_philox4x32_10(_p(c), _p(k), _p(out))
    return out


def uniform(w: int) -> float:
    return lib().orc_uniform(int(w) & 0xFFFFFFFF)


def normals(seed, step, env, agent, n):
    z = np.zeros(n, dtype=np.float32)
    lib().orc_normals(seed, step, env, agent, n, _p(z))
    return z


def clip_action(a: float) -> float:
    return lib().orc_clip_action(a)


def shares_from_action(a: float, hmax: int) -> int:
    return lib().orc_shares_from_action(a, hmax)


def obs(mkt, ecfg, t, cash, shares, K_pad, bf16):
    sh = _c(shares, np.int32)
    if bf16:
        o = np.zeros(K_pad, dtype=np.uint16)
        lib().orc_obs(C.byref(mkt.s), C.byref(ecfg), t, cash, _p(sh), K_pad,
                      None, _p(o))
    else:
        o = np.zeros(K_pad, dtype=np.float32)
        lib().orc_obs(C.byref(mkt.s), C.byref(ecfg), t, cash, _p(sh), K_pad,
                      _p(o), None)
    return o


def env_reset(ecfg, t0, n):
    t0 = _c(t0, np.int64)
    E = t0.shape[0]
    cash = np.zeros(E, dtype=np.float64)
    shares = np.zeros((E, n), dtype=np.int32)
    t = np.zeros(E, dtype=np.int64)
    lib().orc_env_reset(C.byref(ecfg), E, n, _p(t0), _p(cash), _p(shares), _p(t))
    return cash, shares, t


def env_step_one(mkt, ecfg, cash, shares, t, action):
    """One env; returns (reward, new_cash, new_shares, new_t, diag[5])."""
    c = np.array([cash], dtype=np.float64)
    sh = np.array(shares, dtype=np.int32, copy=True)
    tt = np.array([t], dtype=np.int64)
    a = _c(action, np.float32)
    diag = np.zeros(5, dtype=np.float64)
    r = lib().orc_env_step_one(C.byref(mkt.s), C.byref(ecfg), _p(c), _p(sh),
                               _p(tt), _p(a), _p(diag))
    return r, float(c[0]), sh, int(tt[0]), diag


def env_step(mkt, ecfg, cash, shares, t, action, K_pad=0, bf16=False):
    """Batched step; state arrays are updated in place.  Returns (reward, obs)."""
    E, n = shares.shape
    a = _c(action, np.float32)
    r = np.zeros(E, dtype=np.float32)
    obs_f = obs_b = None
    if K_pad:
        if bf16:
            obs_b = np.zeros((E, K_pad), dtype=np.uint16)
        else:
            obs_f = np.zeros((E, K_pad), dtype=np.float32)
    lib().orc_env_step(C.byref(mkt.s), C.byref(ecfg), E, _p(cash), _p(shares),
                       _p(t), _p(a), _p(r), K_pad, _p(obs_f), _p(obs_b))
    return r, (obs_b if bf16 else obs_f)


def mlp(act, agent, x):
    x = _c(x, np.float32)
    M, ld = x.shape
    n = act.s.dims[3]
    mu = np.zeros((M, n), dtype=np.float32)
    lib().orc_mlp(C.byref(act.s), agent, M, _p(x), ld, _p(mu))
    return mu


def rollout(mkt, ecfg, act, cash, shares, t, seed, step0, L, K_pad,
            env_ids=None, teacher=None, want=("obs", "act", "logp", "reward",
                                              "done", "cash", "shares", "mu",
                                              "asset"), omp=False):
    """Run O9 over the envs in (cash, shares, t) (updated in place).

    env_ids: global env index of each row (Philox counter and agent id);
    teacher: raw actions [L][E][n] that drive the env step (teacher forcing);
    omp: run on the OpenMP build (envs over threads, same results).
    Returns a dict of time-major arrays."""
    E, n = shares.shape
    ids = None if env_ids is None else _c(env_ids, np.int32)
    tch = None if teacher is None else _c(teacher, np.float32)
    bf16 = bool(act.s.bf16)
    out = {}
    tr = Traj()
    if "obs" in want:
        out["obs"] = np.zeros((L, E, K_pad), dtype=np.uint16 if bf16 else np.float32)
        if bf16:
            tr.obs_bf16 = _p(out["obs"])
        else:
            tr.obs_f32 = _p(out["obs"])
    for key, shape, dt, fld in (("act", (L, E, n), np.float32, "act"),
                                ("logp", (L, E), np.float32, "logp"),
                                ("reward", (L, E), np.float32, "reward"),
                                ("done", (L, E), np.uint8, "done"),
                                ("cash", (L, E), np.float64, "cash_tap"),
                                ("shares", (L, E, n), np.int32, "shares_tap"),
                                ("mu", (L, E, n), np.float32, "mu"),
                                ("asset", (L, E), np.float64, "asset_tap")):
        if key in want:
            out[key] = np.zeros(shape, dtype=dt)
            setattr(tr, fld, _p(out[key]))
    lib(omp).orc_rollout(C.byref(mkt.s), C.byref(ecfg), C.byref(act.s), E,
                      _p(ids), _p(cash), _p(shares), _p(t), seed, step0, L,
                      K_pad, _p(tch), C.byref(tr))
    return out


def threads(omp: bool = False) -> int:
    """Threads the rollout uses in the plain (1) or the OpenMP build."""
    return lib(omp).orc_threads()


def gae(r, v, d, gamma, lam):
    r = _c(r, np.float32)
    v = _c(v, np.float32)
    d = _c(d, np.uint8)
    L, E = r.shape
    assert v.shape == (L + 1, E) and d.shape == (L, E)
    adv = np.zeros((L, E), dtype=np.float32)
    ret = np.zeros((L, E), dtype=np.float32)
    lib().orc_gae(_p(r), _p(v), _p(d), L, E, gamma, lam, _p(adv), _p(ret))
    return adv, ret


def backtest_metrics(v0, v, periods_per_year, risk_free=0.0):
    """Per-env {cumulative, annual return, annual volatility, Sharpe, max
    drawdown} of the asset series V_0 = v0 [E], V_1..V_T = v [T][E]."""
    v0 = _c(v0, np.float64)
    v = _c(v, np.float64)
    T, E = v.shape
    assert v0.shape == (E,)
    out = np.zeros((E, 5), dtype=np.float64)
    lib().orc_backtest_metrics(_p(v0), _p(v), T, E, periods_per_year, risk_free, _p(out))
    return out


def ensemble_fuse(params):
    """params [N][K][P] fp32 -> every pod of agent g holds the mean of its K pods."""
    p = np.array(params, dtype=np.float32, order="C", copy=True)
    N, K, P = p.shape
    lib().orc_ensemble_fuse(_p(p), N, K, P)
    return p


def fitness(reward, n_agents, gamma):
    """Per-agent mean over envs of sum_j gamma^j r_j (reward [L][E])."""
    r = _c(reward, np.float32)
    L, E = r.shape
    f = np.zeros(n_agents, dtype=np.float64)
    lib().orc_fitness(_p(r), L, E, n_agents, gamma, _p(f))
    return f


def keep_best(fit, best, stall, params, best_params):
    """Evaluator bookkeeping; returns updated copies (best, stall, best_params)."""
    fit = _c(fit, np.float64)
    best = np.array(best, dtype=np.float64, copy=True)
    stall = np.array(stall, dtype=np.int32, copy=True)
    params = _c(params, np.float32)
    bp = np.array(best_params, dtype=np.float32, order="C", copy=True)
    A, P = params.shape
    lib().orc_keep_best(_p(fit), _p(best), _p(stall), _p(params), _p(bp), A, P)
    return best, stall, bp


def select(fit, params, keep):
    """Selector: returns (rank [N], new params [N][P])."""
    fit = _c(fit, np.float64)
    p = np.array(params, dtype=np.float32, order="C", copy=True)
    N, P = p.shape
    rank = np.zeros(N, dtype=np.int32)
    lib().orc_select(_p(fit), _p(p), N, P, keep, _p(rank))
    return rank, p


def minibatch_rows(seed, counter, n_updates, B, L, E, agent, envs_per_agent):
    """Learner minibatch row indices [n_updates][B] (int64) of one agent."""
    idx = np.zeros((n_updates, B), dtype=np.int64)
    lib().orc_minibatch_rows(seed, counter, n_updates, B, L, E, agent, envs_per_agent,
                             _p(idx))
    return idx
