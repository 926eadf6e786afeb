"""Helpers shared by the GPU parity tests: device setup of a workload through
the C ABI, tolerance checks, and teacher-forced oracle replay."""

from __future__ import annotations

import os
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import torch

import oracle
import workloads as W
from paper_2111_05188_amd import problem, tp

# tolerances stated for the hot path: MLP outputs fp32 1e-4 / bf16 2e-2
# relative, cash and asset 1e-6 relative, GAE 1e-5 relative; shares exact.
TOL_MLP = {"f32": 1e-4, "bf16": 2e-2}
TOL_REWARD = 1e-6
TOL_GAE = 1e-5
TOL_LOGP = 1e-5


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def rel_check(name, x, y, tol, quiet=False):
    """|x - y| <= tol * max(|y|, RMS(y)) elementwise (NaN == NaN); returns
    the worst ratio |x - y| / max(|y|, RMS(y)) and prints it."""
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    assert x.shape == y.shape, (name, x.shape, y.shape)
    both_nan = np.isnan(x) & np.isnan(y)
    fin = np.isfinite(y)
    rms = np.sqrt(np.mean(np.square(y[fin]))) if fin.any() else 0.0
    scale = np.maximum(np.abs(y), max(rms, 1e-30))
    bound = tol * scale
    ok = (np.abs(x - y) <= bound) | both_nan
    cmp = ~both_nan
    worst = float(np.nanmax(np.abs(x - y)[cmp] / scale[cmp])) if cmp.any() else 0.0
    if not ok.all():
        idx = np.argwhere(~ok)[:5]
        raise AssertionError(f"{name}: {(~ok).sum()} of {ok.size} outside tol {tol}; "
                             f"worst rel {worst:.3g}; first {idx.tolist()} "
                             f"x={x[tuple(idx[0])]} y={y[tuple(idx[0])]}")
    if not quiet:
        say(f"    {name}: worst rel error {worst:.3g} (tol {tol:g}, {ok.size} values)")
    return worst


def bits16(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def build_problem(cfg, mk, t0, E=None, envs_per_agent=None, store_obs=True,
                  taps=True, obs_last=True, params=None):
    params = W.make_actor(cfg) if params is None else params
    pb = problem.Problem(cfg, mk, params, t0, store_obs=store_obs, taps=taps,
                         obs_last=obs_last, E=E, envs_per_agent=envs_per_agent)
    return pb, params


def _replay_workers():
    try:
        return max(1, min(16, len(os.sched_getaffinity(0))))
    except AttributeError:  # pragma: no cover
        return 4


def oracle_replay(cfg, mk, params, t0_sub, env_ids, seed, L, teacher,
                  envs_per_agent, step0=0, state=None, chunk=8):
    """Oracle rollout of the envs `env_ids`, driven by `teacher` actions
    ([L][len(env_ids)][n]).  Envs are independent, so the replay runs in
    chunks of `chunk` envs on a thread pool (the oracle is plain C called
    through ctypes, which releases the interpreter lock); the chunks'
    results are joined in env order."""
    env_ids = np.asarray(env_ids)
    m = oracle.market(mk.price, mk.ind, mk.row0)
    ecfg = oracle.env_cfg(cfg)
    act = oracle.actor(*params, cfg.dims, cfg.dtype == "bf16", envs_per_agent)
    if state is None:
        cash, sh, t = oracle.env_reset(ecfg, t0_sub, cfg.n)
    else:
        cash, sh, t = (np.array(s, copy=True) for s in state)
    teacher = np.ascontiguousarray(teacher, dtype=np.float32)

    def run(lo):
        hi = min(len(env_ids), lo + chunk)
        c, h, tt = cash[lo:hi].copy(), sh[lo:hi].copy(), t[lo:hi].copy()
        o = oracle.rollout(m, ecfg, act, c, h, tt, seed, step0, L, cfg.K_pad,
                           env_ids=env_ids[lo:hi], teacher=teacher[:, lo:hi])
        o["obs_last"] = np.stack([
            oracle.obs(m, ecfg, int(tt[i]), float(c[i]), h[i], cfg.K_pad,
                       cfg.dtype == "bf16") for i in range(hi - lo)])
        return o, (c, h, tt)

    starts = list(range(0, len(env_ids), chunk))
    if len(starts) > 1:
        with ThreadPoolExecutor(_replay_workers()) as ex:
            parts = list(ex.map(run, starts))
    else:
        parts = [run(0)]
    out = {k: np.concatenate([p[0][k] for p in parts], axis=0 if k == "obs_last" else 1)
           for k in parts[0][0]}
    out["final"] = tuple(np.concatenate([p[1][i] for p in parts]) for i in range(3))
    return out


def compare_rollout(cfg, pb, out, ids, L, check_obs=True):
    """GPU trajectory rows of envs `ids` against the oracle replay."""
    ids_t = torch.as_tensor(ids, device=pb.traj.action.device)
    g_act = pb.traj.action[:L].index_select(1, ids_t).cpu().numpy()
    g_logp = pb.traj.logp[:L].index_select(1, ids_t).cpu().numpy()
    g_rew = pb.traj.reward[:L].index_select(1, ids_t).cpu().numpy()
    g_done = pb.traj.done[:L].index_select(1, ids_t).cpu().numpy()
    if pb.traj.mu_tap is not None:
        # the actor's output itself, element by element, against the
        # oracle's on the same (bit-identical) observations
        g_mu = pb.traj.mu_tap[:L].index_select(1, ids_t).cpu().numpy()
        rel_check("mu", g_mu, out["mu"], TOL_MLP[cfg.dtype])
    rel_check("action", g_act, out["act"], TOL_MLP[cfg.dtype])
    rel_check("logp", g_logp, out["logp"], TOL_LOGP)
    rel_check("reward", g_rew, out["reward"], TOL_REWARD)
    assert np.array_equal(g_done, out["done"])
    if pb.traj.cash_tap is not None:
        g_cash = pb.traj.cash_tap[:L].index_select(1, ids_t).cpu().numpy()
        g_sh = pb.traj.shares_tap[:L].index_select(1, ids_t).cpu().numpy()
        assert np.array_equal(g_sh, out["shares"]), "share counts differ"
        assert np.array_equal(g_cash, out["cash"]), "balances differ"
    if pb.traj.asset_tap is not None:
        # b + p^T h is exact in fp64 (prices in [2^-2, 2^13)), so bit-exact
        g_as = pb.traj.asset_tap[:L].index_select(1, ids_t).cpu().numpy()
        assert np.array_equal(g_as, out["asset"], equal_nan=True), "total assets differ"
    if check_obs and pb.traj.obs is not None:
        K = cfg.K_pad
        g_obs = pb.traj.obs[:L].index_select(1, ids_t)[..., :K]
        if cfg.dtype == "bf16":
            assert np.array_equal(bits16(g_obs), out["obs"]), "observations differ"
        else:
            assert np.array_equal(g_obs.cpu().numpy(), out["obs"]), "observations differ"
