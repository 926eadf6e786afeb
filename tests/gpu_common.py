"""Helpers shared by the GPU parity tests: device setup of a workload through
the C ABI, tolerance checks, and teacher-forced oracle replay."""

from __future__ import annotations

import sys

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


def rel_check(name, x, y, tol):
    """|x - y| <= tol * max(|y|, RMS(y)) elementwise (NaN == NaN)."""
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    assert x.shape == y.shape, (name, x.shape, y.shape)
    both_nan = np.isnan(x) & np.isnan(y)
    fin = np.isfinite(y)
    rms = np.sqrt(np.mean(np.square(y[fin]))) if fin.any() else 0.0
    bound = tol * np.maximum(np.abs(y), max(rms, 1e-30))
    ok = (np.abs(x - y) <= bound) | both_nan
    if not ok.all():
        idx = np.argwhere(~ok)[:5]
        worst = np.nanmax(np.abs(x - y)[~both_nan] / np.maximum(np.abs(y), rms)[~both_nan])
        raise AssertionError(f"{name}: {(~ok).sum()} of {ok.size} outside tol {tol}; "
                             f"worst rel {worst:.3g}; first {idx.tolist()} "
                             f"x={x[tuple(idx[0])]} y={y[tuple(idx[0])]}")


def bits16(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def build_problem(cfg, mk, t0, E=None, envs_per_agent=None, store_obs=True,
                  taps=True, obs_last=True, params=None):
    params = W.make_actor(cfg) if params is None else params
    pb = problem.Problem(cfg, mk, params, t0, store_obs=store_obs, taps=taps,
                         obs_last=obs_last, E=E, envs_per_agent=envs_per_agent)
    return pb, params


def oracle_replay(cfg, mk, params, t0_sub, env_ids, seed, L, teacher,
                  envs_per_agent, step0=0, state=None):
    """Oracle rollout of the envs `env_ids`, driven by `teacher` actions."""
    m = oracle.market(mk.price, mk.ind, mk.row0)
    ecfg = oracle.env_cfg(cfg)
    act = oracle.actor(*params, cfg.dims, cfg.dtype == "bf16", envs_per_agent)
    if state is None:
        cash, sh, t = oracle.env_reset(ecfg, t0_sub, cfg.n)
    else:
        cash, sh, t = (np.array(s, copy=True) for s in state)
    out = oracle.rollout(m, ecfg, act, cash, sh, t, seed, step0, L, cfg.K_pad,
                         env_ids=env_ids, teacher=teacher)
    out["final"] = (cash, sh, t)
    out["obs_last"] = np.stack([
        oracle.obs(m, ecfg, int(t[i]), float(cash[i]), sh[i], cfg.K_pad,
                   cfg.dtype == "bf16") for i in range(len(env_ids))])
    return out


def compare_rollout(cfg, pb, out, ids, L, check_obs=True):
    """GPU trajectory rows of envs `ids` against the oracle replay."""
    ids_t = torch.as_tensor(ids, device=pb.traj.action.device)
    g_act = pb.traj.action[:L].index_select(1, ids_t).cpu().numpy()
    g_logp = pb.traj.logp[:L].index_select(1, ids_t).cpu().numpy()
    g_rew = pb.traj.reward[:L].index_select(1, ids_t).cpu().numpy()
    g_done = pb.traj.done[:L].index_select(1, ids_t).cpu().numpy()
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
