"""Device-side setup of one workload for the C ABI: market tensor resident
in HBM, env state, actor parameters (fp32 masters + packed copy), trajectory
store and GAE buffers.  Plumbing only -- every step of the hot path runs in
libtp.so.

``cfg`` is any object with the workload fields (n, n_ind, E, L, hidden,
dtype, n_agents, hmax, fee, cash0, reward_scale, cash/price/share_scale,
gamma, lam, S, K_pad, dims, envs_per_agent).
"""

from __future__ import annotations

import torch

from . import tp


def env_cfg(cfg, horizon: int | None = None) -> tp.EnvCfg:
    return tp.env_cfg(cfg.hmax, cfg.L if horizon is None else horizon,
                      cfg.fee, cfg.cash0, cfg.reward_scale, cfg.cash_scale,
                      cfg.price_scale, cfg.share_scale)


def actor_dtype(cfg) -> int:
    return tp.TP_BF16 if cfg.dtype == "bf16" else tp.TP_F32


def obs_torch_dtype(cfg):
    return torch.bfloat16 if cfg.dtype == "bf16" else torch.float32


class Problem:
    """Everything one rollout of ``cfg`` needs on the device."""

    def __init__(self, cfg, market, actor_params, t0, device="cuda",
                 store_obs=True, taps=False, obs_last=False, E=None,
                 envs_per_agent=None):
        self.cfg = cfg
        self.device = device
        self.E = cfg.E if E is None else E
        epa = cfg.envs_per_agent if envs_per_agent is None else envs_per_agent
        self.price = torch.from_numpy(market.price).to(device)
        self.ind = torch.from_numpy(market.ind).to(device)
        self.mkt = tp.MarketT(self.price, self.ind)
        self.ecfg = env_cfg(cfg)
        self.t0 = torch.as_tensor(t0, dtype=torch.int64).to(device)
        self.state = tp.StateT.empty(self.E, cfg.n, device)
        W, b, ls = actor_params
        self.actor = tp.ActorT([torch.from_numpy(w).to(device) for w in W],
                               [torch.from_numpy(x).to(device) for x in b],
                               torch.from_numpy(ls).to(device), cfg.dims,
                               actor_dtype(cfg), epa)
        self.actor.pack()
        self.traj = tp.TrajT.alloc(
            cfg.L, self.E, cfg.n, cfg.K_pad if store_obs else None,
            obs_torch_dtype(cfg), taps=taps, obs_last=obs_last, device=device)
        self.adv = torch.empty(cfg.L, self.E, dtype=torch.float32, device=device)
        self.ret = torch.empty_like(self.adv)
        self.values = None

    def set_values(self, values):
        self.values = torch.from_numpy(values).to(self.device)

    def set_critic(self, critic_params):
        """Critic S-H1-H2-1 of the actor's dtype (fp32 masters, packed)."""
        W, b = critic_params
        cfg = self.cfg
        self.critic = tp.CriticT([torch.from_numpy(w).to(self.device) for w in W],
                                 [torch.from_numpy(x).to(self.device) for x in b],
                                 cfg.dims[:3], actor_dtype(cfg), self.actor.s.envs_per_agent)
        self.critic.pack()
        if self.values is None:
            self.values = torch.empty(cfg.L + 1, self.E, dtype=torch.float32,
                                      device=self.device)

    def critic_values(self, stream=None):
        """values [L+1][E] = V(obs_0 .. obs_L) of the stored trajectory."""
        obs = self.traj.obs_all
        if obs is None or obs.shape[0] != self.cfg.L + 1:
            raise ValueError("critic values need the stored observations and obs_last")
        tp.critic_value(self.critic, obs, self.values, stream)

    def reset(self, stream=None):
        tp.env_reset(self.mkt, self.ecfg, self.state, self.t0, None, stream)

    def rollout(self, seed, step0=0, L=None, stream=None, traj=None):
        tp.rollout(self.mkt, self.ecfg, self.state, self.actor, seed, step0,
                   self.cfg.L if L is None else L,
                   self.traj if traj is None else traj, stream)

    def gae(self, stream=None):
        tp.gae(self.traj.reward, self.values, self.traj.done, self.cfg.gamma,
               self.cfg.lam, self.adv, self.ret, stream)

    def step(self, seed, stream=None):
        """One pass of the hot path: reset, L-step rollout, GAE."""
        self.reset(stream)
        self.rollout(seed, 0, None, stream)
        self.gae(stream)
