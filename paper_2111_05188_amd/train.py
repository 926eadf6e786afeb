"""A population's training loop on one GPU, every step a libtp.so call:

  rollout of all envs (worker, Section 4.3)  ->  critic values of the stored
  observations  ->  GAE  ->  per pod, Philox minibatch rows and PPO updates
  (learner, Section 4.3; Table 2)  ->  ensemble fusion of each agent's pods,
  fitness of eq. (1) on the rollout's rewards, keep-best and selection
  (evolution layer, Section 4.2).

Parameters live in one flat fp32 buffer [N][K][P] (N agents x K pods, one
vector per pod in the learner's layout); the rollout and the critic read it
through agent_stride views, so nothing is copied between the stages.  Env e
belongs to pod e / envs_per_pod, pod q to agent q / K.

Readings where the paper is silent: after fusion every pod of an agent
holds the mean of the pods' parameters and of their Adam moments; the
selector replaces the parameters and moments of the agents it drops; an
epoch runs `updates` learner updates per pod (Table 2's repeat count times
the transitions per batch, by default).

Plumbing only (device buffers, streams, loop order); this module does no
arithmetic of the method.
"""

from __future__ import annotations

import torch

from . import tp
from .problem import actor_dtype, env_cfg, obs_torch_dtype


class Trainer:
    def __init__(self, cfg, market, t0, flat_params, n_agents: int, pods: int,
                 batch: int = 1024, updates: int | None = None, keep: int | None = None,
                 seed: int = 0x5EED, device="cuda"):
        self.cfg, self.device = cfg, device
        self.N, self.K = n_agents, pods
        A = n_agents * pods
        self.E = cfg.E
        assert self.E % A == 0, "envs must split evenly over pods"
        self.epa = self.E // A
        S, H1, H2, n = cfg.dims
        self.dims6 = (S, H1, H2, n, H1, H2)
        dt = actor_dtype(cfg)
        self.ppo = tp.ppo_cfg(self.dims6, dt, batch)
        self.P = tp.ppo_param_count(self.ppo)
        flat = torch.as_tensor(flat_params, dtype=torch.float32).to(device)
        assert flat.shape == (A, self.P), f"flat params must be [{A}][{self.P}]"
        self.flat = flat.contiguous()
        self.m = torch.zeros_like(self.flat)
        self.v = torch.zeros_like(self.flat)
        self.best_params = self.flat.clone()
        self.best = torch.full((A,), float("nan"), dtype=torch.float64, device=device)
        self.stall = torch.zeros(A, dtype=torch.int32, device=device)
        self.actor, self.critic = tp.flat_views(self.flat, self.dims6, dt, self.epa)
        # market, envs, trajectory (with the bootstrap observation row)
        self.price = torch.from_numpy(market.price).to(device)
        self.ind = torch.from_numpy(market.ind).to(device)
        self.mkt = tp.MarketT(self.price, self.ind)
        self.ecfg = env_cfg(cfg)
        self.t0 = torch.as_tensor(t0, dtype=torch.int64).to(device)
        self.state = tp.StateT.empty(self.E, n, device)
        self.traj = tp.TrajT.alloc(cfg.L, self.E, n, cfg.K_pad, obs_torch_dtype(cfg),
                                   taps=False, obs_last=True, device=device)
        self.values = torch.empty(cfg.L + 1, self.E, dtype=torch.float32, device=device)
        self.adv = torch.empty(cfg.L, self.E, dtype=torch.float32, device=device)
        self.ret = torch.empty_like(self.adv)
        rows = cfg.L * self.E
        self.updates = (updates if updates is not None
                        else max(1, 8 * (cfg.L * self.epa) // batch))
        self.keep = keep if keep is not None else max(1, n_agents // 2)
        self.idx = torch.empty(A, self.updates, batch, dtype=torch.int64, device=device)
        self.ws = tp.ppo_workspace(self.ppo, device, n_agents=A)
        self.stats = torch.empty(A, self.updates, 4, dtype=torch.float64, device=device)
        self.env_return = torch.empty(self.E, dtype=torch.float64, device=device)
        self.fitness = torch.empty(n_agents, dtype=torch.float64, device=device)
        self.rank = torch.empty(n_agents, dtype=torch.int32, device=device)
        self.seed, self.epoch_no, self.counter, self.step = seed, 0, 0, 1
        self.rows = rows

    def epoch(self, stream=None, evolve: bool = True):
        """One generation: explore, learn, fuse pods, evaluate and select."""
        cfg, A = self.cfg, self.N * self.K
        seed = self.seed + self.epoch_no
        tp.env_reset(self.mkt, self.ecfg, self.state, self.t0, None, stream)
        self.actor.pack(stream)
        tp.rollout(self.mkt, self.ecfg, self.state, self.actor, seed, 0, cfg.L, self.traj,
                   stream)
        self.critic.pack(stream)
        tp.critic_value(self.critic, self.traj.obs_all, self.values, stream)
        tp.gae(self.traj.reward, self.values, self.traj.done, cfg.gamma, cfg.lam, self.adv,
               self.ret, stream)
        K_pad, n = cfg.K_pad, cfg.n
        obs = self.traj.obs_all[:cfg.L].reshape(self.rows, K_pad)
        act = self.traj.action.reshape(self.rows, n)
        logp = self.traj.logp.reshape(self.rows)
        adv, ret = self.adv.reshape(self.rows), self.ret.reshape(self.rows)
        # every learner (agent x pod) draws its own rows, then all of them
        # update together, each launch covering every learner
        for q in range(A):
            tp.minibatch_rows(seed, self.counter, self.updates, self.ppo.batch, cfg.L, self.E,
                              q, self.epa, out=self.idx[q], stream=stream)
        tp.ppo_update_agents(self.ppo, self.flat, self.m, self.v, self.step, obs, act, logp, adv,
                             ret, self.idx, self.ws, stats=self.stats, stream=stream)
        self.counter += self.updates
        self.step += self.updates
        if evolve:
            self.evolve(stream)
        self.epoch_no += 1

    def evolve(self, stream=None):
        """Ensemble fusion of each agent's pods, then the evaluator and the
        selector over agents (scored on the rollout this epoch explored)."""
        N, K, P = self.N, self.K, self.P
        for buf in (self.flat, self.m, self.v):
            tp.ensemble_fuse(buf.view(N, K, P), stream)
        tp.fitness(self.traj.reward, N, self.cfg.gamma, env_return=self.env_return,
                   out=self.fitness, stream=stream)
        # keep-best per agent (its first pod stands for the fused agent)
        fit_pods = self.fitness.repeat_interleave(K)
        tp.keep_best(fit_pods, self.best, self.stall, self.flat, self.best_params, stream)
        if N > 1:
            for buf in (self.m, self.v):
                tp.select(self.fitness, buf.view(N, K * P), self.keep, rank=self.rank,
                          stream=stream)
            tp.select(self.fitness, self.flat.view(N, K * P), self.keep, rank=self.rank,
                      stream=stream)
