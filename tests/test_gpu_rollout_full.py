"""Full-size GPU parity: every workload at its real shape and in the launch
configuration the benchmark times, checked against the teacher-forced oracle
on sampled envs (the oracle replays them one by one), plus GAE over the
full rollout on sampled columns."""

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_common import (build_problem, compare_rollout, oracle_replay,
                        rel_check, say, TOL_GAE)

pytestmark = pytest.mark.gpu

SEED = 0x5EED0FF12C


@pytest.fixture(scope="module")
def minute_market():
    say("[full] generating the 100-stock minute market")
    return W.make_market(W.get_config("nasdaq100"))


def _full(cfg, mk, ids, store_obs=True, taps=True):
    t0 = W.make_t0(cfg)
    pb, params = build_problem(cfg, mk, t0, store_obs=store_obs, taps=taps,
                               obs_last=store_obs)
    pb.set_values(W.make_values(cfg))
    say(f"[full] {cfg.name} E={cfg.E} L={cfg.L}: reset + rollout + gae")
    pb.step(SEED)
    torch.cuda.synchronize()
    ids = np.asarray(ids)
    teacher = pb.traj.action.index_select(1, torch.as_tensor(ids, device="cuda")).cpu().numpy()
    out = oracle_replay(cfg, mk, params, t0[ids], ids, SEED, cfg.L, teacher,
                        cfg.envs_per_agent)
    compare_rollout(cfg, pb, out, ids, cfg.L)
    # GAE on the GPU rewards/done at sampled columns
    cols = torch.as_tensor(ids, device="cuda")
    r = pb.traj.reward.index_select(1, cols).cpu().numpy()
    d = pb.traj.done.index_select(1, cols).cpu().numpy()
    v = pb.values.index_select(1, cols).cpu().numpy()
    a_o, r_o = oracle.gae(r, v, d, cfg.gamma, cfg.lam)
    rel_check("adv", pb.adv.index_select(1, cols).cpu().numpy(), a_o, TOL_GAE)
    rel_check("ret", pb.ret.index_select(1, cols).cpu().numpy(), r_o, TOL_GAE)
    return pb


def _spread(blocks, per_block, block_envs, seed):
    """One env from each of `blocks` workgroup-sized blocks of `block_envs`
    envs (every `per_block`-th block), at a varying position in the block."""
    rng = np.random.default_rng(seed)
    return [b * block_envs + int(rng.integers(block_envs)) for b in range(0, blocks, per_block)]


def test_dow30_full():
    cfg = W.get_config("dow30")
    mk = W.make_market(cfg)
    # 4 envs per workgroup on the generic kernel: 32 envs spread over all 256
    _full(cfg, mk, [0, 1, 1023] + _spread(256, 9, 4, 1))


def test_nasdaq100_full(minute_market):
    cfg = W.get_config("nasdaq100")
    # one env from every one of the 256 workgroups (16 envs each)
    _full(cfg, minute_market, sorted(set([0, 15, 16, 4095] + _spread(256, 1, 16, 2))))


@pytest.mark.parametrize("H", [256, 768])
def test_nasdaq_other_widths_full(minute_market, H):
    # the role-split kernel at its other widths (market batches of three
    # steps at 256, two at 768): 32 envs spread over all 256 workgroups
    cfg = W.get_config("nasdaq100").with_(hidden=(H, H))
    _full(cfg, minute_market, sorted(set([0, 4095] + _spread(256, 8, 16, 5 + H))))


@pytest.mark.parametrize("I", [4, 10])
def test_other_markets_full_launch(I):
    # the bench's launch (4,096 envs x 390 steps, 256 workgroups) on the
    # markets with 4 and 10 indicators per stock (a 60-day market: the
    # start rows, not the market's length, decide what the kernel does):
    # 32 envs spread over all 256 workgroups
    cfg = W.get_config("nasdaq100").with_(n_ind=I, N=60 * 390)
    mk = W.make_market(cfg)
    _full(cfg, mk, sorted(set([0, 4095] + _spread(256, 8, 16, 7 + I))))


def test_ensemble_full(minute_market):
    cfg = W.get_config("ensemble")
    # 8 envs of each of the 16 agents, including each agent's first and
    # last env
    ids = []
    rng = np.random.default_rng(3)
    for a in range(16):
        base = a * 1024
        ids += [base, base + 1023] + [base + int(x) for x in rng.choice(np.arange(1, 1023), 6,
                                                                         replace=False)]
    _full(cfg, minute_market, sorted(ids))


def test_stress_full(minute_market):
    cfg = W.get_config("stress")
    # 64 envs spread over the 4,096 workgroups, observations stored and checked
    _full(cfg, minute_market, sorted(set([0, 65535] + _spread(4096, 64, 16, 4))),
          store_obs=True, taps=True)
