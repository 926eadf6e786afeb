"""GPU parity of tp_env_reset / tp_env_step against the oracle on the same
seeded inputs (generator-made states and actions, including NaN / +-Inf /
out-of-range actions, exhausted budgets and ragged batch sizes)."""

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_common import bits16, rel_check, say, TOL_REWARD
from paper_2111_05188_amd import problem, tp

pytestmark = pytest.mark.gpu


# the largest market the boundary takes: 128 stocks x 8 indicators
_EXTRA = {
    "largest_f32": W.get_config("tiny").with_(name="largest_f32", n=128, n_ind=8),
    "largest_bf16": W.get_config("tiny").with_(name="largest_bf16", n=128, n_ind=8, dtype="bf16"),
}


def _setup(name, E, rows, seed):
    cfg = _EXTRA[name] if name in _EXTRA else W.get_config(name)
    mk = W.make_market(cfg, rows=(0, rows))
    rng = np.random.default_rng(seed)
    cash = np.concatenate([rng.uniform(0, 2e6, E - E // 4), rng.uniform(0, 200, E // 4)])
    shares = rng.integers(0, 400, (E, cfg.n)).astype(np.int32)
    shares[rng.random((E, cfg.n)) < 0.3] = 0
    # room for the four chained steps of the test
    t = rng.integers(0, rows - 1 - 4, E).astype(np.int64)
    act = W.make_actions(seed + 1, E, cfg.n)
    return cfg, mk, cash, shares, t, act


@pytest.mark.parametrize("name,E,rows", [("tiny", 64, 257), ("tiny", 37, 257),
                                         ("largest_f32", 40, 257), ("largest_bf16", 33, 257),
                                         ("dow30", 1000, 2521),
                                         ("nasdaq100", 515, 5000)])
def test_env_step_teacher_forced(name, E, rows):
    say(f"[env_step] {name} E={E}")
    cfg, mk, cash, shares, t, act = _setup(name, E, rows, 17 + E)
    dev = "cuda"
    mkt = tp.MarketT(torch.from_numpy(mk.price).to(dev), torch.from_numpy(mk.ind).to(dev))
    ecfg = problem.env_cfg(cfg)
    st = tp.StateT(torch.from_numpy(cash).to(dev), torch.from_numpy(shares).to(dev),
                   torch.from_numpy(t).to(dev))
    obs_dt = problem.obs_torch_dtype(cfg)
    ld = (cfg.K_pad + 7) // 8 * 8 + 8
    m = oracle.market(mk.price, mk.ind)
    oc = oracle.env_cfg(cfg)
    c_cash, c_sh, c_t = cash.copy(), shares.copy(), t.copy()
    for k in range(4):                 # chained steps: state stays in lock step
        a = act if k == 0 else W.make_actions(100 + k, E, cfg.n)
        g_a = torch.from_numpy(a).to(dev)
        rew = torch.empty(E, dtype=torch.float32, device=dev)
        obs = torch.full((E, ld), 7.0, dtype=obs_dt, device=dev)
        tp.env_step(mkt, ecfg, st, g_a, rew, obs)
        torch.cuda.synchronize()
        r_o, obs_o = oracle.env_step(m, oc, c_cash, c_sh, c_t, a, cfg.K_pad,
                                     cfg.dtype == "bf16")
        assert np.array_equal(st.shares.cpu().numpy(), c_sh), "shares"
        assert np.array_equal(st.cash.cpu().numpy(), c_cash), "cash"
        assert np.array_equal(st.t.cpu().numpy(), c_t), "t"
        rel_check("reward", rew.cpu().numpy(), r_o, TOL_REWARD)
        g = obs[:, :cfg.K_pad]
        if cfg.dtype == "bf16":
            assert np.array_equal(bits16(g), obs_o)
        else:
            assert np.array_equal(g.cpu().numpy(), obs_o)
        # columns past K_pad are left untouched
        assert (obs[:, cfg.K_pad:].float() == 7.0).all()
        assert (c_cash >= 0).all() and (c_sh >= 0).all()


def test_env_step_out_of_range_env_is_noop():
    say("[env_step] invalid t")
    cfg = W.get_config("tiny")
    mk = W.make_market(cfg)
    dev = "cuda"
    mkt = tp.MarketT(torch.from_numpy(mk.price).to(dev), torch.from_numpy(mk.ind).to(dev))
    st = tp.StateT.empty(3, cfg.n, count_invalid=True)
    st.n_invalid.fill_(77)
    st.cash.fill_(5.0)
    st.t.copy_(torch.tensor([-1, cfg.T1 - 1, 10]))
    a = torch.full((3, cfg.n), 0.5, device=dev)
    rew = torch.empty(3, device=dev)
    tp.env_step(mkt, problem.env_cfg(cfg), st, a, rew)
    torch.cuda.synchronize()
    r = rew.cpu().numpy()
    assert np.isnan(r[0]) and np.isnan(r[1]) and np.isfinite(r[2])
    assert st.t.cpu().tolist() == [-1, cfg.T1 - 1, 11]
    assert st.cash.cpu().numpy()[0] == 5.0
    assert st.n_invalid.item() == 2        # the two envs that were not stepped


@pytest.mark.parametrize("name", ["tiny", "nasdaq100"])
def test_env_reset(name):
    say(f"[env_reset] {name}")
    cfg = W.get_config(name)
    rows = 3000 if name == "nasdaq100" else cfg.T1
    mk = W.make_market(cfg, rows=(0, rows))
    E = 70
    t0 = np.random.default_rng(3).integers(0, rows - 1, E).astype(np.int64)
    t0[5] = -3
    t0[6] = rows - 1        # no next row: invalid
    dev = "cuda"
    mkt = tp.MarketT(torch.from_numpy(mk.price).to(dev), torch.from_numpy(mk.ind).to(dev))
    st = tp.StateT.empty(E, cfg.n, count_invalid=True)
    st.shares.fill_(9)
    obs = torch.empty(E, cfg.K_pad, dtype=problem.obs_torch_dtype(cfg), device=dev)
    tp.env_reset(mkt, problem.env_cfg(cfg), st, torch.from_numpy(t0).to(dev), obs)
    torch.cuda.synchronize()
    m = oracle.market(mk.price, mk.ind)
    oc = oracle.env_cfg(cfg)
    assert (st.cash.cpu().numpy() == cfg.cash0).all() and (st.shares.cpu().numpy() == 0).all()
    tt = st.t.cpu().numpy()
    assert tt[5] == -1 and tt[6] == -1
    assert st.n_invalid.item() == 2
    for e in range(E):
        if e in (5, 6):
            continue
        assert tt[e] == t0[e]
        o = oracle.obs(m, oc, int(t0[e]), cfg.cash0, np.zeros(cfg.n, np.int32),
                       cfg.K_pad, cfg.dtype == "bf16")
        g = bits16(obs[e]) if cfg.dtype == "bf16" else obs[e].cpu().numpy()
        assert np.array_equal(g, o)
    assert (obs[5].float() == 0).all()


def test_env_step_bf16_rows_with_envs_not_stepped():
    """bf16 observation rows of the 100-stock shape (the aligned-store path)
    when envs that are not stepped (t = -1 or the last market row) share
    waves and workgroups with envs that are: the stepped envs' rows equal
    the oracle's bit for bit, the others are all NaN, rewards NaN."""
    rows = 300
    cfg, mk, cash, shares, _, act = _setup("nasdaq100", 10, rows, 23)
    t = np.array([-1, rows - 1, 10, 11, -1, 12, rows - 1, 3, 4, 5], np.int64)
    live = (t >= 0) & (t < rows - 1)
    say("[env_step] nasdaq100 bf16 rows, envs not stepped mixed in")
    dev = "cuda"
    mkt = tp.MarketT(torch.from_numpy(mk.price).to(dev), torch.from_numpy(mk.ind).to(dev))
    st = tp.StateT(torch.from_numpy(cash).to(dev), torch.from_numpy(shares).to(dev),
                   torch.from_numpy(t).to(dev))
    rew = torch.empty(10, dtype=torch.float32, device=dev)
    obs = torch.full((10, cfg.K_pad), 7.0, dtype=torch.bfloat16, device=dev)
    tp.env_step(mkt, problem.env_cfg(cfg), st, torch.from_numpy(act).to(dev), rew, obs)
    torch.cuda.synchronize()
    m, oc = oracle.market(mk.price, mk.ind), oracle.env_cfg(cfg)
    c_cash, c_sh, c_t = cash[live].copy(), shares[live].copy(), t[live].copy()
    r_o, obs_o = oracle.env_step(m, oc, c_cash, c_sh, c_t, act[live], cfg.K_pad, True)
    assert np.array_equal(bits16(obs[torch.from_numpy(live).to(dev)]), obs_o)
    rel_check("reward", rew.cpu().numpy()[live], r_o, TOL_REWARD)
    assert np.isnan(rew.cpu().numpy()[~live]).all()
    assert torch.isnan(obs[torch.from_numpy(~live).to(dev)].float()).all()


@pytest.mark.parametrize("obs_dtype", [torch.bfloat16, torch.float32])
def test_env_step_market_without_indicators(obs_dtype):
    """A market with no indicators (n_ind = 0: the state is balance, prices
    and holdings only) and 8 stocks: reset and chained steps against the
    oracle, observation rows bit for bit.  With bf16 rows and a stock count
    divisible by 4 this once took the aligned row writer, which reads
    indicator chunks and has none to read."""
    say(f"[env_step] n_ind = 0, {obs_dtype}")
    cfg = W.get_config("tiny").with_(n=8, n_ind=0)
    rows = 200
    mk = W.make_market(cfg, rows=(0, rows))
    assert mk.ind.shape == (rows, 8, 0)
    E = 21
    dev = "cuda"
    mkt = tp.MarketT(torch.from_numpy(mk.price).to(dev),
                     torch.empty(rows, 8, 0, dtype=torch.float32, device=dev))
    ecfg = problem.env_cfg(cfg)
    K = cfg.K_pad
    bf = obs_dtype == torch.bfloat16
    t0 = np.random.default_rng(5).integers(0, rows - 10, E).astype(np.int64)
    st = tp.StateT.empty(E, cfg.n, count_invalid=True)
    obs = torch.full((E, K), 7.0, dtype=obs_dtype, device=dev)
    tp.env_reset(mkt, ecfg, st, torch.from_numpy(t0).to(dev), obs)
    m, oc = oracle.market(mk.price, mk.ind), oracle.env_cfg(cfg)
    c_cash, c_sh, c_t = oracle.env_reset(oc, t0, cfg.n)
    torch.cuda.synchronize()
    for e in range(E):
        o = oracle.obs(m, oc, int(t0[e]), cfg.cash0, np.zeros(cfg.n, np.int32), K, bf)
        g = bits16(obs[e]) if bf else obs[e].cpu().numpy()
        assert np.array_equal(g, o)
    assert st.n_invalid.item() == 0
    for k in range(5):
        a = W.make_actions(40 + k, E, cfg.n)
        rew = torch.empty(E, dtype=torch.float32, device=dev)
        obs = torch.full((E, K), 7.0, dtype=obs_dtype, device=dev)
        tp.env_step(mkt, ecfg, st, torch.from_numpy(a).to(dev), rew, obs)
        torch.cuda.synchronize()
        r_o, obs_o = oracle.env_step(m, oc, c_cash, c_sh, c_t, a, K, bf)
        assert np.array_equal(st.shares.cpu().numpy(), c_sh), "shares"
        assert np.array_equal(st.cash.cpu().numpy(), c_cash), "cash"
        rel_check("reward", rew.cpu().numpy(), r_o, TOL_REWARD)
        g = bits16(obs) if bf else obs.cpu().numpy()
        assert np.array_equal(g, obs_o)
        assert st.n_invalid.item() == 0
