"""Sanity of the seeded synthetic inputs (shapes and distributions of the
paper's workloads; the paper's own datasets are not available here)."""

import json
import os

import numpy as np
import pytest

import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")


def test_configs_use_paper_constants():
    g = json.load(open(GOLD))
    for cfg in W.CONFIGS.values():
        assert cfg.gamma == g["gamma"]["value"]
        assert cfg.cash0 == g["cash0"]["value"]
    nas = W.get_config("nasdaq100")
    assert nas.L == g["minutes_per_day"]["value"]
    assert nas.T1 == 10 * 252 * 390 + 1


def test_config_shapes():
    c = W.CONFIGS
    assert c["tiny"].S == 31 and c["tiny"].K_pad == 32
    assert c["dow30"].S == 301 and c["dow30"].K_pad == 320
    assert c["nasdaq100"].S == 1001 and c["nasdaq100"].K_pad == 1024
    assert c["nasdaq100"].flops_per_env_step() == 1651712
    assert c["stress"].flops_per_env_step() == 2 * (1001 * 1024 + 1024 * 1024 + 1024 * 100)
    assert c["ensemble"].n_agents == 16 and c["ensemble"].envs_per_agent == 1024


def test_market_statistics_and_range():
    cfg = W.get_config("dow30")
    m = W.make_market(cfg)
    assert m.price.shape == (2521, 30) and m.ind.shape == (2521, 30, 8)
    assert m.price.dtype == np.float32
    assert m.price.min() >= 0.25 and m.price.max() <= 8191
    lr = np.diff(np.log(m.price.astype(np.float64)), axis=0)
    ok = (m.price[1:] > 0.25) & (m.price[1:] < 8191) & (m.price[:-1] > 0.25)
    lr = lr[ok]
    assert abs(lr.mean() + 0.5 * cfg.sigma ** 2) < 3 * cfg.sigma / np.sqrt(lr.size)
    assert abs(lr.std() / cfg.sigma - 1) < 0.02
    assert abs(m.ind.mean()) < 0.01 and abs(m.ind.std() - 1) < 0.01
    assert (m.price[0] >= 20).all() and (m.price[0] <= 200).all()


def test_market_rows_are_regenerable():
    cfg = W.get_config("nasdaq100").with_(N=20000)
    full = W.make_market(cfg)
    part = W.make_market(cfg, rows=(9000, 13000))
    assert np.array_equal(part.price, full.price[9000:13000])
    assert np.array_equal(part.ind, full.ind[9000:13000])


def test_t0_and_values():
    cfg = W.get_config("nasdaq100")
    t0 = W.make_t0(cfg)
    assert t0.shape == (cfg.E,) and (t0 % 390 == 0).all()
    assert t0.min() >= 0 and (t0 + cfg.L).max() <= cfg.T1 - 1
    assert (W.make_t0(W.get_config("tiny")) == 0).all()
    v = W.make_values(cfg)
    assert v.shape == (cfg.L + 1, cfg.E) and v.dtype == np.float32


def test_actor_init():
    cfg = W.get_config("ensemble")
    Wt, b, ls = W.make_actor(cfg)
    assert Wt[0].shape == (16, 512, 1001) and b[2].shape == (16, 100)
    assert np.abs(Wt[0]).max() <= 1 / np.sqrt(1001)
    assert not np.array_equal(Wt[0][0], Wt[0][1])
    assert (ls == -0.5).all()


def test_actions_have_special_values():
    a = W.make_actions(1, 64, 100)
    assert np.isnan(a).any() and np.isposinf(a).any() and np.isneginf(a).any()
    assert (a == 1).any() and (a == -1).any() and (a == 0).any()
