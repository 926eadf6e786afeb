"""GPU parity of the backtest path (Section 5.2, "Evaluation metrics"): a
deterministic-policy rollout (log_std = -inf, so a = mu) over a held-out
segment of the synthetic market, its total-asset tap against the oracle's
teacher-forced replay, and tp_backtest_metrics against the oracle's metrics
of the same series, for the daily and the minute workload shapes."""

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_common import build_problem, oracle_replay, say
from paper_2111_05188_amd import tp

pytestmark = pytest.mark.gpu

SEED = 0x5EED0FF12C


def _deterministic(params):
    W_, b_, ls = params
    return W_, b_, np.full_like(ls, -np.inf)


def _backtest(cfg, E, L, rows, ppy, held_out_from):
    c = cfg.with_(N=rows - 1, E=E)
    mk = W.make_market(c)
    # held-out segment: episodes start in the last part of the market
    rng = np.random.default_rng(17)
    t0 = rng.integers(held_out_from, rows - 1 - L, E).astype(np.int64)
    params = _deterministic(W.make_actor(c))
    pb, _ = build_problem(c, mk, t0, params=params)
    pb.reset()
    v0 = pb.state.cash.clone()
    say(f"[backtest] {cfg.name} E={E} L={L}")
    pb.rollout(SEED, 0, L)
    torch.cuda.synchronize()
    # the tap against the oracle replay (teacher-forced by the GPU actions)
    ids = np.arange(E)
    teacher = pb.traj.action[:L].cpu().numpy()
    assert np.all(np.isfinite(teacher))
    out = oracle_replay(c, mk, params, t0, ids, SEED, L, teacher, E)
    g_asset = pb.traj.asset_tap[:L].cpu().numpy()
    assert np.array_equal(g_asset, out["asset"])
    # metrics on the GPU against the oracle's on the same series
    met = tp.backtest_metrics(v0, pb.traj.asset_tap[:L], ppy, 0.02)
    torch.cuda.synchronize()
    want = oracle.backtest_metrics(v0.cpu().numpy(), g_asset, ppy, 0.02)
    np.testing.assert_allclose(met.cpu().numpy(), want, rtol=1e-12, atol=1e-15)
    return met.cpu().numpy()


def test_backtest_daily():
    cfg = W.get_config("dow30")
    _backtest(cfg, 64, 252, 2521, 252.0, 2000)


def test_backtest_minute():
    cfg = W.get_config("nasdaq100")
    m = _backtest(cfg, 48, 390, 30 * 390 + 1, 252.0 * 390, 20 * 390)
    assert np.all(m[:, 4] >= 0) and np.all(m[:, 4] < 1)


def test_metrics_edge_cases():
    # constant series (zero deviation), one period, a single env
    dev = "cuda"
    v0 = torch.tensor([1e6, 5e5], dtype=torch.float64, device=dev)
    v = torch.tensor([[1e6, 6e5]], dtype=torch.float64, device=dev)
    met = tp.backtest_metrics(v0, v, 252.0).cpu().numpy()
    want = oracle.backtest_metrics(v0.cpu().numpy(), v.cpu().numpy(), 252.0)
    np.testing.assert_allclose(met, want, rtol=1e-14)
    assert met[0, 2] == 0.0 and met[0, 3] == 0.0
    with pytest.raises(tp.TPError):
        tp.backtest_metrics(v0, v, 0.0)
