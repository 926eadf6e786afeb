"""GPU parity of the backtest path (Section 5.2, "Evaluation metrics"): a
deterministic-policy rollout (log_std = -inf, so a = mu) over a held-out
segment of the synthetic market, its total-asset tap against the oracle's
teacher-forced replay, and tp_backtest_metrics against the oracle's metrics
of the same series, for the daily and the minute workload shapes, and on
synthetic series that exercise every launch geometry (a year of minute bars
for a few envs, empty time chunks, 64-env groups, a NaN series).

Tolerances: the cumulative return and the drawdown are computed from the
same operands as the oracle's serial walk (drawdown bit-exact); the annual
return differs by the device pow's rounding; the volatility and the Sharpe
ratio come from sums that the GPU adds in a different (tree) order, so their
tolerance is the reassociation bound |d sum| <= T u sum|x| (u = 2^-53)
carried through the mean, the sample deviation and the ratio."""

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
    # metrics on the GPU (of its own tap) against the oracle's metrics of the
    # oracle's own series (equal to the tap, as just checked)
    met = tp.backtest_metrics(v0, pb.traj.asset_tap[:L], ppy, 0.02)
    torch.cuda.synchronize()
    o_v0 = np.full(E, c.cash0)
    want = oracle.backtest_metrics(o_v0, out["asset"], ppy, 0.02)
    check_metrics(met.cpu().numpy(), want, o_v0, out["asset"], ppy, 0.02)
    return met.cpu().numpy()


U = 2.0 ** -53


def check_metrics(got, want, v0, v, P, rf):
    """got/want [E][5]; v0 [E], v [T][E] the series both were computed from."""
    T = v.shape[0]
    s = np.concatenate([v0[None], v])
    r = s[1:] / s[:-1] - 1.0
    mean = r.mean(0)
    d = r - mean
    ss = (d * d).sum(0)
    sd = np.sqrt(ss / max(T - 1, 1))
    d_mean = 4 * U * np.abs(r).sum(0)                       # 4x the first-order bound
    d_ss = 4 * T * U * ss + 2 * np.abs(d).sum(0) * d_mean
    with np.errstate(divide="ignore", invalid="ignore"):
        d_sd_rel = np.where(ss > 0, d_ss / (2 * ss), 0.0)
        d_sharpe = np.sqrt(P) * np.where(
            sd > 0, d_mean / sd + np.abs(mean - rf / P) / sd * d_sd_rel, 0.0)
    np.testing.assert_array_equal(got[:, 0], want[:, 0])
    np.testing.assert_array_equal(got[:, 4], want[:, 4])
    np.testing.assert_allclose(got[:, 1], want[:, 1], rtol=1e-13, atol=1e-16)
    ok = np.isfinite(want[:, 2])
    assert np.array_equal(ok, np.isfinite(got[:, 2]))
    # plus a few ulps of the final roundings, which can flip on tiny input changes
    ulps = 8 * U * np.abs(want[ok])
    assert np.all(np.abs(got[ok, 2] - want[ok, 2]) <= sd[ok] * np.sqrt(P) * d_sd_rel[ok] + ulps[:, 2])
    assert np.all(np.abs(got[ok, 3] - want[ok, 3]) <= d_sharpe[ok] + ulps[:, 3])


@pytest.mark.parametrize("T,E", [(98280, 3), (1000, 1), (390, 4096), (5, 70000), (7, 130)])
def test_metrics_launch_geometries(T, E):
    say(f"[metrics] T={T} E={E}")
    rng = np.random.default_rng(T + E)
    v0 = np.full(E, 1e6) * rng.uniform(0.5, 2.0, E)
    steps = 1.0 + rng.normal(2e-5, 1e-3, (T, E))
    v = v0[None] * np.cumprod(steps, axis=0)
    if E > 2:
        v[T // 2:, 1] = np.nan            # a series that stops (NaN from then on)
    dv0, dv = torch.from_numpy(v0).cuda(), torch.from_numpy(v).cuda()
    met = tp.backtest_metrics(dv0, dv, 252.0 * 390, 0.02)
    torch.cuda.synchronize()
    want = oracle.backtest_metrics(v0, v, 252.0 * 390, 0.02)
    check_metrics(met.cpu().numpy(), want, v0, v, 252.0 * 390, 0.02)


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
