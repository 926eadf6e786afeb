"""Pins for the oracle's backtest metrics (Section 5.2, "Evaluation
metrics") and its total-asset tap: a hand case, drawdown by brute force over
all pairs, closed forms for constant, geometric and alternating series,
Sharpe ratio and volatility against numpy, and the asset tap tied to the
reward of eq. (2)."""

from fractions import Fraction

import numpy as np

import oracle
import workloads as W

P_DAILY = 252.0


def _one(series, P=P_DAILY, rf=0.0):
    s = np.asarray(series, np.float64)
    return oracle.backtest_metrics(s[:1], s[1:, None], P, rf)[0]


def test_hand_case():
    # 100 -> 120 -> 90 -> 130 -> 65: returns .2, -.25, 4/9, -.5
    m = _one([100, 120, 90, 130, 65])
    assert m[0] == -0.35
    r = np.array([0.2, -0.25, 4 / 9, -0.5])
    assert abs(m[1] - ((0.65 ** (P_DAILY / 4)) - 1)) < 1e-15
    assert abs(m[2] - np.std(r, ddof=1) * np.sqrt(P_DAILY)) < 1e-12
    # the peak 130 falls to 65
    assert m[4] == 0.5


def test_drawdown_equals_brute_force_over_pairs():
    rng = np.random.default_rng(3)
    for _ in range(20):
        T = int(rng.integers(1, 60))
        v = np.cumprod(1 + rng.normal(0, 0.05, T + 1)) * 1e6
        want = 0.0
        for u in range(T + 1):
            for t in range(u, T + 1):
                want = max(want, 1 - v[t] / v[u])
        assert abs(_one(v)[4] - want) < 1e-15


def test_constant_series_is_flat():
    m = _one([1e6] * 50)
    assert list(m) == [0.0, 0.0, 0.0, 0.0, 0.0]


def test_geometric_growth_closed_form():
    g, T, P = 0.001, 390, 98280.0
    v = 1e6 * (1 + g) ** np.arange(T + 1)
    m = _one(v, P)
    assert abs(m[0] - ((1 + g) ** T - 1)) < 1e-12
    assert abs(m[1] - ((1 + g) ** P - 1)) / ((1 + g) ** P) < 1e-9
    assert m[2] < 1e-10          # returns equal g up to rounding
    assert m[4] == 0.0           # never below its running peak


def test_alternating_returns_closed_form():
    a, b, T = 0.03, -0.01, 40
    v = [Fraction(10 ** 6)]
    for t in range(T):
        v.append(v[-1] * (Fraction(103, 100) if t % 2 == 0 else Fraction(99, 100)))
    m = _one([float(x) for x in v])
    mean, sd = (a + b) / 2, abs(a - b) / 2 * np.sqrt(T / (T - 1))
    assert abs(m[2] - sd * np.sqrt(P_DAILY)) < 1e-9
    assert abs(m[3] - mean / sd * np.sqrt(P_DAILY)) < 1e-7
    # the drawdown of one down step from a peak
    assert abs(m[4] - 0.01) < 1e-12


def test_sharpe_and_volatility_against_numpy():
    rng = np.random.default_rng(9)
    T, E, P, rf = 300, 7, 98280.0, 0.02
    v = np.cumprod(1 + rng.normal(2e-5, 1e-3, (T + 1, E)), axis=0) * 1e6
    m = oracle.backtest_metrics(v[0], v[1:], P, rf)
    r = v[1:] / v[:-1] - 1
    sd = np.std(r, axis=0, ddof=1)
    np.testing.assert_allclose(m[:, 2], sd * np.sqrt(P), rtol=1e-12)
    np.testing.assert_allclose(m[:, 3], (r.mean(0) - rf / P) / sd * np.sqrt(P), rtol=1e-9)
    np.testing.assert_allclose(m[:, 0], v[-1] / v[0] - 1, rtol=1e-12)


def test_single_period_has_no_deviation():
    m = _one([100.0, 110.0])
    assert m[2] == 0.0 and m[3] == 0.0
    assert abs(m[0] - 0.1) < 1e-15


def test_asset_tap_matches_state_and_reward():
    """V_{j+1} = b + p^T h after the step (exact rationals from the state
    taps), and the reward is 2^-12 (V_{j+1} - V_j) (eq. (2))."""
    cfg = W.get_config("tiny")
    mk = W.make_market(cfg)
    m = oracle.market(mk.price, mk.ind)
    ec = oracle.env_cfg(cfg)
    act = oracle.actor(*W.make_actor(cfg), cfg.dims, False, cfg.envs_per_agent)
    E, L = 6, 40
    cash, sh, t = oracle.env_reset(ec, np.arange(E, dtype=np.int64) * 3, cfg.n)
    t_start = t.copy()
    out = oracle.rollout(m, ec, act, cash, sh, t, 11, 0, L, cfg.K_pad,
                         want=("reward", "cash", "shares", "asset"))
    for j in range(L):
        for e in range(E):
            p = mk.price[t_start[e] + j + 1]
            v = Fraction(float(out["cash"][j, e]))
            for i in range(cfg.n):
                v += Fraction(float(p[i])) * int(out["shares"][j, e, i])
            assert out["asset"][j, e] == float(v)
    v_prev = np.concatenate([np.full((1, E), cfg.cash0), out["asset"][:-1]])
    want = (2.0 ** -12 * (out["asset"] - v_prev)).astype(np.float32)
    np.testing.assert_array_equal(out["reward"], want)
