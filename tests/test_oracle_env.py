"""Pins for the oracle's env step (paper Section 3, eqs. (2)-(4)).

Nothing here compares the oracle with itself.  The expected values come from:
  * hand-worked tiny cases (E1, E2, E2b), re-derived below in exact rational
    arithmetic from eq. (3) (fee-free balance), eq. (4) and eq. (2) with the
    transaction cost c_t = fee * traded value;
  * a brute-force enumeration of every buy vector (the buy rule is the
    lexicographically largest affordable vector, a different statement of
    "largest affordable q in ascending stock order");
  * invariants: total asset = balance + p^T h; zero action leaves the
    portfolio unchanged and earns h^T (p_{t+1} - p_t); balance and holdings
    never go negative; eq. (2) with c_t equals the fee-charged balance
    update; exact-sum order independence.
"""

import itertools
import math
from fractions import Fraction as F

import numpy as np
import pytest

import oracle
import workloads as W


def mk_market(prices, n_ind=1, ind=None):
    p = np.asarray(prices, dtype=np.float32)
    rows, n = p.shape
    if ind is None:
        ind = np.zeros((rows, n, n_ind), dtype=np.float32)
    return oracle.market(p, ind)


def ecfg(hmax=64, fee=1e-3, scale=1.0, horizon=1):
    return oracle.EnvCfg(hmax, horizon, fee, 1e6, scale, 2.0 ** -20, 2.0 ** -7,
                         2.0 ** -7)


def exact_step(p0, p1, b, h, k, fee, scale):
    """Exact-rational env step straight from eqs. (2)-(4) and the readings.

    Sell set: min(-k, h) shares at p_t, credited with (1 - fee) (rounded
    once to fp64, as the balance is an fp64 number).  Buy vector: the
    lexicographically largest q in prod [0, k_i] whose cost with fee fits the
    post-sale balance (enumerated, not greedy).  Returns (h', b', r, c_t,
    fee-free eq.(3) balance)."""
    n = len(p0)
    P0 = [F(float(x)) for x in p0]
    P1 = [F(float(x)) for x in p1]
    fs, fb = F(1.0 - fee), F(1.0 + fee)
    hh = list(h)
    S = F(0)
    for i in range(n):
        if k[i] < 0:
            s = min(-k[i], hh[i])
            hh[i] -= s
            S += P0[i] * s
    b_s = F(float(F(b) + fs * S))           # one rounding (fma)
    buy = [max(k[i], 0) for i in range(n)]
    best = None
    for q in itertools.product(*[range(x + 1) for x in buy]):
        G = sum(P0[i] * q[i] for i in range(n))
        if fb * G <= b_s and (best is None or q > best):
            best = q
    G = sum(P0[i] * best[i] for i in range(n))
    hh = [hh[i] + best[i] for i in range(n)]
    nb = max(F(0), F(float(b_s - fb * G)))  # one rounding (fma), clamp
    V = F(b) + sum(P0[i] * h[i] for i in range(n))
    V1 = nb + sum(P1[i] * hh[i] for i in range(n))
    c_t = F(fee) * (S + G)
    b_eq3 = F(b) + S - G
    r = scale * (V1 - V)
    return hh, float(nb), float(r), c_t, b_eq3, V, V1


def actions_for(k, hmax):
    """Raw actions that map exactly onto the integers k (k/hmax is a dyadic
    rational for hmax a power of two)."""
    return np.array([ki / hmax for ki in k], dtype=np.float32)


# ---------------------------------------------------------------- hand cases

def test_E1_sell_then_buy_hand_example():
    # b=1000; p=[10,20] -> [11,19]; h=[5,0]; k=[-3,+40]; fee 0.001
    m = mk_market([[10, 20], [11, 19]])
    c = ecfg(hmax=64, fee=1e-3)
    r, nb, h1, t1, diag = oracle.env_step_one(m, c, 1000.0, [5, 0], 0,
                                              actions_for([-3, 40], 64))
    assert list(h1) == [2, 40] and t1 == 1
    # eq.(3) fee-free balance: 1000 + 3*10 - 40*20 = 230; fee paid 0.83
    assert nb == pytest.approx(229.17, abs=1e-9)
    # V = 1050, V' = 229.17 + 2*11 + 40*19 = 1011.17;
    # eq.(2): (230 + 782) - 1050 - c_t, c_t = 0.001*(30+800) = 0.83 -> -38.83
    assert diag[0] == 1050.0
    assert diag[1] == pytest.approx(1011.17, abs=1e-9)
    assert r == pytest.approx(-38.83, rel=1e-6)


def test_E2_cash_clamp_and_E2b_order_matters():
    c = ecfg(hmax=64, fee=1e-3)
    # b=100; p=[10,20]; k=[5,5]: 5 of stock 0 (50.05), then 2 of stock 1
    m = mk_market([[10, 20], [10, 20]])
    r, nb, h1, _, _ = oracle.env_step_one(m, c, 100.0, [0, 0], 0,
                                          actions_for([5, 5], 64))
    assert list(h1) == [5, 2]
    assert nb == pytest.approx(100 - 90 * 1.001, abs=1e-12)   # 9.91
    # same stocks in reverse index order: 4 of the 20-dollar stock, then 1
    m2 = mk_market([[20, 10], [20, 10]])
    r, nb2, h2, _, _ = oracle.env_step_one(m2, c, 100.0, [0, 0], 0,
                                           actions_for([5, 5], 64))
    assert list(h2) == [4, 1]
    assert nb2 == pytest.approx(9.91, abs=1e-12)


# ------------------------------------------------- brute force, random cases

def _random_case(rng, n, hmax):
    # prices inside [2^-2, 2^13) with a mix of magnitudes, fp32
    p0 = np.exp(rng.uniform(np.log(0.25), np.log(8000), n)).astype(np.float32)
    p1 = (p0 * np.exp(rng.normal(0, 0.05, n))).astype(np.float32)
    p1 = np.clip(p1, np.float32(0.25), np.float32(8191))
    h = rng.integers(0, 3 * hmax, n)
    k = rng.integers(-hmax, hmax + 1, n)
    b = float(rng.choice([0.0, rng.uniform(0, 50), rng.uniform(0, 5e3),
                          rng.uniform(0, 1e6)]))
    return p0, p1, b, h, k


@pytest.mark.parametrize("seed", range(6))
def test_step_matches_exact_bruteforce(seed):
    rng = np.random.default_rng(1000 + seed)
    hmax = 8
    fee = [1e-3, 2e-3, 0.0, 0.01, 1e-3, 0.05][seed]
    scale = 2.0 ** -12
    for _ in range(150):
        n = int(rng.integers(1, 5))
        p0, p1, b, h, k = _random_case(rng, n, hmax)
        m = mk_market([p0, p1])
        c = ecfg(hmax=hmax, fee=fee, scale=scale)
        a = actions_for(k, hmax)
        r, nb, h1, _, diag = oracle.env_step_one(m, c, b, h, 0, a)
        eh, eb, er, c_t, b_eq3, V, V1 = exact_step(p0, p1, b, h, list(k),
                                                   fee, scale)
        assert list(h1) == eh                       # bit-exact shares
        assert nb == eb                             # bit-exact balance
        assert r == pytest.approx(np.float32(er), rel=1e-6, abs=1e-12)
        # eq.(2): r/scale = [b_eq3 + p1^T h'] - [b + p0^T h] - c_t
        eq2 = float((b_eq3 + sum(F(float(p1[i])) * eh[i] for i in range(n)))
                    - V - c_t)
        assert (diag[1] - diag[0]) == pytest.approx(eq2, rel=1e-9, abs=1e-7)


def test_buy_rule_is_lexicographic_max_exhaustive():
    # every k vector for n=3, hmax=4 at a budget that binds
    m = mk_market([[3.25, 7.5, 1.75], [3.25, 7.5, 1.75]])
    c = ecfg(hmax=4, fee=1e-3)
    for k in itertools.product(range(-4, 5), repeat=3):
        for b in (0.0, 5.0, 13.37, 29.0, 60.0):
            h = [2, 1, 3]
            r, nb, h1, _, _ = oracle.env_step_one(m, c, b, h, 0,
                                                  actions_for(k, 4))
            eh, eb, *_ = exact_step([3.25, 7.5, 1.75], [3.25, 7.5, 1.75], b,
                                    h, list(k), 1e-3, 1.0)
            assert list(h1) == eh and nb == eb, (k, b)


# --------------------------------------------------------------- invariants

def _dow_market(rows=2521):
    cfg = W.get_config("dow30")
    mk = W.make_market(cfg, rows=(0, rows))
    return cfg, oracle.market(mk.price, mk.ind), mk


def test_zero_action_keeps_portfolio_and_earns_price_change():
    cfg, m, mk = _dow_market(64)
    c = oracle.env_cfg(cfg)
    rng = np.random.default_rng(5)
    E = 32
    cash = rng.uniform(0, 1e6, E)
    shares = rng.integers(0, 5000, (E, cfg.n)).astype(np.int32)
    t = rng.integers(0, 60, E).astype(np.int64)
    c0, s0, t_0 = cash.copy(), shares.copy(), t.copy()
    r, _ = oracle.env_step(m, c, cash, shares, t, np.zeros((E, cfg.n), np.float32))
    assert np.array_equal(cash, c0) and np.array_equal(shares, s0)
    assert np.array_equal(t, t_0 + 1)
    for e in range(E):
        dp = mk.price[t_0[e] + 1].astype(np.float64) - mk.price[t_0[e]]
        expect = np.float32(cfg.reward_scale * float(np.dot(s0[e], dp)))
        assert r[e] == pytest.approx(expect, rel=1e-6, abs=1e-9)


def test_nonnegative_and_asset_identity_under_adversarial_actions():
    """>= 10^5 env-steps of all-buy / all-sell / alternating / NaN / +-Inf
    actions: balance and holdings stay >= 0; V' = b' + p_{t+1}^T h'."""
    cfg, m, mk = _dow_market()
    c = oracle.env_cfg(cfg)
    E, n = 48, cfg.n
    cash, shares, t = oracle.env_reset(c, np.zeros(E, np.int64), n)
    pats = [np.ones(n), -np.ones(n), np.where(np.arange(n) % 2, 1.0, -1.0),
            np.full(n, np.nan), np.full(n, np.inf), np.full(n, -np.inf)]
    rng = np.random.default_rng(11)
    steps = 2200
    for j in range(steps):
        a = np.empty((E, n), np.float32)
        for e in range(E):
            a[e] = pats[(e + j // 7) % len(pats)] if e % 3 else \
                rng.normal(0, 2, n)
        t_before = t.copy()
        r, _ = oracle.env_step(m, c, cash, shares, t, a)
        assert (cash >= 0).all() and (shares >= 0).all()
        if j % 97 == 0:
            for e in range(E):
                V1 = cash[e] + float(np.dot(shares[e].astype(np.float64),
                                            mk.price[t_before[e] + 1]))
                assert np.isfinite(V1) and V1 >= 0
    assert E * steps >= 10 ** 5


def test_fee_identity_from_state_changes():
    """eq.(2) with c_t = fee*(S+G) equals the fee-charged balance update,
    with S, G recovered from the holdings change only."""
    cfg, m, mk = _dow_market(200)
    c = oracle.env_cfg(cfg)
    rng = np.random.default_rng(3)
    E, n = 40, cfg.n
    cash = rng.uniform(0, 2e5, E)
    shares = rng.integers(0, 300, (E, n)).astype(np.int32)
    t = rng.integers(0, 190, E).astype(np.int64)
    for _ in range(5):
        a = rng.normal(0, 0.8, (E, n)).astype(np.float32)
        c0, s0, t0 = cash.copy(), shares.copy(), t.copy()
        r, _ = oracle.env_step(m, c, cash, shares, t, a)
        for e in range(E):
            p0 = mk.price[t0[e]].astype(np.float64)
            p1 = mk.price[t0[e] + 1].astype(np.float64)
            d = shares[e].astype(np.int64) - s0[e]
            S = float(np.dot(p0, np.maximum(-d, 0)))
            G = float(np.dot(p0, np.maximum(d, 0)))
            assert cash[e] == pytest.approx(
                c0[e] + (1 - cfg.fee) * S - (1 + cfg.fee) * G, rel=1e-12,
                abs=1e-6)
            V = c0[e] + float(np.dot(p0, s0[e]))
            V1 = (c0[e] + S - G) + float(np.dot(p1, shares[e]))
            eq2 = V1 - V - cfg.fee * (S + G)
            assert r[e] == pytest.approx(np.float32(cfg.reward_scale * eq2),
                                         rel=2e-6, abs=1e-6)
            # a stock is never both sold and bought in one step; trades
            # never exceed hmax
            assert (np.abs(d) <= cfg.hmax).all()


def test_exact_sums_are_order_independent():
    """Inside the price range, p*q sums (q <= 128, n <= 128) are exact in
    fp64: serial, reversed and pairwise-tree orders agree bitwise."""
    rng = np.random.default_rng(0)
    for _ in range(2000):
        n = int(rng.integers(1, 129))
        p = np.exp(rng.uniform(np.log(0.25), np.log(8191), n)).astype(np.float32)
        q = rng.integers(0, 129, n)
        terms = p.astype(np.float64) * q
        s1 = 0.0
        for x in terms:
            s1 += x
        s2 = 0.0
        for x in terms[::-1]:
            s2 += x
        tt = list(terms)
        while len(tt) > 1:
            tt = [tt[i] + tt[i + 1] if i + 1 < len(tt) else tt[i]
                  for i in range(0, len(tt), 2)]
        exact = sum(F(float(x)) for x in terms)
        assert s1 == s2 == tt[0] == float(exact) and F(s1) == exact


# ---------------------------------------------------------- action mapping

def test_action_mapping():
    hmax = 100
    cases = {0.0: 0, 1.0: 100, -1.0: -100, 7.0: 100, -3.0: -100,
             float("nan"): 0, float("inf"): 100, float("-inf"): -100,
             0.019999: 1, -0.019999: -1, 0.0099999: 0, 0.5: 50, -0.5: -50}
    for a, k in cases.items():
        assert oracle.shares_from_action(a, hmax) == k, a
    # the product is taken in fp32 and truncated toward zero
    rng = np.random.default_rng(2)
    for a in rng.uniform(-1, 1, 2000).astype(np.float32):
        prod = np.float32(a) * np.float32(hmax)
        assert oracle.shares_from_action(float(a), hmax) == int(math.trunc(float(prod)))


def test_reset():
    c = ecfg()
    t0 = np.array([0, 390, 780], np.int64)
    cash, shares, t = oracle.env_reset(c, t0, 7)
    assert (cash == 1e6).all() and (shares == 0).all() and np.array_equal(t, t0)


def test_env_without_next_row_is_not_stepped():
    """An env at the last market row (or before the first) keeps its state
    and reports a NaN reward instead of reading past the market."""
    m = mk_market([[10, 20], [11, 19]])
    c = ecfg(hmax=64)
    for t in (1, -1, 5):
        r, nb, h1, t1, _ = oracle.env_step_one(m, c, 100.0, [3, 4], t,
                                               actions_for([5, -5], 64))
        assert np.isnan(r) and nb == 100.0 and list(h1) == [3, 4] and t1 == t


# ----------------------------------------------------------- observation

def test_observation_layout_and_power_of_two_scales():
    """The state of Section 3 ("State space") is the balance, the prices,
    the holdings and the indicators.  Pinned without the scale constants:
    perturbing one state component moves exactly one observation entry, at
    [balance | n prices | n holdings | n*I indicators, stock-major | zero
    padding]; each block scales its inputs by one power of two, the same for
    every stock (so the observation is exact); indicators enter unscaled;
    the bf16 observation is torch's RNE rounding of the fp32 one.  Which
    powers of two is a reading (the paper gives none)."""
    import torch
    rng = np.random.default_rng(5)
    n, nI, rows = 5, 3, 4
    S = 1 + 2 * n + n * nI
    K_pad = 32
    prices = np.ldexp(rng.integers(1 << 10, 1 << 20, (rows, n)), rng.integers(-10, 4, (rows, n)))
    prices = np.clip(prices, 0.25, 8191.0).astype(np.float32)
    ind = rng.normal(0, 3, (rows, n, nI)).astype(np.float32)
    c = ecfg()
    cash = 765432.0                                  # exact in fp32
    shares = rng.integers(0, 5000, n).astype(np.int32)

    def obs(p=prices, x=ind, b=cash, h=shares, t=2, bf16=False):
        return oracle.obs(oracle.market(p, x), c, t, b, h, K_pad, bf16)

    base = obs()
    assert base.shape == (K_pad,) and (base[S:] == 0).all()
    # one component -> one entry
    moved = []
    moved.append(np.flatnonzero(obs(b=cash + 4096.0) != base))
    for i in range(n):
        p2 = prices.copy()
        p2[2, i] *= 2
        moved.append(np.flatnonzero(obs(p=p2) != base))
    for i in range(n):
        h2 = shares.copy()
        h2[i] += 7
        moved.append(np.flatnonzero(obs(h=h2) != base))
    for i in range(n):
        for k in range(nI):
            x2 = ind.copy()
            x2[2, i, k] += 1.0
            moved.append(np.flatnonzero(obs(x=x2) != base))
    assert [list(m) for m in moved] == [[j] for j in range(S)]
    # other market rows do not enter the observation of row t
    p3, x3 = prices.copy(), ind.copy()
    p3[[0, 1, 3]] *= 2
    x3[[0, 1, 3]] += 1
    assert np.array_equal(obs(p=p3, x=x3), base)

    def pow2_ratio(num, den):
        r = np.asarray(num, np.float64) / np.asarray(den, np.float64)
        e = np.log2(r)
        assert np.all(r > 0) and np.all(e == np.round(e)), r
        return set(np.round(e).astype(int).tolist())

    # one power of two per block, shared by every stock, row and value
    e_cash = pow2_ratio([obs(b=b)[0] for b in (cash, 1.0, 3.0 * 2 ** 20, 123456.0)],
                        [cash, 1.0, 3.0 * 2 ** 20, 123456.0])
    e_p = pow2_ratio(np.concatenate([obs(t=t)[1:1 + n] for t in range(rows)]), prices.ravel())
    nz = shares != 0
    e_h = pow2_ratio(base[1 + n:1 + 2 * n][nz], shares[nz])
    assert len(e_cash) == 1 and len(e_p) == 1 and len(e_h) == 1
    assert np.array_equal(np.concatenate([obs(t=t)[1 + 2 * n:S] for t in range(rows)]),
                          ind.reshape(rows, -1).ravel())
    # bf16 = RNE of the fp32 observation
    want = torch.from_numpy(base).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(obs(bf16=True), want)


def test_parallel_replay_equals_serial():
    """The GPU tests replay sampled envs through the oracle in chunks on a
    thread pool; the joined result equals one serial call bit for bit."""
    import workloads as W
    from gpu_common import oracle_replay
    cfg = W.get_config("tiny")
    mk = W.make_market(cfg)
    t0 = W.make_t0(cfg)
    params = W.make_actor(cfg)
    ids = np.array([0, 3, 5, 9, 17, 33, 40, 41, 50, 63])
    teacher = np.random.default_rng(1).normal(0, 0.7, (60, len(ids), cfg.n)).astype(np.float32)
    a = oracle_replay(cfg, mk, params, t0[ids], ids, 99, 60, teacher, cfg.envs_per_agent, chunk=3)
    b = oracle_replay(cfg, mk, params, t0[ids], ids, 99, 60, teacher, cfg.envs_per_agent,
                      chunk=100)
    assert a.keys() == b.keys()
    for k in a:
        if k == "final":
            for x, y in zip(a[k], b[k]):
                assert np.array_equal(x, y)
        else:
            assert np.array_equal(a[k], b[k], equal_nan=True), k


def test_openmp_build_equals_plain_build():
    """The CPU baseline's all-core leg runs the OpenMP build of the same
    oracle source; its free-running rollout equals the plain build's bit
    for bit (envs are independent), here on 24 envs of the 100-stock shape
    with a small actor and on the tiny workload."""
    import oracle
    import workloads as W
    assert oracle.threads(False) == 1 and oracle.threads(True) >= 1
    for cfg in (W.get_config("nasdaq100").with_(N=3 * 390, E=24, hidden=(128, 128)),
                W.get_config("tiny")):
        mk = W.make_market(cfg)
        t0 = W.make_t0(cfg)
        params = W.make_actor(cfg)
        m = oracle.market(mk.price, mk.ind)
        ec = oracle.env_cfg(cfg)
        act = oracle.actor(*params, cfg.dims, cfg.dtype == "bf16", cfg.envs_per_agent)
        outs = []
        for omp in (False, True):
            cash, sh, t = oracle.env_reset(ec, t0, cfg.n)
            o = oracle.rollout(m, ec, act, cash, sh, t, 5, 0, 40, cfg.K_pad, omp=omp)
            o["state"] = (cash, sh, t)
            outs.append(o)
        a, b = outs
        for k in a:
            if k == "state":
                assert all(np.array_equal(x, y) for x, y in zip(a[k], b[k]))
            else:
                assert np.array_equal(a[k], b[k], equal_nan=True), k
