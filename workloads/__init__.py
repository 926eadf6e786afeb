"""Seeded synthetic workloads shared by the GPU path's tests/bench and the oracle.

This module holds the five workload configurations and the seeded input
generators: the market tensor (closing prices + technical indicators), the
episode start rows, the actor's fp32 master weights, the critic values fed to
GAE and adversarial action batches.  It holds none of the method's arithmetic
(no env step, no MLP, no sampling, no GAE): both the HIP path and the oracle
receive exactly these arrays as inputs.

The paper trains on NASDAQ-100 minute and daily bars (Section 5.2, "Data
pre-processing"; Dow 30 is named as the small universe in Section 3); those datasets are not available here, so geometric
Brownian motion prices with N(0,1) indicators of the same shapes stand in for
them (state definition: Section 3, "State space").

Every generator is deterministic in (seed, shape) and independent of the
number of worker threads: the market is produced in fixed row blocks, each
from its own ``numpy.random.Generator`` derived from ``SeedSequence(seed,
block)``, so any row range can be regenerated on its own.
"""

from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field, replace

import numpy as np

__all__ = [
    "Config", "CONFIGS", "get_config", "Market", "make_market", "make_t0",
    "make_actor", "make_critic", "make_values", "make_actions", "K_PAD_MULTIPLE",
    "make_flat_params", "make_learner_data", "LOG_RATIO_OFFSETS",
]

# Observation rows are padded to a multiple of the bf16 MFMA k-step.
K_PAD_MULTIPLE = 32
# Row block used by the market generator (fixed: part of the data definition).
_BLOCK_ROWS = 4096
# Minutes per trading day and trading days per year for the minute workloads.
MINUTES_PER_DAY = 390
DAYS_PER_YEAR = 252


@dataclass(frozen=True)
class Config:
    """One workload: market shape, env batch, actor shape and MDP constants."""
    name: str
    n: int                 # stocks
    n_ind: int             # technical indicators per stock
    N: int                 # GBM increments; the market has T1 = N + 1 rows
    sigma: float           # per-bar log-return volatility
    E: int                 # envs (all agents together)
    L: int                 # rollout length (= episode length, horizon)
    t0_mode: str           # "zero": every env starts at row 0; "day": 390*d
    hidden: tuple          # (H1, H2)
    dtype: str             # "f32" or "bf16" (actor + observation storage)
    n_agents: int = 1
    hmax: int = 100
    fee: float = 1e-3
    cash0: float = 1e6
    gamma: float = 0.99
    lam: float = 0.95
    reward_scale: float = 2.0 ** -12
    cash_scale: float = 2.0 ** -20
    price_scale: float = 2.0 ** -7
    share_scale: float = 2.0 ** -7
    log_std_init: float = -0.5
    seeds: dict = field(default_factory=lambda: dict(
        market=20211109, t0=7, actor=1234, values=99, philox=0x5EED_0F_F1_2C,
        critic=4321, learner=2718))

    @property
    def T1(self) -> int:
        return self.N + 1

    @property
    def S(self) -> int:
        """State dimension: balance, n prices, n holdings, n*I indicators."""
        return 1 + 2 * self.n + self.n * self.n_ind

    @property
    def K_pad(self) -> int:
        return -(-self.S // K_PAD_MULTIPLE) * K_PAD_MULTIPLE

    @property
    def dims(self) -> tuple:
        return (self.S, self.hidden[0], self.hidden[1], self.n)

    @property
    def envs_per_agent(self) -> int:
        assert self.E % self.n_agents == 0
        return self.E // self.n_agents

    def flops_per_env_step(self) -> int:
        """2 * sum(in*out) over the three actor layers (unpadded)."""
        S, H1, H2, n = self.dims
        return 2 * (S * H1 + H1 * H2 + H2 * n)

    def with_(self, **kw) -> "Config":
        return replace(self, **kw)


_TINY = Config("tiny", n=5, n_ind=4, N=256, sigma=0.02, E=64, L=256,
               t0_mode="zero", hidden=(64, 64), dtype="f32")
_DOW = Config("dow30", n=30, n_ind=8, N=2520, sigma=0.015, E=1024, L=2520,
              t0_mode="zero", hidden=(256, 256), dtype="f32")
_NASDAQ = Config("nasdaq100", n=100, n_ind=8,
                 N=10 * DAYS_PER_YEAR * MINUTES_PER_DAY, sigma=0.001, E=4096,
                 L=MINUTES_PER_DAY, t0_mode="day", hidden=(512, 512),
                 dtype="bf16")
_ENSEMBLE = _NASDAQ.with_(name="ensemble", E=16 * 1024, n_agents=16)
_STRESS = _NASDAQ.with_(name="stress", E=65536, hidden=(1024, 1024))

CONFIGS = {c.name: c for c in (_TINY, _DOW, _NASDAQ, _ENSEMBLE, _STRESS)}


def get_config(name: str) -> Config:
    return CONFIGS[name]


# --------------------------------------------------------------------------
# market
# --------------------------------------------------------------------------

@dataclass
class Market:
    """price fp32 [T1][n]; ind fp32 [T1][n][I]; rows [row0, row0+rows)."""
    price: np.ndarray
    ind: np.ndarray
    row0: int = 0


def _block_rng(seed: int, stream: int, block: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([seed & 0xFFFFFFFF, stream, block])))


def _workers() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def make_market(cfg: Config, seed: int | None = None, rows: tuple | None = None,
                with_ind: bool = True) -> Market:
    """Seeded GBM close prices and N(0,1) indicators.

    Prices: S0_i ~ U[20, 200]; log p_{t+1} = log p_t - sigma^2/2 + sigma*Z in
    fp64 (drift 0, Ito-corrected so prices are a martingale), cast to fp32 and
    clamped to [0.25, 8191] so every price lies in [2^-2, 2^13).
    Indicators: N(0,1) fp32, stock-major within a row ([n][I]).

    ``rows=(r0, r1)`` returns only rows r0..r1-1 (the price walk is still
    integrated from row 0, block by block).
    """
    seed = cfg.seeds["market"] if seed is None else seed
    n, I, T1 = cfg.n, cfg.n_ind, cfg.T1
    r0, r1 = (0, T1) if rows is None else rows
    assert 0 <= r0 < r1 <= T1
    s0 = _block_rng(seed, 0, 0).uniform(20.0, 200.0, size=n)
    half_var = 0.5 * cfg.sigma * cfg.sigma

    def incr(b):
        # increments that lead INTO rows b*BR .. (b+1)*BR-1 (row 0 has none)
        lo, hi = b * _BLOCK_ROWS, min(T1, (b + 1) * _BLOCK_ROWS)
        z = _block_rng(seed, 1, b).standard_normal((hi - lo, n),
                                                  dtype=np.float32)
        d = z.astype(np.float64) * cfg.sigma - half_var
        if lo == 0:
            d[0] = 0.0
        return d

    blk_lo, blk_hi = r0 // _BLOCK_ROWS, (r1 - 1) // _BLOCK_ROWS
    # log-price offset at the start of each needed block: sum of all earlier
    # blocks' increments (computed block-wise, in parallel)
    with ThreadPoolExecutor(_workers()) as ex:
        sums = list(ex.map(lambda b: incr(b).sum(axis=0), range(blk_lo)))
    base = np.log(s0)
    for s in sums:          # sequential, same order as the prefix below
        base = base + s

    price = np.empty((r1 - r0, n), dtype=np.float32)
    ind = np.empty((r1 - r0, n, I), dtype=np.float32) if with_ind else None

    def fill(b, start_log):
        lo, hi = b * _BLOCK_ROWS, min(T1, (b + 1) * _BLOCK_ROWS)
        lp = start_log + np.cumsum(incr(b), axis=0)
        p = np.clip(np.exp(lp).astype(np.float32), np.float32(0.25),
                    np.float32(8191.0))
        a, c = max(lo, r0), min(hi, r1)
        if a < c:
            price[a - r0:c - r0] = p[a - lo:c - lo]
            if with_ind:
                g = _block_rng(seed, 2, b).standard_normal(
                    (hi - lo, n, I), dtype=np.float32)
                ind[a - r0:c - r0] = g[a - lo:c - lo]

    # block starting log-prices need a sequential prefix; compute sums first
    with ThreadPoolExecutor(_workers()) as ex:
        bsums = list(ex.map(lambda b: incr(b).sum(axis=0),
                            range(blk_lo, blk_hi + 1)))
    starts, acc = [], base
    for s in bsums:
        starts.append(acc)
        acc = acc + s
    with ThreadPoolExecutor(_workers()) as ex:
        list(ex.map(lambda a: fill(*a),
                    zip(range(blk_lo, blk_hi + 1), starts)))
    return Market(price=price, ind=ind if with_ind else None, row0=r0)


# --------------------------------------------------------------------------
# env start rows, actor weights, values, actions
# --------------------------------------------------------------------------

def make_t0(cfg: Config, seed: int | None = None, E: int | None = None):
    """Episode start rows int64 [E]: 0, or 390*d with d ~ U{0..days-1}."""
    seed = cfg.seeds["t0"] if seed is None else seed
    E = cfg.E if E is None else E
    if cfg.t0_mode == "zero":
        return np.zeros(E, dtype=np.int64)
    days = (cfg.T1 - 1) // MINUTES_PER_DAY
    # an episode of L steps needs rows t0..t0+L; the last day ends at row N
    max_day = (cfg.T1 - 1 - cfg.L) // MINUTES_PER_DAY
    assert max_day < days
    d = np.random.default_rng(seed).integers(0, max_day + 1, size=E)
    return (d * MINUTES_PER_DAY).astype(np.int64)


def make_actor(cfg: Config, seed: int | None = None, n_agents: int | None = None):
    """fp32 master weights: W_l [A][out][in], b_l [A][out] ~ U(+-1/sqrt(in));
    log_std [A][n] = log_std_init.  Each agent draws from its own stream."""
    seed = cfg.seeds["actor"] if seed is None else seed
    A = cfg.n_agents if n_agents is None else n_agents
    S, H1, H2, n = cfg.dims
    shapes = [(H1, S), (H2, H1), (n, H2)]
    W = [np.empty((A,) + s, dtype=np.float32) for s in shapes]
    b = [np.empty((A, s[0]), dtype=np.float32) for s in shapes]
    for a in range(A):
        rng = _block_rng(seed, 3, a)
        for l, (o, i) in enumerate(shapes):
            bound = 1.0 / math.sqrt(i)
            W[l][a] = rng.uniform(-bound, bound, size=(o, i)).astype(np.float32)
            b[l][a] = rng.uniform(-bound, bound, size=o).astype(np.float32)
    log_std = np.full((A, n), cfg.log_std_init, dtype=np.float32)
    return W, b, log_std


def make_critic(cfg: Config, seed: int | None = None, n_agents: int | None = None):
    """fp32 master weights of the critic S-H1-H2-1: W_l [A][out][in] (the last
    one [A][H2]), b_l [A][out] (the last one [A]) ~ U(+-1/sqrt(in)), one
    stream per agent."""
    seed = cfg.seeds["critic"] if seed is None else seed
    A = cfg.n_agents if n_agents is None else n_agents
    S, H1, H2, _ = cfg.dims
    shapes = [(H1, S), (H2, H1), (1, H2)]
    W = [np.empty((A,) + s, dtype=np.float32) for s in shapes]
    b = [np.empty((A, s[0]), dtype=np.float32) for s in shapes]
    for a in range(A):
        rng = _block_rng(seed, 4, a)
        for l, (o, i) in enumerate(shapes):
            bound = 1.0 / math.sqrt(i)
            W[l][a] = rng.uniform(-bound, bound, size=(o, i)).astype(np.float32)
            b[l][a] = rng.uniform(-bound, bound, size=o).astype(np.float32)
    W[2] = W[2].reshape(A, H2)
    b[2] = b[2].reshape(A)
    return W, b


def make_values(cfg: Config, seed: int | None = None, L: int | None = None,
                E: int | None = None):
    """Critic values fp32 [L+1][E] ~ N(0,1) (the last row is the bootstrap)."""
    seed = cfg.seeds["values"] if seed is None else seed
    L = cfg.L if L is None else L
    E = cfg.E if E is None else E
    return np.random.default_rng(seed).standard_normal(
        (L + 1, E), dtype=np.float32)


def make_actions(seed: int, E: int, n: int, special: bool = True):
    """Raw actions fp32 [E][n]: mostly N(0, 0.6^2); with ``special`` a share
    of entries is set to exactly +-1, 0, values beyond the clip range, NaN and
    +-Inf (the adversarial cases of the action mapping)."""
    rng = np.random.default_rng(seed)
    a = (0.6 * rng.standard_normal((E, n))).astype(np.float32)
    if special:
        m = rng.random((E, n))
        a[m < 0.03] = 1.0
        a[(m >= 0.03) & (m < 0.06)] = -1.0
        a[(m >= 0.06) & (m < 0.08)] = 0.0
        a[(m >= 0.08) & (m < 0.10)] = np.float32(3.5)
        a[(m >= 0.10) & (m < 0.11)] = np.nan
        a[(m >= 0.11) & (m < 0.115)] = np.inf
        a[(m >= 0.115) & (m < 0.12)] = -np.inf
    return a


def make_flat_params(cfg: Config, agent: int = 0) -> np.ndarray:
    """One agent's actor and critic (make_actor, make_critic) as one flat fp32
    vector, segments in the order W1, b1, W2, b2, W3, b3, log_std, Wc1, bc1,
    Wc2, bc2, wc3, bc3."""
    # each agent draws from its own stream, so agent a's vector does not
    # depend on how many agents the config has
    A = max(cfg.n_agents, agent + 1)
    W, b, ls = make_actor(cfg, n_agents=A)
    Wc, bc = make_critic(cfg, n_agents=A)
    parts = [W[0][agent], b[0][agent], W[1][agent], b[1][agent], W[2][agent], b[2][agent],
             ls[agent], Wc[0][agent], bc[0][agent], Wc[1][agent], bc[1][agent], Wc[2][agent],
             bc[2][agent:agent + 1]]
    return np.concatenate([np.asarray(p, np.float32).reshape(-1) for p in parts])


# log(rho) offsets the learner inputs draw from: two inside the ratio clip
# (|log rho| = 0.1), two well outside (0.6), one at rho = 1; none within
# reach of the clip edges ln(0.75) and ln(1.25).
LOG_RATIO_OFFSETS = (-0.6, -0.1, 0.0, 0.1, 0.6)


def make_learner_data(cfg: Config, rows: int, seed: int | None = None):
    """Synthetic stored transitions for the learner: observation rows fp32
    [rows][K_pad] with the observation's structure (cash scaled near 1,
    prices and holdings scaled by 2^-7, N(0,1) indicators, zero padding),
    raw actions N(0, 0.6^2) [rows][n], advantages and returns N(0,1) [rows],
    and an index into LOG_RATIO_OFFSETS per row (the test turns it into the
    stored log-probability)."""
    seed = cfg.seeds["learner"] if seed is None else seed
    rng = _block_rng(seed, 5, 0)
    n, I, K = cfg.n, cfg.n_ind, cfg.K_pad
    obs = np.zeros((rows, K), dtype=np.float32)
    obs[:, 0] = rng.uniform(0.5, 1.5, rows)
    obs[:, 1:1 + n] = rng.uniform(20.0, 200.0, (rows, n)) / 128.0
    obs[:, 1 + n:1 + 2 * n] = rng.integers(0, 300, (rows, n)) / 128.0
    obs[:, 1 + 2 * n:1 + 2 * n + n * I] = rng.standard_normal((rows, n * I))
    action = (0.6 * rng.standard_normal((rows, n))).astype(np.float32)
    adv = rng.standard_normal(rows).astype(np.float32)
    ret = rng.standard_normal(rows).astype(np.float32)
    which = rng.integers(0, len(LOG_RATIO_OFFSETS), rows)
    return obs, action, adv, ret, which
