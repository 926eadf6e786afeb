"""GPU parity of the evolution layer (Section 4.2) against the oracle:
ensemble fusion, the fitness of eq. (1) with envs that were not stepped,
keep-best bookkeeping over a sequence of evaluations, and the selector with
ties and NaN fitness, all bit-exact (every reduction runs in the oracle's
order and the library is built without fma contraction)."""

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_common import build_problem, say
from paper_2111_05188_amd import tp

pytestmark = pytest.mark.gpu


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("N,K,P", [(3, 4, 100003), (1, 1, 7), (4, 2, 1 << 20), (2, 8, 513)])
def test_ensemble_fuse(N, K, P):
    say(f"[fuse] N={N} K={K} P={P}")
    rng = np.random.default_rng(N * 1000 + K)
    p = rng.standard_normal((N, K, P)).astype(np.float32)
    d = _dev(p)
    tp.ensemble_fuse(d)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(d.cpu().numpy(), oracle.ensemble_fuse(p))


@pytest.mark.parametrize("L,E,A,gamma", [(390, 4096, 4, 0.99), (7, 300, 3, 1.0),
                                         (1, 1, 1, 0.5), (391, 1000, 8, 0.999)])
def test_fitness(L, E, A, gamma):
    say(f"[fitness] L={L} E={E} A={A} gamma={gamma}")
    rng = np.random.default_rng(L + E)
    r = (rng.standard_normal((L, E)) * 2.0 ** -8).astype(np.float32)
    # envs never stepped (NaN rewards), a whole agent among them when A > 1
    r[:, rng.random(E) < 0.1] = np.nan
    if A > 1:
        r[:, : E // A] = np.nan
    d = _dev(r)
    fit, ret = tp.fitness(d, A, gamma)
    torch.cuda.synchronize()
    want = oracle.fitness(r, A, gamma)
    np.testing.assert_array_equal(fit.cpu().numpy(), want)
    if A > 1:
        assert np.isnan(want[0])


def test_fitness_of_a_rollout():
    """Fitness of the rewards a GPU rollout wrote (the evaluator's input)."""
    cfg = W.get_config("ensemble")
    c = cfg.with_(N=20 * 390, E=240, L=60)
    mk = W.make_market(c)
    pb, _ = build_problem(c, mk, W.make_t0(c), taps=False)
    pb.reset()
    pb.rollout(0xE7A1, 0, c.L)
    torch.cuda.synchronize()
    r = pb.traj.reward.cpu().numpy()
    fit, _ = tp.fitness(pb.traj.reward, c.n_agents, 0.99)
    np.testing.assert_array_equal(fit.cpu().numpy(), oracle.fitness(r, c.n_agents, 0.99))


def test_keep_best_sequence():
    A, P = 5, 70001
    rng = np.random.default_rng(11)
    best = np.full(A, np.nan)
    stall = np.zeros(A, np.int32)
    bp = np.zeros((A, P), np.float32)
    db, ds, dbp = _dev(best), _dev(stall), _dev(bp)
    for it in range(4):
        fit = rng.integers(0, 4, A).astype(np.float64)
        fit[rng.random(A) < 0.2] = np.nan
        params = rng.standard_normal((A, P)).astype(np.float32)
        say(f"[keep_best] call {it} fit={fit}")
        tp.keep_best(_dev(fit), db, ds, _dev(params), dbp)
        best, stall, bp = oracle.keep_best(fit, best, stall, params, bp)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(db.cpu().numpy(), best)
        np.testing.assert_array_equal(ds.cpu().numpy(), stall)
        np.testing.assert_array_equal(dbp.cpu().numpy(), bp)


@pytest.mark.parametrize("N,P,keep", [(1, 5, 1), (8, 1001, 3), (100, 4099, 25),
                                      (1024, 257, 512), (37, 65536 + 3, 37)])
def test_select(N, P, keep):
    say(f"[select] N={N} P={P} keep={keep}")
    rng = np.random.default_rng(N + P)
    fit = rng.integers(0, max(2, N // 4), N).astype(np.float64)   # ties on purpose
    fit[rng.random(N) < 0.15] = np.nan
    params = rng.standard_normal((N, P)).astype(np.float32)
    dp = _dev(params)
    rank = tp.select(_dev(fit), dp, keep)
    torch.cuda.synchronize()
    want_rank, want_p = oracle.select(fit, params, keep)
    np.testing.assert_array_equal(rank.cpu().numpy(), want_rank)
    np.testing.assert_array_equal(dp.cpu().numpy(), want_p)
