"""Pins for the oracle's evolution layer (Section 4.2): ensemble fusion
against numpy's mean, the fitness of eq. (1) against closed forms and exact
rational brute force, keep-best bookkeeping on a hand sequence, and the
selector's ranking and redistribution against a sort written from the
definition."""

import math
from fractions import Fraction

import numpy as np

import oracle


def test_fuse_is_the_mean_over_pods():
    rng = np.random.default_rng(1)
    p = rng.standard_normal((3, 4, 257)).astype(np.float32)
    f = oracle.ensemble_fuse(p)
    want = p.astype(np.float64).mean(axis=1).astype(np.float32)
    for k in range(4):
        np.testing.assert_array_equal(f[:, k], want)
    # integer data: the mean is exact
    q = rng.integers(-50, 50, (2, 5, 33)).astype(np.float32) * 5
    np.testing.assert_array_equal(oracle.ensemble_fuse(q)[:, 0], q.sum(axis=1) / 5)


def test_fuse_single_pod_is_identity():
    p = np.random.default_rng(2).standard_normal((4, 1, 100)).astype(np.float32)
    np.testing.assert_array_equal(oracle.ensemble_fuse(p), p)


def test_fitness_closed_forms():
    L, E, A, g = 390, 8, 2, 0.99
    r = np.full((L, E), 0.25, np.float32)
    f = oracle.fitness(r, A, g)
    np.testing.assert_allclose(f, 0.25 * (1 - g ** L) / (1 - g), rtol=1e-12)
    # gamma = 1: the plain sum
    r = np.random.default_rng(3).standard_normal((50, E)).astype(np.float32)
    f = oracle.fitness(r, 4, 1.0)
    want = r.astype(np.float64).sum(0).reshape(4, 2).mean(1)
    np.testing.assert_allclose(f, want, rtol=1e-12)


def test_fitness_brute_force_rationals():
    rng = np.random.default_rng(4)
    L, E, A = 7, 6, 3
    r = (rng.integers(-20, 20, (L, E)) / 8).astype(np.float32)   # exact in fp32
    g = 0.5                                                     # exact powers
    f = oracle.fitness(r, A, g)
    for a in range(A):
        tot = Fraction(0)
        for e in range(2 * a, 2 * a + 2):
            tot += sum(Fraction(float(r[j, e])) * Fraction(1, 2 ** j) for j in range(L))
        assert f[a] == float(tot / 2)


def test_fitness_skips_envs_that_were_not_stepped():
    r = np.ones((5, 4), np.float32)
    r[:, 1] = np.nan
    r[:, 2:] = np.nan
    f = oracle.fitness(r, 2, 1.0)
    assert f[0] == 5.0 and math.isnan(f[1])


def test_keep_best_sequence():
    P = 3
    params = np.arange(2 * P, dtype=np.float32).reshape(2, P)
    best = np.array([np.nan, 1.0])
    stall = np.zeros(2, np.int32)
    bp = np.zeros((2, P), np.float32)
    best, stall, bp = oracle.keep_best([0.5, 0.9], best, stall, params, bp)
    assert list(best) == [0.5, 1.0] and list(stall) == [0, 1]
    np.testing.assert_array_equal(bp[0], params[0])
    np.testing.assert_array_equal(bp[1], 0)
    best, stall, bp = oracle.keep_best([0.4, 1.5], best, stall, params + 10, bp)
    assert list(best) == [0.5, 1.5] and list(stall) == [1, 0]
    np.testing.assert_array_equal(bp[0], params[0])
    np.testing.assert_array_equal(bp[1], params[1] + 10)
    best, stall, bp = oracle.keep_best([np.nan, 1.5], best, stall, params, bp)
    assert list(stall) == [2, 1]       # NaN never beats; a tie is no improvement


def test_select_against_definition():
    rng = np.random.default_rng(5)
    for _ in range(30):
        N = int(rng.integers(1, 20))
        fit = rng.integers(0, 5, N).astype(np.float64)      # ties on purpose
        fit[rng.random(N) < 0.2] = np.nan
        keep = int(rng.integers(1, N + 1))
        P = 4
        params = rng.standard_normal((N, P)).astype(np.float32)
        rank, newp = oracle.select(fit, params, keep)
        order = sorted(range(N), key=lambda i: (math.isnan(fit[i]),
                                                -fit[i] if not math.isnan(fit[i]) else 0, i))
        assert [int(rank[i]) for i in order] == list(range(N))
        for r, i in enumerate(order):
            src = i if r < keep else order[(r - keep) % keep]
            np.testing.assert_array_equal(newp[i], params[src])
