"""Pins for the oracle's GAE / reward-to-go.

GAE is PPO's advantage estimator (PPO is named in the paper's Section 5.2;
gamma = 0.99 from Table 2; the return definition is eq. (1)).  Expected
values come from hand-worked cases in exact rationals, the lambda = 0 and
lambda = 1 closed forms (TD residual; discounted return minus V) and the
geometric-series closed form for constant inputs.
"""

from fractions import Fraction as F

import numpy as np
import pytest

import oracle


def run(r, v, d, g, lam):
    r = np.asarray(r, np.float32).reshape(-1, 1)
    v = np.asarray(v, np.float32).reshape(-1, 1)
    d = np.asarray(d, np.uint8).reshape(-1, 1)
    adv, ret = oracle.gae(r, v, d, g, lam)
    return adv[:, 0], ret[:, 0]


def test_G1_hand_example():
    # L=3, gamma=0.9, lambda=0.5, r=[1,2,3], V=[0.5,1,1.5,2], no done.
    # delta = [1+0.9*1-0.5, 2+0.9*1.5-1, 3+0.9*2-1.5] = [1.4, 2.35, 3.3]
    # A2 = 3.3; A1 = 2.35 + 0.45*3.3 = 3.835; A0 = 1.4 + 0.45*3.835 = 3.12575
    adv, ret = run([1, 2, 3], [0.5, 1, 1.5, 2], [0, 0, 0], 0.9, 0.5)
    assert adv == pytest.approx([3.12575, 3.835, 3.3], rel=1e-6)
    assert ret == pytest.approx([3.62575, 4.835, 4.8], rel=1e-6)
    # lambda = 1: A0 = 1 + 0.9*2 + 0.81*3 + 0.729*2 - 0.5 = 6.188
    adv1, _ = run([1, 2, 3], [0.5, 1, 1.5, 2], [0, 0, 0], 0.9, 1.0)
    assert adv1[0] == pytest.approx(6.188, rel=1e-6)
    # lambda = 0: A = delta
    adv0, _ = run([1, 2, 3], [0.5, 1, 1.5, 2], [0, 0, 0], 0.9, 0.0)
    assert adv0 == pytest.approx([1.4, 2.35, 3.3], rel=1e-6)


def test_G2_done_cuts_bootstrap_and_carry():
    # as G1 with d = [0, 1, 0]: step 1 ends an episode.
    # delta1 = 2 - 1 = 1 (no bootstrap), A1 = 1 (no carry)
    # A0 = 1.4 + 0.45 * 1 = 1.85; A2 = 3.3
    adv, _ = run([1, 2, 3], [0.5, 1, 1.5, 2], [0, 1, 0], 0.9, 0.5)
    assert adv == pytest.approx([1.85, 1.0, 3.3], rel=1e-6)


def _exact_lambda_return(r, v, d, g, lam):
    """Exact rationals, straight from the n-step definition: the GAE(lambda)
    advantage is the (1-lambda)-weighted mix of k-step advantages, which for
    lambda in {0, 1} reduces to the TD residual / discounted return - V."""
    L = len(r)
    g = F(float(np.float32(g)))
    out = []
    for j in range(L):
        if lam == 0.0:
            nd = 0 if d[j] else 1
            out.append(F(float(r[j])) + g * nd * F(float(v[j + 1])) - F(float(v[j])))
        else:  # lam == 1: discounted return to the episode end (+ bootstrap)
            acc, disc, k = F(0), F(1), j
            while True:
                acc += disc * F(float(r[k]))
                if d[k]:
                    break
                disc *= g
                k += 1
                if k == L:
                    acc += disc * F(float(v[L]))
                    break
            out.append(acc - F(float(v[j])))
    return out


@pytest.mark.parametrize("lam", [0.0, 1.0])
def test_lambda_closed_forms_random(lam):
    rng = np.random.default_rng(int(lam * 10) + 1)
    L, E = 120, 6
    r = rng.normal(size=(L, E)).astype(np.float32)
    v = rng.normal(size=(L + 1, E)).astype(np.float32)
    d = (rng.random((L, E)) < 0.05).astype(np.uint8)
    adv, ret = oracle.gae(r, v, d, 0.99, lam)
    for e in range(E):
        ex = _exact_lambda_return(r[:, e], v[:, e], d[:, e], 0.99, lam)
        scale = max(1.0, float(np.sqrt(np.mean(np.square(adv[:, e])))))
        for j in range(L):
            assert abs(adv[j, e] - float(ex[j])) <= 1e-6 * max(abs(float(ex[j])), scale)
            assert ret[j, e] == pytest.approx(np.float32(float(ex[j]) + float(v[j, e])),
                                              rel=1e-6, abs=1e-6)


def test_constant_inputs_geometric_closed_form_long_horizon():
    # constant r, V, no done, L = 2520 (the Dow-30 daily episode):
    # A_j = delta * (1 - (g*l)^(L-j)) / (1 - g*l),  delta = r + (g-1) V
    L, r0, v0 = 2520, 0.37, 1.25
    g, lam = np.float32(0.99), np.float32(0.95)
    adv, _ = run(np.full(L, r0), np.full(L + 1, v0), np.zeros(L), g, lam)
    gd, gl = float(g), float(g) * float(lam)
    delta = float(np.float32(r0)) + (gd - 1) * float(np.float32(v0))
    for j in (0, 1, 100, 1000, L - 2, L - 1):
        expect = delta * (1 - gl ** (L - j)) / (1 - gl)
        assert adv[j] == pytest.approx(expect, rel=1e-6)


def test_envs_are_independent_columns():
    rng = np.random.default_rng(9)
    L, E = 50, 5
    r = rng.normal(size=(L, E)).astype(np.float32)
    v = rng.normal(size=(L + 1, E)).astype(np.float32)
    d = (rng.random((L, E)) < 0.1).astype(np.uint8)
    adv, ret = oracle.gae(r, v, d, 0.99, 0.95)
    for e in range(E):
        a1, r1 = oracle.gae(r[:, e:e + 1], v[:, e:e + 1], d[:, e:e + 1], 0.99, 0.95)
        assert np.array_equal(a1[:, 0], adv[:, e]) and np.array_equal(r1[:, 0], ret[:, e])
