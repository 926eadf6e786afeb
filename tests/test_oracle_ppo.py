"""Pins for the oracle's PPO learner (Section 5.2, PPO; Table 2): the
log-density and entropy against scipy, the whole gradient against central
finite differences of the loss (actor and critic, both clip branches
present), the clipped-surrogate case analysis of Schulman et al. (which
samples contribute), the closed form at rho = 1, the entropy term's
gradient, and Adam against torch.optim.Adam."""

import math

import numpy as np
import pytest
import scipy.stats
import torch

from oracle import ppo

DIMS = (7, 6, 5, 3, 4, 5)          # S, H1, H2, n, C1, C2


def _params(rng, dims=DIMS, scale=0.6):
    P = ppo.param_count(*dims)
    flat = rng.uniform(-scale, scale, P)
    p = ppo.unflatten(flat, dims)
    p["log_std"][:] = rng.uniform(-0.7, 0.2, dims[3])
    return flat


def _batch(rng, flat, B=9, dims=DIMS, spread=0.4):
    S, n = dims[0], dims[3]
    x = rng.standard_normal((B, S))
    p = ppo.unflatten(flat, dims)
    f = ppo.forward(p, x, bf16=False, exact=True)
    a = f["mu"] + rng.standard_normal((B, n)) * np.exp(p["log_std"])
    lp = ppo.log_prob(a, f["mu"], p["log_std"])
    # old log-probabilities spread so that rho lands on both sides of the clip
    logp_old = lp + rng.uniform(-spread, spread, B)
    adv = rng.standard_normal(B)
    ret = rng.standard_normal(B)
    return x, a, logp_old, adv, ret


def test_log_prob_and_entropy_against_scipy():
    rng = np.random.default_rng(1)
    mu = rng.standard_normal((5, 4))
    ls = rng.uniform(-1, 0.5, 4)
    a = rng.standard_normal((5, 4))
    want = scipy.stats.norm.logpdf(a, loc=mu, scale=np.exp(ls)).sum(axis=1)
    np.testing.assert_allclose(ppo.log_prob(a, mu, ls), want, rtol=1e-13)
    want_h = scipy.stats.norm(scale=np.exp(ls)).entropy().sum()
    assert abs(ppo.entropy(ls) - want_h) < 1e-13


def test_gradient_against_finite_differences():
    rng = np.random.default_rng(2)
    flat = _params(rng)
    batch = _batch(rng, flat)
    stats, g = ppo.loss_and_grad(flat, DIMS, *batch, exact=True)
    rho = np.exp(ppo.log_prob(batch[1], ppo.forward(ppo.unflatten(flat, DIMS), batch[0],
                                                     False, True)["mu"],
                              ppo.unflatten(flat, DIMS)["log_std"]) - batch[2])
    # both branches of the clip are exercised
    assert np.any(np.abs(rho - 1) > 0.25) and np.any(np.abs(rho - 1) < 0.25)
    h = 1e-6
    fd = np.empty_like(flat)
    for i in range(flat.shape[0]):
        e = np.zeros_like(flat)
        e[i] = h
        fd[i] = (ppo.loss(flat + e, DIMS, *batch, exact=True)
                 - ppo.loss(flat - e, DIMS, *batch, exact=True)) / (2 * h)
    np.testing.assert_allclose(g, fd, rtol=1e-6, atol=1e-8)


def test_clip_case_analysis():
    """A sample contributes to the actor gradient unless the clip is active
    on the side its advantage points to: rho > 1 + eps with A > 0, or
    rho < 1 - eps with A < 0."""
    rng = np.random.default_rng(3)
    flat = _params(rng)
    x, a, _, _, ret = _batch(rng, flat, B=4)
    p = ppo.unflatten(flat, DIMS)
    f = ppo.forward(p, x, False, True)
    lp = ppo.log_prob(a, f["mu"], p["log_std"])
    log_rho = np.log(np.array([1.5, 0.5, 1.5, 0.5]))     # rho on both sides, outside
    adv = np.array([1.0, -1.0, -1.0, 1.0])               # clipped, clipped, live, live
    _, g = ppo.loss_and_grad(flat, DIMS, x, a, lp - log_rho, adv, ret, exact=True)
    # the two live samples alone (scaled by 1/B with B = 4 either way)
    adv2 = np.array([0.0, 0.0, -1.0, 1.0])
    _, g2 = ppo.loss_and_grad(flat, DIMS, x, a, lp - log_rho, adv2, ret, exact=True)
    np.testing.assert_allclose(g, g2, rtol=1e-14, atol=1e-16)
    # and a live sample's gradient is not zero
    adv3 = np.array([0.0, 0.0, -1.0, 0.0])
    _, g3 = ppo.loss_and_grad(flat, DIMS, x, a, lp - log_rho, adv3, ret, exact=True)
    seg = ppo.unflatten(g3, DIMS)
    assert np.abs(seg["W3"]).max() > 1e-3


def test_closed_form_at_rho_one():
    """At the old policy (rho = 1), dL/dmu_ik = -(1/B) A_i (a_ik - mu_ik) /
    sigma_k^2, so g_b3 is its column sum, and the log_std gradient is
    -(1/B) sum_i A_i ((a - mu)^2 / sigma^2 - 1) - c_ent."""
    rng = np.random.default_rng(4)
    flat = _params(rng)
    x, a, _, adv, ret = _batch(rng, flat, B=6)
    p = ppo.unflatten(flat, DIMS)
    f = ppo.forward(p, x, False, True)
    lp = ppo.log_prob(a, f["mu"], p["log_std"])
    stats, g = ppo.loss_and_grad(flat, DIMS, x, a, lp, adv, ret, exact=True)
    seg = ppo.unflatten(g, DIMS)
    var = np.exp(2 * p["log_std"])
    d = a - f["mu"]
    np.testing.assert_allclose(seg["b3"], (-(adv[:, None]) * d / var).sum(0) / 6, rtol=1e-12)
    want_ls = (-(adv[:, None]) * (d * d / var - 1)).sum(0) / 6 - 0.02
    np.testing.assert_allclose(seg["log_std"], want_ls, rtol=1e-12)
    assert abs(stats[0] + adv.mean()) < 1e-14           # L_clip = -mean(A)
    assert stats[3] == 0.0                               # nothing clipped


def test_entropy_gradient_is_the_coefficient():
    """With zero advantages only the entropy bonus reaches log_std."""
    rng = np.random.default_rng(5)
    flat = _params(rng)
    x, a, lo, _, ret = _batch(rng, flat)
    _, g = ppo.loss_and_grad(flat, DIMS, x, a, lo, np.zeros(9), ret, ent_coef=0.02,
                             exact=True)
    seg = ppo.unflatten(g, DIMS)
    np.testing.assert_array_equal(seg["log_std"], np.full(3, -0.02))
    assert np.all(seg["W1"] == 0) and np.all(seg["b3"] == 0)


def test_critic_output_layer_closed_form():
    rng = np.random.default_rng(6)
    flat = _params(rng)
    x, a, lo, adv, ret = _batch(rng, flat)
    p = ppo.unflatten(flat, DIMS)
    f = ppo.forward(p, x, False, True)
    _, g = ppo.loss_and_grad(flat, DIMS, x, a, lo, adv, ret, exact=True)
    seg = ppo.unflatten(g, DIMS)
    r = f["v"] - ret
    assert abs(seg["bc3"][0] - 2 * r.sum() / 9) < 1e-14
    np.testing.assert_allclose(seg["wc3"], 2 * (r[:, None] * f["hc2"]).sum(0) / 9, rtol=1e-12)


def test_adam_against_torch():
    rng = np.random.default_rng(7)
    theta0 = rng.standard_normal(50)
    t = torch.tensor(theta0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([t], lr=2.0 ** -14, betas=(0.9, 0.999), eps=1e-8)
    theta, m, v = theta0.copy(), np.zeros(50), np.zeros(50)
    for step in range(1, 5):
        g = rng.standard_normal(50) * 10.0 ** rng.integers(-6, 2, 50)
        t.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        theta, m, v = ppo.adam(theta, m, v, g, step)
        np.testing.assert_allclose(theta, t.detach().numpy(), rtol=0, atol=1e-15)


def test_first_adam_step_moves_each_weight_by_lr():
    """Bias correction makes the first step lr * g / (|g| + eps)."""
    g = np.array([3.0, -1e-3, 0.5, -20.0])
    theta, _, _ = ppo.adam(np.zeros(4), np.zeros(4), np.zeros(4), g, 1)
    np.testing.assert_allclose(theta, -2.0 ** -14 * g / (np.abs(g) + 1e-8), rtol=1e-12)


def test_bf16_forward_rounds_like_the_actor_oracle():
    """The learner's forward in bf16 mode gives the actor oracle's mu."""
    import oracle
    rng = np.random.default_rng(8)
    dims = (31, 64, 64, 5, 64, 64)
    flat = _params(rng, dims, scale=0.2).astype(np.float32).astype(np.float64)
    p = ppo.unflatten(flat, dims)
    x = ppo.bf16_round(rng.standard_normal((5, 31)).astype(np.float32)).astype(np.float64)
    f = ppo.forward(p, x, bf16=True)
    W = [p["W1"][None].astype(np.float32), p["W2"][None].astype(np.float32),
         p["W3"][None].astype(np.float32)]
    b = [p["b1"][None].astype(np.float32), p["b2"][None].astype(np.float32),
         p["b3"][None].astype(np.float32)]
    act = oracle.actor(W, b, p["log_std"][None].astype(np.float32), dims[:4], True, 1)
    mu = oracle.mlp(act, 0, x.astype(np.float32))
    np.testing.assert_array_equal(f["mu"].astype(np.float32), mu)


def test_minibatch_rows_stay_in_the_agents_transitions():
    import oracle
    L, E, A = 13, 12, 3
    epa = E // A
    for agent in range(A):
        idx = oracle.minibatch_rows(99, 5, 4, 64, L, E, agent, epa)
        j, e = idx // E, idx % E
        assert np.all((0 <= j) & (j < L))
        assert np.all((agent * epa <= e) & (e < (agent + 1) * epa))


def test_minibatch_rows_are_uniform():
    """Chi-square over the R = L epa transitions of one agent."""
    import oracle
    L, E, A, agent = 10, 8, 2, 1
    epa = E // A
    idx = oracle.minibatch_rows(2021, 0, 200, 256, L, E, agent, epa).reshape(-1)
    cells = (idx // E) * epa + (idx % E - agent * epa)
    counts = np.bincount(cells, minlength=L * epa)
    chi2 = ((counts - counts.mean()) ** 2 / counts.mean()).sum()
    # 39 degrees of freedom: the 0.9999 quantile is about 80
    assert chi2 < 80
    assert scipy.stats.chi2.sf(chi2, L * epa - 1) > 1e-4


def test_minibatch_rows_differ_across_counters_and_agents():
    import oracle
    a = oracle.minibatch_rows(7, 0, 2, 128, 390, 64, 0, 16)
    b = oracle.minibatch_rows(7, 1, 1, 128, 390, 64, 0, 16)
    # update 1 of a call at counter 0 is update 0 of a call at counter 1
    np.testing.assert_array_equal(a[1], b[0])
    assert np.mean(a[0] == a[1]) < 0.05
    c = oracle.minibatch_rows(7, 0, 1, 128, 390, 64, 1, 16)
    assert np.mean((a[0] % 64) // 16 == 0) == 1.0 and np.mean((c[0] % 64) // 16 == 1) == 1.0
