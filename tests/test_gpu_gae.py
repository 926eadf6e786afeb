"""GPU parity of tp_gae against the oracle (seeded generator inputs), at
small and full sizes, ragged env counts, L = 1, episode ends inside the
rollout, the lambda = 0 / 1 special cases, and shapes on both sides of the
switch between the two GAE kernels."""

import numpy as np
import pytest
import torch

import oracle
from gpu_common import rel_check, say, TOL_GAE
from paper_2111_05188_amd import tp

pytestmark = pytest.mark.gpu


def _inputs(L, E, seed, p_done=0.02):
    rng = np.random.default_rng(seed)
    r = (rng.standard_normal((L, E)) * 0.3).astype(np.float32)
    v = rng.standard_normal((L + 1, E)).astype(np.float32)
    d = (rng.random((L, E)) < p_done).astype(np.uint8)
    return r, v, d


@pytest.mark.parametrize("L,E,gamma,lam", [
    (1, 1, 0.99, 0.95), (3, 5, 0.9, 0.5), (256, 64, 0.99, 0.95),
    (390, 100, 0.99, 0.95), (390, 4096, 0.99, 0.95), (2520, 1024, 0.99, 0.95),
    (17, 130, 0.99, 0.0), (45, 65, 0.97, 1.0), (1000, 3, 1.0, 1.0),
    # both sides of the boundaries between the kernels: rollouts of 512
    # steps (the longest chunks) and 513; 16,383 envs and 16,384 (and a
    # ragged count above it)
    (512, 1000, 0.99, 0.95), (513, 200, 0.99, 0.95), (64, 16383, 0.99, 0.95),
    (7, 16384, 0.99, 0.95), (512, 16400, 0.99, 0.95),
    # the four-envs-per-lane kernel (E a multiple of 4 from 16,384 envs,
    # rollouts up to 416 steps): full and ragged chunk counts, a ragged
    # last workgroup, one step, lambda 1, and both sides of its length limit
    (390, 16384, 0.99, 0.95), (416, 16388, 0.99, 0.95), (417, 16384, 0.99, 0.95),
    (33, 20000, 0.97, 0.9), (1, 16388, 0.99, 0.95), (390, 32772, 0.99, 1.0),
    (390, 16386, 0.99, 0.95)])
def test_gae_parity(L, E, gamma, lam):
    say(f"[gae] L={L} E={E} gamma={gamma} lambda={lam}")
    r, v, d = _inputs(L, E, L * 7 + E)
    dev = "cuda"
    gr, gv, gd = (torch.from_numpy(x).to(dev) for x in (r, v, d))
    adv = torch.empty(L, E, device=dev)
    ret = torch.empty(L, E, device=dev)
    tp.gae(gr, gv, gd, gamma, lam, adv, ret)
    torch.cuda.synchronize()
    a_o, r_o = oracle.gae(r, v, d, gamma, lam)
    rel_check("adv", adv.cpu().numpy(), a_o, TOL_GAE)
    rel_check("ret", ret.cpu().numpy(), r_o, TOL_GAE)


def test_gae_stress_shape_sampled():
    """Full stress size (L=390, E=65536): GPU vs oracle on every column (the
    name is historical) -- the oracle's scan takes well under a second."""
    L, E = 390, 65536
    say(f"[gae] stress L={L} E={E}")
    r, v, d = _inputs(L, E, 5)
    dev = "cuda"
    gr, gv, gd = (torch.from_numpy(x).to(dev) for x in (r, v, d))
    adv = torch.empty(L, E, device=dev)
    ret = torch.empty(L, E, device=dev)
    tp.gae(gr, gv, gd, 0.99, 0.95, adv, ret)
    torch.cuda.synchronize()
    a_o, r_o = oracle.gae(r, v, d, 0.99, 0.95)
    rel_check("adv", adv.cpu().numpy(), a_o, TOL_GAE)
    rel_check("ret", ret.cpu().numpy(), r_o, TOL_GAE)


def test_gae_deterministic():
    r, v, d = _inputs(390, 777, 3)
    dev = "cuda"
    gr, gv, gd = (torch.from_numpy(x).to(dev) for x in (r, v, d))
    outs = []
    for _ in range(2):
        adv = torch.empty(390, 777, device=dev)
        ret = torch.empty(390, 777, device=dev)
        tp.gae(gr, gv, gd, 0.99, 0.95, adv, ret)
        outs.append((adv.cpu(), ret.cpu()))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
