"""GPU parity of tp_critic_value (the PPO critic's forward pass over a
trajectory's observations) against the oracle's MLP: the bf16 MFMA kernel at
512- and 1024-wide layers (one agent and several agents, ragged row blocks),
the generic kernel (fp32 and another bf16 shape), the full 100-stock minute
trajectory shape on sampled rows, and determinism.

Observation blocks [T][E][K_pad] come from the seeded generator
(workloads.make_learner_data: the observation's structure and scales, zero
padding), rounded to bf16 on the CPU for bf16 critics; both sides read the
same values."""

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_common import TOL_MLP, rel_check, say
from paper_2111_05188_amd import tp

pytestmark = pytest.mark.gpu


def _oracle_critic(cfg, params, A):
    """The critic as an oracle MLP with one output (log_std unused)."""
    Wc, bc = params
    S, H1, H2, _ = cfg.dims
    Wo = [Wc[0], Wc[1], Wc[2].reshape(A, 1, H2)]
    bo = [bc[0], bc[1], bc[2].reshape(A, 1)]
    return oracle.actor(Wo, bo, np.zeros((A, 1), np.float32), (S, H1, H2, 1),
                        cfg.dtype == "bf16", cfg.E // A)


POOL = 65536


def _obs_block(c, T, E, seed):
    """[T][E][K_pad] observation rows of the critic's dtype on the device,
    row r = t E + e holding generated row r mod POOL, and the host values
    of the generated rows (what the oracle reads)."""
    n = min(T * E, POOL)
    obs, *_ = W.make_learner_data(c, n, seed=seed)
    base = torch.from_numpy(obs)
    if c.dtype == "bf16":
        base = base.to(torch.bfloat16)
    host = base.float().numpy()
    dev = base.cuda()
    sel = torch.arange(T * E, device="cuda") % n
    return dev.index_select(0, sel).reshape(T, E, c.K_pad), host


def _run(cfg, E, L, n_agents=1, sample=None):
    c = cfg.with_(E=E, n_agents=n_agents, L=L)
    T1 = L + 1
    obs_all, host = _obs_block(c, T1, E, seed=E * 7 + L)
    cp = W.make_critic(c)
    dt = tp.TP_BF16 if c.dtype == "bf16" else tp.TP_F32
    crit = tp.CriticT([torch.from_numpy(w).cuda() for w in cp[0]],
                      [torch.from_numpy(x).cuda() for x in cp[1]], c.dims[:3], dt,
                      E // n_agents)
    crit.pack()
    values = torch.empty(T1, E, dtype=torch.float32, device="cuda")
    say(f"[critic] {cfg.name} E={E} T={T1} agents={n_agents}")
    tp.critic_value(crit, obs_all, values)
    torch.cuda.synchronize()
    v = values.cpu().numpy()                          # [L+1][E]
    act = _oracle_critic(c, cp, n_agents)
    epa = E // n_agents
    if sample is None:
        rows_ = [(t, e) for t in range(T1) for e in range(E)]
    else:
        rng = np.random.default_rng(5)
        rows_ = [(int(rng.integers(T1)), int(rng.integers(E))) for _ in range(sample)]
    got, want = [], []
    for a in range(n_agents):
        sel = [(t, e) for (t, e) in rows_ if e // epa == a]
        if not sel:
            continue
        x = host[[(t * E + e) % host.shape[0] for t, e in sel], :c.S]
        want.append(oracle.mlp(act, a, x)[:, 0])
        got.append(np.array([v[t, e] for t, e in sel]))
    got, want = np.concatenate(got), np.concatenate(want)
    rel_check(f"critic {cfg.name}", got, want, TOL_MLP[c.dtype])
    return crit, obs_all, values


def test_critic_mfma_512_ragged():
    # 1001-512-512-1 bf16: 300 envs = two 128-row blocks and a ragged 44
    _run(W.get_config("nasdaq100"), 300, 6)


def test_critic_mfma_1024():
    _run(W.get_config("stress"), 70, 4)


def test_critic_mfma_three_agents():
    # agent blocks of 45 envs: every block of rows stays inside one agent
    _run(W.get_config("ensemble"), 135, 5, n_agents=3)


def test_critic_generic_fp32():
    _run(W.get_config("tiny"), 40, 30)
    _run(W.get_config("dow30"), 33, 20)


def test_critic_generic_bf16_other_shape():
    _run(W.get_config("dow30").with_(dtype="bf16"), 33, 20)


def test_critic_full_nasdaq_trajectory_sampled():
    cfg = W.get_config("nasdaq100")
    crit, obs_all, values = _run(cfg, cfg.E, cfg.L, sample=256)
    # determinism: a second call gives the same bits
    v0 = values.clone()
    tp.critic_value(crit, obs_all, values)
    torch.cuda.synchronize()
    assert torch.equal(v0, values)
