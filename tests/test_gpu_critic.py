"""GPU parity of tp_critic_value (the PPO critic's forward pass over a
trajectory's observations) against the oracle's MLP, on observation rows a
rollout writes: the bf16 MFMA kernel at 512- and 1024-wide layers (one agent
and several agents, ragged row blocks), the generic kernel (fp32 and another
bf16 shape), the full 100-stock minute trajectory on sampled rows, and
determinism."""

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_common import TOL_MLP, build_problem, rel_check, say

pytestmark = pytest.mark.gpu

SEED = 0x5EED0FF12C


def _oracle_critic(cfg, params, A):
    """The critic as an oracle MLP with one output (log_std unused)."""
    Wc, bc = params
    S, H1, H2, _ = cfg.dims
    Wo = [Wc[0], Wc[1], Wc[2].reshape(A, 1, H2)]
    bo = [bc[0], bc[1], bc[2].reshape(A, 1)]
    return oracle.actor(Wo, bo, np.zeros((A, 1), np.float32), (S, H1, H2, 1),
                        cfg.dtype == "bf16", cfg.E // A)


def _obs_f32(obs):
    return obs.float().cpu().numpy()


def _run(cfg, E, L, rows, n_agents=1, sample=None):
    # episode length L, so that the bootstrap row obs_L is row L of the block
    c = cfg.with_(N=rows - 1, E=E, n_agents=n_agents, L=L)
    mk = W.make_market(c)
    t0 = W.make_t0(c)
    pb, _ = build_problem(c, mk, t0, taps=False)
    pb.reset()
    pb.rollout(SEED, 0, L)
    cp = W.make_critic(c)
    pb.set_critic(cp)
    say(f"[critic] {cfg.name} E={E} L={L} agents={n_agents} mfma={pb.critic.s.dims[:]}")
    pb.critic_values()
    torch.cuda.synchronize()
    v = pb.values.cpu().numpy()                       # [L+1][E]
    obs = pb.traj.obs_all[:, :, :c.S]                 # [L+1][E][S]
    act = _oracle_critic(c, cp, n_agents)
    epa = E // n_agents
    T1 = L + 1
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
        ts = torch.as_tensor([t for t, _ in sel], device="cuda")
        es = torch.as_tensor([e for _, e in sel], device="cuda")
        x = _obs_f32(obs[ts, es])
        want.append(oracle.mlp(act, a, x)[:, 0])
        got.append(np.array([v[t, e] for t, e in sel]))
    got, want = np.concatenate(got), np.concatenate(want)
    # rows of envs that were not stepped hold no observation: skip them
    ok = np.isfinite(want)
    rel_check(f"critic {cfg.name}", got[ok], want[ok], TOL_MLP[c.dtype])
    return pb


def test_critic_mfma_512_ragged():
    # 1001-512-512-1 bf16: 300 envs = two 128-row blocks and a ragged 44
    _run(W.get_config("nasdaq100"), 300, 6, 20 * 390 + 1)


def test_critic_mfma_1024():
    _run(W.get_config("stress"), 70, 4, 20 * 390 + 1)


def test_critic_mfma_three_agents():
    # agent blocks of 45 envs: every block of rows stays inside one agent
    _run(W.get_config("ensemble"), 135, 5, 20 * 390 + 1, n_agents=3)


def test_critic_generic_fp32():
    _run(W.get_config("tiny"), 40, 30, 257)
    _run(W.get_config("dow30"), 33, 20, 2521)


def test_critic_generic_bf16_other_shape():
    _run(W.get_config("dow30").with_(dtype="bf16"), 33, 20, 2521)


def test_critic_full_nasdaq_trajectory_sampled():
    cfg = W.get_config("nasdaq100")
    pb = _run(cfg, cfg.E, cfg.L, cfg.T1, sample=256)
    # determinism: a second call gives the same bits
    v0 = pb.values.clone()
    pb.critic_values()
    torch.cuda.synchronize()
    assert torch.equal(v0, pb.values)
