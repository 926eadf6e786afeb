"""GPU parity of tp_rollout (fused actor + sampling + env step + trajectory
store) against a teacher-forced oracle replay, at sizes the oracle finishes
in seconds: several workgroups of envs, ragged tails, every actor shape
family (fp32 VALU, bf16 MFMA 256- to 1024-wide on the role-split kernel,
bf16 of another shape on the generic kernel, multi-agent), plus
determinism, split/resume, and envs whose start row leaves no room."""

import numpy as np
import pytest
import torch

import workloads as W
from gpu_common import (bits16, build_problem, compare_rollout, oracle_replay,
                        rel_check, say)
from paper_2111_05188_amd import tp

pytestmark = pytest.mark.gpu

SEED = 0x5EED0FF12C


def _run_case(cfg, E, L, rows=None, n_agents=1, cmp_ids=None, step0=0):
    rows = cfg.T1 if rows is None else rows
    c = cfg.with_(N=rows - 1, E=E, n_agents=n_agents)
    mk = W.make_market(c)
    t0 = W.make_t0(c)
    pb, params = build_problem(c, mk, t0)
    pb.reset()
    say(f"[rollout] {cfg.name} E={E} L={L} agents={n_agents} rows={rows}")
    pb.rollout(SEED, step0, L)
    torch.cuda.synchronize()
    ids = np.arange(E) if cmp_ids is None else np.asarray(cmp_ids)
    teacher = pb.traj.action[:L].index_select(
        1, torch.as_tensor(ids, device="cuda")).cpu().numpy()
    out = oracle_replay(c, mk, params, t0[ids], ids, SEED, L, teacher,
                        c.envs_per_agent, step0=step0)
    compare_rollout(c, pb, out, ids, L)
    cash, sh, t = out["final"]
    ids_t = torch.as_tensor(ids, device="cuda")
    assert np.array_equal(pb.state.cash.index_select(0, ids_t).cpu().numpy(), cash)
    assert np.array_equal(pb.state.shares.index_select(0, ids_t).cpu().numpy(), sh)
    assert np.array_equal(pb.state.t.index_select(0, ids_t).cpu().numpy(), t)
    ol = pb.traj.obs_last.index_select(0, ids_t)[:, :c.K_pad]
    g = bits16(ol) if c.dtype == "bf16" else ol.cpu().numpy()
    assert np.array_equal(g, out["obs_last"])
    return pb


def test_tiny_full():
    _run_case(W.get_config("tiny"), 64, 256)


def test_tiny_ragged_env_count():
    _run_case(W.get_config("tiny"), 7, 50)


def test_nasdaq_shape_small_market_ragged():
    # full n, I and 1001-512-512-100 bf16 actor; 3 workgroups, ragged tail
    _run_case(W.get_config("nasdaq100"), 37, 60, rows=40 * 390 + 1)


def test_ensemble_shape_three_agents_ragged():
    _run_case(W.get_config("ensemble"), 60, 40, rows=20 * 390 + 1, n_agents=3)


@pytest.mark.parametrize("L", [1, 2, 4, 5])
def test_nasdaq_shape_short_rollouts(L):
    """Rollouts shorter than, or not a multiple of, the role-split kernel's
    market batch of three steps: the partial final batch, the bootstrap
    observation row and the final state."""
    _run_case(W.get_config("nasdaq100"), 20, L, rows=6 * 390 + 1)


def test_stress_shape_small():
    _run_case(W.get_config("stress"), 20, 30, rows=20 * 390 + 1)


@pytest.mark.parametrize("I,H,L", [(4, 512, 50), (4, 256, 4), (4, 768, 5), (4, 1024, 3),
                                   (10, 512, 50), (10, 256, 4), (10, 768, 5), (10, 1024, 3)])
def test_role_split_other_markets(I, H, L):
    """The role-split kernel on the 100-stock markets with 4 and 10
    indicators per stock (601 and 1201 inputs: 20 and 40 k-steps, observation
    rows of 608 and 1,216 columns), at every width, three workgroups with a
    ragged tail, rollouts that end inside a market batch."""
    cfg = W.get_config("nasdaq100").with_(n_ind=I, hidden=(H, H))
    pb = _run_case(cfg, 37, L, rows=20 * 390 + 1)
    assert tp.rollout_path(pb.mkt, pb.actor) == 1


@pytest.mark.parametrize("I,H,agents,E", [(10, 768, 3, 60), (4, 512, 2, 34), (10, 512, 1, 1),
                                          (10, 1024, 1, 17)])
def test_role_split_agents_and_env_counts(I, H, agents, E):
    """Several agents per launch (each agent's blocks in its own run of
    workgroups, ragged per agent), a single env, and one env past a
    workgroup, on the market-batch and single-step paths."""
    cfg = W.get_config("nasdaq100").with_(n_ind=I, hidden=(H, H))
    pb = _run_case(cfg, E, 20, rows=20 * 390 + 1, n_agents=agents)
    assert tp.rollout_path(pb.mkt, pb.actor) == 1


@pytest.mark.parametrize("H,L", [(256, 50), (256, 4), (768, 50), (768, 3)])
def test_role_split_other_widths(H, L):
    """The role-split kernel at its other hidden widths (256: market batches
    of three steps; 768: of two), three workgroups with a ragged tail, and
    rollouts that end inside a batch."""
    pb = _run_case(W.get_config("nasdaq100").with_(hidden=(H, H)), 37, L, rows=20 * 390 + 1)
    assert tp.rollout_path(pb.mkt, pb.actor) == 1


def test_dow_shape_small():
    _run_case(W.get_config("dow30"), 9, 300, rows=2521)


def test_bf16_actor_of_another_shape():
    # a bf16 actor outside the shapes with a specialised kernel (301 inputs,
    # 256-wide layers) runs the generic MFMA rollout kernel
    _run_case(W.get_config("dow30").with_(dtype="bf16"), 21, 120, rows=2521)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_largest_market(dtype):
    # 128 stocks x 8 indicators (n * n_ind = 1024, the largest market the
    # boundary takes; 1281 inputs) on the generic kernel, fp32 and bf16
    cfg = W.get_config("tiny").with_(n=128, n_ind=8, dtype=dtype, hidden=(128, 128))
    pb = _run_case(cfg, 20, 40)
    assert tp.rollout_path(pb.mkt, pb.actor) == 0


def test_bf16_100_stock_actor_outside_the_role_split_shapes():
    # unequal hidden widths (512-256) on the 100 x 8 market: the generic
    # MFMA kernel takes it, with the same results contract
    cfg = W.get_config("nasdaq100").with_(hidden=(512, 256))
    pb = _run_case(cfg, 21, 30, rows=20 * 390 + 1)
    assert tp.rollout_path(pb.mkt, pb.actor) == 0


def test_deterministic_and_resumable():
    """Two identical runs are bitwise equal; rollout(L) equals rollout(j)
    followed by rollout(L-j, step0=j) from the saved state."""
    cfg = W.get_config("nasdaq100").with_(N=20 * 390, E=40)
    mk = W.make_market(cfg)
    t0 = W.make_t0(cfg)
    L, j = 40, 15
    runs = []
    for _ in range(2):
        pb, _ = build_problem(cfg, mk, t0)
        pb.reset()
        say("[rollout] determinism run")
        pb.rollout(SEED, 0, L)
        torch.cuda.synchronize()
        runs.append(pb)
    a, b = runs
    # only the first L rows were written (the store holds a full episode)
    for name in ("action", "logp", "reward", "done", "cash_tap", "shares_tap", "obs"):
        assert torch.equal(getattr(a.traj, name)[:L], getattr(b.traj, name)[:L]), name
    # split run
    pb, _ = build_problem(cfg, mk, t0)
    pb.reset()
    t1 = tp.TrajT.alloc(j, cfg.E, cfg.n, cfg.K_pad, torch.bfloat16, taps=True, obs_last=True)
    t2 = tp.TrajT.alloc(L - j, cfg.E, cfg.n, cfg.K_pad, torch.bfloat16, taps=True, obs_last=True)
    say("[rollout] split run")
    pb.rollout(SEED, 0, j, traj=t1)
    pb.rollout(SEED, j, L - j, traj=t2)
    torch.cuda.synchronize()
    for name in ("action", "logp", "reward", "done", "cash_tap", "shares_tap", "obs"):
        full = getattr(a.traj, name)[:L]
        assert torch.equal(full[:j], getattr(t1, name)), name
        assert torch.equal(full[j:], getattr(t2, name)), name
    assert torch.equal(t1.obs_last, a.traj.obs[j])
    assert torch.equal(t2.obs_last, a.traj.obs_last)
    for s in ("cash", "shares", "t"):
        assert torch.equal(getattr(pb.state, s), getattr(a.state, s)), s


def test_env_without_room_is_not_stepped():
    cfg = W.get_config("tiny")
    mk = W.make_market(cfg)
    t0 = np.zeros(20, np.int64)
    pb, _ = build_problem(cfg.with_(E=20), mk, t0, E=20, envs_per_agent=20)
    pb.state = tp.StateT.empty(20, cfg.n, count_invalid=True)
    pb.reset()
    assert pb.state.n_invalid.item() == 0
    # env 3 starts too late for L steps; env 4 has an invalid (negative) row
    pb.state.t[3] = cfg.T1 - 10
    pb.state.t[4] = -1
    say("[rollout] envs without room")
    pb.rollout(SEED, 0, 50)
    torch.cuda.synchronize()
    r = pb.traj.reward[:50].cpu().numpy()
    assert np.isnan(r[:, 3]).all() and np.isnan(r[:, 4]).all()
    assert np.isfinite(r[:, [0, 1, 2, 5]]).all()
    assert (pb.traj.done[:50].cpu().numpy()[:, 3] == 0).all()
    assert np.isnan(pb.traj.action[:50, 3].cpu().numpy()).all()
    assert np.isnan(pb.traj.mu_tap[:50, [3, 4]].cpu().numpy()).all()
    assert np.isfinite(pb.traj.mu_tap[:50, [0, 1, 2, 5]].cpu().numpy()).all()
    assert pb.state.t[3].item() == cfg.T1 - 10 and pb.state.t[4].item() == -1
    assert pb.state.t[0].item() == 50
    assert pb.state.n_invalid.item() == 2
    # the host check names the first env without room
    with pytest.raises(tp.TPError) as ei:
        tp.check_starts(pb.state.t.cpu().numpy(), cfg.T1, 50)
    assert ei.value.code == tp.TP_ERANGE and "env 3" in str(ei.value)


def test_env_without_room_role_split_kernel():
    """The same on the role-split kernel (100-stock bf16 actor): an env
    whose start row leaves no room is counted, its rows are NaN, and the
    envs sharing its waves are stepped as usual."""
    cfg = W.get_config("nasdaq100").with_(N=4 * 390, E=20)
    mk = W.make_market(cfg)
    t0 = W.make_t0(cfg)
    pb, params = build_problem(cfg, mk, t0)
    assert tp.rollout_path(pb.mkt, pb.actor) == 1
    pb.state = tp.StateT.empty(20, cfg.n, count_invalid=True)
    pb.reset()
    pb.state.t[6] = cfg.T1 - 5
    pb.state.t[9] = -7
    say("[rollout] role-split kernel, envs without room")
    pb.rollout(SEED, 0, 30)
    torch.cuda.synchronize()
    assert pb.state.n_invalid.item() == 2
    r = pb.traj.reward[:30].cpu().numpy()
    assert np.isnan(r[:, [6, 9]]).all() and np.isfinite(np.delete(r, [6, 9], axis=1)).all()
    assert np.isnan(pb.traj.mu_tap[:30, [6, 9]].cpu().numpy()).all()
    ids = np.array([0, 7, 8, 19])
    teacher = pb.traj.action[:30].index_select(1, torch.as_tensor(ids, device="cuda")).cpu().numpy()
    out = oracle_replay(cfg, mk, params, t0[ids], ids, SEED, 30, teacher, cfg.envs_per_agent)
    compare_rollout(cfg, pb, out, ids, 30)


def test_rollout_errors():
    cfg = W.get_config("tiny")
    mk = W.make_market(cfg)
    pb, _ = build_problem(cfg, mk, W.make_t0(cfg))
    with pytest.raises(tp.TPError) as ei:
        pb.rollout(SEED, 200, 100)          # beyond the horizon
    assert ei.value.code == tp.TP_ERANGE
    other = tp.TrajT.alloc(10, cfg.E, cfg.n, cfg.K_pad, torch.float32)
    bad = tp.TrajT(other.action, other.logp, other.reward, other.done,
                   other.obs, 33)           # ld_obs not a multiple of 8
    with pytest.raises(tp.TPError) as ei:
        pb.rollout(SEED, 0, 10, traj=bad)
    assert ei.value.code == tp.TP_EINVAL and "ld_obs" in str(ei.value)
