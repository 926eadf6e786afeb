"""GPU parity of tp_ppo_update (PPO, Section 5.2; Table 2) against the
oracle's learner: the gradient of one update segment by segment, the loss
statistics, the parameters after one and after several Adam steps, and
determinism, for the fp32 tiny and DOW-30 shapes and the bf16
1001-512-512-100 shape at the paper's batch of 2^10.

Inputs are seeded and synthetic (workloads.make_learner_data); the stored
log-probabilities are the oracle's log-density of the stored action under
the starting parameters, shifted by log-ratio offsets that keep every row
clearly inside or clearly outside the clip (so both sides take the same
branch).  Tolerances: every gradient element is held to 1e-4 (fp32: the
tanh and summation order differ) or 2e-2 (bf16: operands rounded to bf16
as the kernels do) of max(|g|, RMS of its segment); parameters by the Adam
step they moved, in units of the learning rate.

Several updates in a row are compared as two independent chains.  At the
paper's learning rate one Adam step moves every weight by about lr, which
moves log rho by up to about 1, so after the first update some rows cross
the clip edge; a row whose ratio lands within rounding of the edge takes
different branches on the two sides and the chains separate (measured: 4
such rows after one bf16 update, 16 after two).  The bf16 multi-update test
therefore runs at lr = 2^-22, where ratios move by ~0.005 and stay clear
of the edges; the fp32 one keeps 2^-14."""

import numpy as np
import pytest
import torch

import workloads as W
from gpu_common import say
from oracle import ppo
from paper_2111_05188_amd import tp

pytestmark = pytest.mark.gpu

GRAD_TOL = {"f32": 1e-4, "bf16": 2e-2}


def _dims(cfg):
    S, H1, H2, n = cfg.dims
    return (S, H1, H2, n, H1, H2)


def _setup(cfg, rows, B, lr=2.0 ** -14):
    dims = _dims(cfg)
    bf = cfg.dtype == "bf16"
    flat = W.make_flat_params(cfg)
    obs, action, adv, ret, which = W.make_learner_data(cfg, rows)
    # observation values as the kernels see them (bf16 rows for bf16 configs)
    obs_t = torch.from_numpy(obs)
    if bf:
        obs_t = obs_t.to(torch.bfloat16)
    obs_vals = obs_t.float().numpy()
    p = ppo.unflatten(flat.astype(np.float64), dims)
    f = ppo.forward(p, obs_vals[:, :dims[0]], bf16=bf)
    lp = ppo.log_prob(action, f["mu"], p["log_std"])
    logp = (lp - np.asarray(W.LOG_RATIO_OFFSETS)[which]).astype(np.float32)
    host = dict(flat=flat, obs=obs_vals, action=action, logp=logp, adv=adv, ret=ret)
    dev = dict(obs=obs_t.cuda(), action=torch.from_numpy(action).cuda(),
               logp=torch.from_numpy(logp).cuda(), adv=torch.from_numpy(adv).cuda(),
               ret=torch.from_numpy(ret).cuda())
    c = tp.ppo_cfg(dims, tp.TP_BF16 if bf else tp.TP_F32, B, lr=lr)
    return dims, bf, c, host, dev


def _oracle_batch(host, idx, S):
    return ppo.gather(host["obs"], host["action"], host["logp"], host["adv"], host["ret"],
                      idx, S)


def _rel(a, b):
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))


def _check_grad(dims, g_gpu, g_orc, tol, what):
    """Every gradient element within tol * max(|g|, RMS of its segment)
    (the relative tolerance read per compared tensor); the per-segment
    relative L2 error is printed beside it as a diagnostic."""
    seg_g, seg_o = ppo.unflatten(g_gpu.astype(np.float64), dims), ppo.unflatten(g_orc, dims)
    worst = worst_l2 = 0.0
    for name, _ in ppo.layout(*dims):
        g, o = np.asarray(seg_g[name]).ravel(), np.asarray(seg_o[name]).ravel()
        scale = np.maximum(np.abs(o), max(np.sqrt(np.mean(o * o)), 1e-30))
        ratio = np.abs(g - o) / scale
        k = int(np.argmax(ratio))
        e = float(ratio[k])
        worst = max(worst, e)
        worst_l2 = max(worst_l2, _rel(g, o))
        assert e <= tol, (f"{what}: gradient of {name}: {(ratio > tol).sum()} of {ratio.size} "
                          f"elements outside {tol}; worst {e:.3g} at {k} (gpu {g[k]:.6g}, "
                          f"oracle {o[k]:.6g})")
    say(f"[ppo] {what}: worst element error {worst:.3g} (tol {tol:g}); "
        f"worst segment L2 error {worst_l2:.3g}")


def _run(cfg, rows, B, n_updates, seed=7, lr=2.0 ** -14):
    dims, bf, c, host, dev = _setup(cfg, rows, B, lr)
    P = tp.ppo_param_count(c)
    assert P == ppo.param_count(*dims) == host["flat"].shape[0]
    rng = np.random.default_rng(seed)
    idx = np.stack([rng.choice(rows, B, replace=False) for _ in range(n_updates)])
    params = torch.from_numpy(host["flat"].copy()).cuda()
    m = torch.zeros(P, device="cuda")
    v = torch.zeros(P, device="cuda")
    grad = torch.empty(P, device="cuda")
    stats = torch.empty(n_updates, 4, dtype=torch.float64, device="cuda")
    ws = tp.ppo_workspace(c)
    say(f"[ppo] {cfg.name} dtype={cfg.dtype} P={P} rows={rows} B={B} updates={n_updates}")
    tp.ppo_update(c, params, m, v, 1, dev["obs"], dev["action"], dev["logp"], dev["adv"],
                  dev["ret"], torch.from_numpy(idx).cuda(), ws, grad=grad, stats=stats)
    torch.cuda.synchronize()
    # the oracle, update by update from the same start
    theta, mo, vo = host["flat"].astype(np.float64), np.zeros(P), np.zeros(P)
    st_o, g_o = [], None
    for u in range(n_updates):
        batch = _oracle_batch(host, idx[u], dims[0])
        th32, mo, vo, st, g_o = ppo.update(theta, mo, vo, u + 1, dims, batch, lr=lr, bf16=bf)
        theta = th32.astype(np.float64)
        st_o.append(st)
    return dict(dims=dims, bf=bf, c=c, lr=lr, host=host, dev=dev, idx=idx, params=params, m=m, v=v,
                grad=grad.cpu().numpy(), stats=stats.cpu().numpy(), theta_o=theta,
                g_o=g_o, stats_o=np.array(st_o), ws=ws)


CASES = [("tiny", 512, 64), ("dow30", 1024, 256), ("nasdaq100", 4096, 1024)]


@pytest.mark.parametrize("name,rows,B", CASES)
def test_gradient_and_stats_of_one_update(name, rows, B):
    cfg = W.get_config(name)
    r = _run(cfg, rows, B, 1)
    _check_grad(r["dims"], r["grad"], r["g_o"], GRAD_TOL[cfg.dtype], name)
    st, so = r["stats"][0], r["stats_o"][0]
    rt = 1e-5 if cfg.dtype == "f32" else 2e-3
    np.testing.assert_allclose(st[:3], so[:3], rtol=rt, atol=1e-6)
    assert st[3] == so[3]                    # the same rows are clipped
    assert 0.2 < st[3] < 0.6                 # both branches present


def _check_params(r, n_updates, frac_tol):
    lr = r["lr"]
    got = r["params"].cpu().numpy().astype(np.float64)
    start = r["host"]["flat"].astype(np.float64)
    want = r["theta_o"]
    step_g, step_o = (got - start) / lr, (want - start) / lr
    # no weight moves further than the oracle's furthest (Adam's step is
    # bounded by lr (1 - b1) / sqrt(1 - b2) per update, Kingma and Ba 2.1)
    assert np.abs(step_g).max() <= np.abs(step_o).max() * 1.001 + 1e-3
    assert np.abs(step_o).max() <= n_updates * 0.1 / np.sqrt(0.001) + 1e-6
    off = np.abs(step_g - step_o)
    tol = 0.05 if r["bf"] else 2e-3
    frac = float(np.mean(off > tol))
    say(f"[ppo] params: {frac:.4%} of weights differ by more than {tol} lr")
    assert frac < frac_tol


@pytest.mark.parametrize("name,rows,B", CASES)
def test_parameters_after_one_update(name, rows, B):
    r = _run(W.get_config(name), rows, B, 1)
    # the first step is lr g / (|g| + eps): only weights with a near-zero
    # gradient (sign decided by rounding) may move differently
    _check_params(r, 1, 0.02 if r["bf"] else 0.002)


@pytest.mark.parametrize("name,rows,B,lr", [("tiny", 512, 64, 2.0 ** -14),
                                            ("nasdaq100", 4096, 1024, 2.0 ** -22)])
def test_three_updates_and_determinism(name, rows, B, lr):
    cfg = W.get_config(name)
    r = _run(cfg, rows, B, 3, lr=lr)
    _check_params(r, 3, 0.03 if r["bf"] else 0.003)
    rt = 1e-5 if cfg.dtype == "f32" else 2e-3
    np.testing.assert_allclose(r["stats"][:, :3], r["stats_o"][:, :3], rtol=rt, atol=1e-6)
    # the same call from the same start gives the same bits
    P = r["params"].numel()
    p2 = torch.from_numpy(r["host"]["flat"].copy()).cuda()
    m2, v2 = torch.zeros(P, device="cuda"), torch.zeros(P, device="cuda")
    d = r["dev"]
    tp.ppo_update(r["c"], p2, m2, v2, 1, d["obs"], d["action"], d["logp"], d["adv"], d["ret"],
                  torch.from_numpy(r["idx"]).cuda(), r["ws"])
    torch.cuda.synchronize()
    assert torch.equal(p2, r["params"]) and torch.equal(m2, r["m"]) and torch.equal(v2, r["v"])


def test_minimal_batch_and_rollout_rows():
    """B = 32 (one k-step of the batch products) on rows of a real
    trajectory layout: obs with a wider stride than K_pad."""
    cfg = W.get_config("tiny")
    dims, bf, c, host, dev = _setup(cfg, 100, 32)
    wide = torch.zeros(100, cfg.K_pad + 8, device="cuda")
    wide[:, :cfg.K_pad] = dev["obs"]
    P = tp.ppo_param_count(c)
    params = torch.from_numpy(host["flat"].copy()).cuda()
    m, v = torch.zeros(P, device="cuda"), torch.zeros(P, device="cuda")
    grad = torch.empty(P, device="cuda")
    idx = np.random.default_rng(3).choice(100, 32, replace=False)[None]
    tp.ppo_update(c, params, m, v, 1, wide, dev["action"], dev["logp"], dev["adv"], dev["ret"],
                  torch.from_numpy(idx).cuda(), tp.ppo_workspace(c), grad=grad)
    torch.cuda.synchronize()
    _, g_o = ppo.loss_and_grad(host["flat"].astype(np.float64), dims,
                               *_oracle_batch(host, idx[0], dims[0]))
    _check_grad(dims, grad.cpu().numpy(), g_o, GRAD_TOL["f32"], "tiny B=32")


@pytest.mark.parametrize("name,rows,B,A", [("tiny", 512, 64, 3), ("nasdaq100", 4096, 1024, 3),
                                            ("nasdaq100", 4096, 1024, 8),
                                            ("nasdaq100", 4096, 1024, 11)])
def test_agents_in_one_call_equal_single_calls(name, rows, B, A):
    """tp_ppo_update_agents: A agents with their own parameters, moments
    and minibatches, laid out with a stride wider than P, give bit for bit
    what A tp_ppo_update calls give (two updates, so the second reads
    moments the first wrote); the padding between agents is left alone.
    With eight or eleven 1001-512-512-100 agents the launches with at
    least 512 tiles' worth of 128 x 128 run the 256 x 128 product kernel,
    which keeps the k order of the 64 x 64 one, so the bits still agree;
    eleven agents leave padding slots in its XCD-aware dealing."""
    cfg = W.get_config(name)
    dims, bf, c, host, dev = _setup(cfg, rows, B)
    P = tp.ppo_param_count(c)
    U, stride = 2, P + 7
    rng = np.random.default_rng(21)
    idx = np.stack([np.stack([rng.choice(rows, B, replace=False) for _ in range(U)])
                    for _ in range(A)])
    start = np.stack([W.make_flat_params(cfg, agent=a) for a in range(A)])
    say(f"[ppo-agents] {name} A={A} U={U} P={P} stride={stride} B={B}")
    prm = torch.full((A, stride), 7.0, device="cuda")
    prm[:, :P] = torch.from_numpy(start).cuda()
    m = torch.full((A, stride), 5.0, device="cuda")
    v = torch.full((A, stride), 3.0, device="cuda")
    m[:, :P] = 0.0
    v[:, :P] = 0.0
    grad = torch.empty(A, P, device="cuda")
    stats = torch.empty(A, U, 4, dtype=torch.float64, device="cuda")
    tp.ppo_update_agents(c, prm, m, v, 1, dev["obs"], dev["action"], dev["logp"], dev["adv"],
                         dev["ret"], torch.from_numpy(idx).cuda(), tp.ppo_workspace(c, n_agents=A),
                         grad=grad, stats=stats)
    torch.cuda.synchronize()
    assert (prm[:, P:] == 7.0).all() and (m[:, P:] == 5.0).all() and (v[:, P:] == 3.0).all()
    ws = tp.ppo_workspace(c)
    for a in range(A):
        p1 = torch.from_numpy(start[a].copy()).cuda()
        m1, v1 = torch.zeros(P, device="cuda"), torch.zeros(P, device="cuda")
        g1 = torch.empty(P, device="cuda")
        s1 = torch.empty(U, 4, dtype=torch.float64, device="cuda")
        tp.ppo_update(c, p1, m1, v1, 1, dev["obs"], dev["action"], dev["logp"], dev["adv"],
                      dev["ret"], torch.from_numpy(idx[a]).cuda(), ws, grad=g1, stats=s1)
        torch.cuda.synchronize()
        assert torch.equal(prm[a, :P], p1), a
        assert torch.equal(m[a, :P], m1) and torch.equal(v[a, :P], v1), a
        assert torch.equal(grad[a], g1) and torch.equal(stats[a], s1), a
    # the agents really differ
    assert not torch.equal(prm[0, :P], prm[1, :P])


def test_agents_at_the_maximum_count():
    """1,024 learners (the documented maximum; a grid dimension of 1,024) of
    the tiny fp32 shape in one call: sampled agents equal their own
    tp_ppo_update calls bit for bit."""
    cfg = W.get_config("tiny")
    rows, B, A = 512, 64, 1024
    dims, bf, c, host, dev = _setup(cfg, rows, B)
    P = tp.ppo_param_count(c)
    rng = np.random.default_rng(33)
    idx = rng.integers(0, rows, (A, 1, B))
    start = np.stack([host["flat"] * (1.0 + 1e-3 * (a % 7)) for a in range(A)]).astype(np.float32)
    say(f"[ppo-agents] tiny A={A} P={P} B={B}")
    prm = torch.from_numpy(start).cuda()
    m, v = torch.zeros_like(prm), torch.zeros_like(prm)
    grad = torch.empty(A, P, device="cuda")
    tp.ppo_update_agents(c, prm, m, v, 1, dev["obs"], dev["action"], dev["logp"], dev["adv"],
                         dev["ret"], torch.from_numpy(idx).cuda(), tp.ppo_workspace(c, n_agents=A),
                         grad=grad)
    torch.cuda.synchronize()
    ws = tp.ppo_workspace(c)
    for a in (0, 1, 517, 1023):
        p1 = torch.from_numpy(start[a].copy()).cuda()
        m1, v1 = torch.zeros(P, device="cuda"), torch.zeros(P, device="cuda")
        g1 = torch.empty(P, device="cuda")
        tp.ppo_update(c, p1, m1, v1, 1, dev["obs"], dev["action"], dev["logp"], dev["adv"],
                      dev["ret"], torch.from_numpy(idx[a]).cuda(), ws, grad=g1)
        torch.cuda.synchronize()
        assert torch.equal(prm[a], p1) and torch.equal(grad[a], g1), a
        assert torch.equal(m[a], m1) and torch.equal(v[a], v1), a


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_critic_widths_other_than_the_actors(dtype):
    """The critic's widths are free (multiples of 32): the tiny 31-64-64-5
    actor with a 96-32 critic, whose first layer joins the actor's in the
    concatenated [W1; Wc1] product.  In bf16 these widths take the unstaged
    product kernel (K not in {128, 512, 1024}).  Gradient against the
    oracle, per segment."""
    cfg = W.get_config("tiny").with_(dtype=dtype)
    S, H1, H2, n = cfg.dims
    dims = (S, H1, H2, n, 96, 32)
    bf = dtype == "bf16"
    rows, B = 512, 64
    rng = np.random.default_rng(57)
    parts = []
    for name, shape in ppo.layout(*dims):
        if name == "log_std":
            parts.append(np.full(shape, -0.5))
        elif len(shape) == 2:
            parts.append(rng.uniform(-1, 1, shape) / np.sqrt(shape[1]))
        else:
            parts.append(rng.uniform(-0.1, 0.1, shape))
    flat = np.concatenate([p.reshape(-1) for p in parts]).astype(np.float32)
    obs, action, adv, ret, which = W.make_learner_data(cfg, rows)
    obs_t = torch.from_numpy(obs)
    if bf:
        obs_t = obs_t.to(torch.bfloat16)
    obs_vals = obs_t.float().numpy()
    p = ppo.unflatten(flat.astype(np.float64), dims)
    f = ppo.forward(p, obs_vals[:, :S], bf16=bf)
    logp = (ppo.log_prob(action, f["mu"], p["log_std"])
            - np.asarray(W.LOG_RATIO_OFFSETS)[which]).astype(np.float32)
    c = tp.ppo_cfg(dims, tp.TP_BF16 if bf else tp.TP_F32, B)
    P = tp.ppo_param_count(c)
    assert P == flat.shape[0]
    idx = rng.choice(rows, B, replace=False)[None]
    say(f"[ppo] tiny actor, 96-32 critic, {dtype}, P={P}")
    prm = torch.from_numpy(flat.copy()).cuda()
    m, v = torch.zeros(P, device="cuda"), torch.zeros(P, device="cuda")
    grad = torch.empty(P, device="cuda")
    tp.ppo_update(c, prm, m, v, 1, obs_t.cuda(), torch.from_numpy(action).cuda(),
                  torch.from_numpy(logp).cuda(), torch.from_numpy(adv).cuda(),
                  torch.from_numpy(ret).cuda(), torch.from_numpy(idx).cuda(), tp.ppo_workspace(c),
                  grad=grad)
    torch.cuda.synchronize()
    batch = ppo.gather(obs_vals, action, logp, adv, ret, idx[0], S)
    _, _, _, _, g_o = ppo.update(flat.astype(np.float64), np.zeros(P), np.zeros(P), 1, dims,
                                 batch, bf16=bf)
    _check_grad(dims, grad.cpu().numpy(), g_o, GRAD_TOL[dtype], f"critic 96-32 {dtype}")


def test_partial_column_blocks_in_staged_products():
    """A second actor layer 480 wide (1001-512-480-100 bf16 with a 512-512
    critic, batch 512): the forward of layer 2 and the first backward group
    take the LDS-staged product kernels, and their 480 columns end in a
    32-wide block, which the staged epilogue stores element by element.  One
    learner (64 x 64 tiles) is compared with the oracle per element; 16
    learners in one call (256 x 128 tiles for those launches) must give the
    single call's bits, parameters and moments included."""
    cfg = W.get_config("nasdaq100")
    S, H1, _, n = cfg.dims
    dims = (S, H1, 480, n, H1, H1)
    rows, B, A = 2048, 512, 16
    rng = np.random.default_rng(91)
    parts = []
    for name, shape in ppo.layout(*dims):
        if name == "log_std":
            parts.append(np.full(shape, -0.5))
        elif len(shape) == 2:
            parts.append(rng.uniform(-1, 1, shape) / np.sqrt(shape[1]))
        else:
            parts.append(rng.uniform(-0.1, 0.1, shape))
    flat = np.concatenate([p.reshape(-1) for p in parts]).astype(np.float32)
    obs, action, adv, ret, which = W.make_learner_data(cfg, rows)
    obs_t = torch.from_numpy(obs).to(torch.bfloat16)
    obs_vals = obs_t.float().numpy()
    p = ppo.unflatten(flat.astype(np.float64), dims)
    f = ppo.forward(p, obs_vals[:, :S], bf16=True)
    logp = (ppo.log_prob(action, f["mu"], p["log_std"])
            - np.asarray(W.LOG_RATIO_OFFSETS)[which]).astype(np.float32)
    c = tp.ppo_cfg(dims, tp.TP_BF16, B)
    P = tp.ppo_param_count(c)
    assert P == flat.shape[0]
    idx = rng.choice(rows, B, replace=False)
    dev = [torch.from_numpy(x).cuda() for x in (action, logp, adv, ret)]
    say(f"[ppo] 1001-512-480-100 bf16, 512-512 critic, B={B}, P={P}, one learner then {A}")
    prm = torch.from_numpy(flat.copy()).cuda()
    m, v = torch.zeros(P, device="cuda"), torch.zeros(P, device="cuda")
    grad = torch.empty(P, device="cuda")
    tp.ppo_update(c, prm, m, v, 1, obs_t.cuda(), *dev, torch.from_numpy(idx[None]).cuda(),
                  tp.ppo_workspace(c), grad=grad)
    torch.cuda.synchronize()
    batch = ppo.gather(obs_vals, action, logp, adv, ret, idx, S)
    _, _, _, _, g_o = ppo.update(flat.astype(np.float64), np.zeros(P), np.zeros(P), 1, dims,
                                 batch, bf16=True)
    _check_grad(dims, grad.cpu().numpy(), g_o, GRAD_TOL["bf16"], "1001-512-480-100 bf16")
    # the same minibatch for every learner: each must reproduce the single call
    pa = torch.from_numpy(np.tile(flat, (A, 1))).cuda()
    ma, va = torch.zeros(A, P, device="cuda"), torch.zeros(A, P, device="cuda")
    ga = torch.empty(A, P, device="cuda")
    tp.ppo_update_agents(c, pa, ma, va, 1, obs_t.cuda(), *dev,
                         torch.from_numpy(np.tile(idx, (A, 1, 1))).cuda(),
                         tp.ppo_workspace(c, n_agents=A), grad=ga)
    torch.cuda.synchronize()
    for a in range(A):
        assert torch.equal(ga[a], grad), a
        assert torch.equal(pa[a], prm) and torch.equal(ma[a], m) and torch.equal(va[a], v), a
