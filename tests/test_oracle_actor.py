"""Pins for the oracle's actor MLP, bf16 rounding, Philox stream, Gaussian
sampling and log-probability.

* MLP: against numpy fp64 matmul + tanh (a library routine).
* bf16 round-to-nearest-even: against torch's CPU float32 -> bfloat16 cast.
* Philox4x32-10 (Salmon et al., SC'11): against ROCm's rocRAND host
  implementation of the same generator (its header-only engine, compiled
  here with g++ from `tests/philox_rocrand.cpp`), on random and edge-case
  counters and keys and on the counter patterns the sampling and the
  minibatch draws use; further, an inverse written independently from the
  round's definition recovers the counter, and statistics (uniformity,
  avalanche).
* Box-Muller normals: moments and a KS test against N(0,1); independence
  across counters.
* Sampling: sigma -> 0 gives a = mu exactly; logp equals the analytic
  Gaussian log-density of the sampled action (scipy).
"""

import numpy as np
import pytest
import scipy.stats as st
import torch

import oracle
import workloads as W


# ------------------------------------------------------------------ bf16

def test_bf16_rne_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.normal(0, 1, 20000).astype(np.float32),
        rng.normal(0, 1e-30, 2000).astype(np.float32),
        (rng.normal(0, 1, 2000) * 1e30).astype(np.float32),
        np.array([0.0, -0.0, 1.0, -1.0, np.inf, -np.inf, 3.4e38, -3.4e38,
                  1e-45, -1e-45], np.float32)])
    # exact halfway cases: low 16 bits = 0x8000 with even and odd kept part
    u = rng.integers(0, 2 ** 32, 4000, dtype=np.uint64).astype(np.uint32)
    u = (u & np.uint32(0xFFFF0000)) | np.uint32(0x8000)
    halfway = u.view(np.float32)
    halfway = halfway[np.isfinite(halfway)]
    x = np.concatenate([x, halfway])
    ours = oracle.bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    assert np.isnan(oracle.bf16_value(oracle.bf16_bits(np.array([np.nan], np.float32))))


# ------------------------------------------------------------------- MLP

def _np_mlp(W, b, x, bf16):
    def r(a):
        if not bf16:
            return a
        return torch.from_numpy(np.asarray(a, np.float32)).to(torch.bfloat16).float().numpy()
    h = r(x).astype(np.float64)
    for l in range(3):
        y = h @ r(W[l]).astype(np.float64).T + b[l].astype(np.float64)
        y = y.astype(np.float32)
        if l < 2:
            y = np.tanh(y.astype(np.float64)).astype(np.float32)
            y = r(y)
        h = y.astype(np.float64)
    return h.astype(np.float32)


@pytest.mark.parametrize("name", ["tiny", "dow30"])
def test_mlp_fp32_vs_numpy(name):
    cfg = W.get_config(name)
    Wt, b, ls = W.make_actor(cfg)
    act = oracle.actor(Wt, b, ls, cfg.dims, False, cfg.envs_per_agent)
    x = np.random.default_rng(1).normal(0, 1, (32, cfg.S)).astype(np.float32)
    mu = oracle.mlp(act, 0, x)
    ref = _np_mlp([w[0] for w in Wt], [v[0] for v in b], x, False)
    scale = np.sqrt(np.mean(ref ** 2))
    assert np.max(np.abs(mu - ref) / np.maximum(np.abs(ref), scale)) < 1e-6


def test_mlp_bf16_vs_numpy_small():
    cfg = W.get_config("nasdaq100").with_(n=12, n_ind=3, hidden=(64, 64))
    Wt, b, ls = W.make_actor(cfg)
    act = oracle.actor(Wt, b, ls, cfg.dims, True, 1)
    x = np.random.default_rng(2).normal(0, 1, (16, cfg.S)).astype(np.float32)
    mu = oracle.mlp(act, 0, x)
    ref = _np_mlp([w[0] for w in Wt], [v[0] for v in b], x, True)
    # hidden activations are rounded to bf16 on both sides; a tanh ulp
    # difference can flip one bf16 rounding, hence a small tolerance
    scale = np.sqrt(np.mean(ref ** 2))
    assert np.max(np.abs(mu - ref) / np.maximum(np.abs(ref), scale)) < 1e-2
    assert np.mean(np.abs(mu - ref)) < 1e-4 * scale


def test_mlp_agents_use_their_own_weights():
    cfg = W.get_config("tiny").with_(n_agents=3, E=6)
    Wt, b, ls = W.make_actor(cfg)
    act = oracle.actor(Wt, b, ls, cfg.dims, False, 2)
    x = np.random.default_rng(3).normal(0, 1, (4, cfg.S)).astype(np.float32)
    for a in range(3):
        ref = _np_mlp([w[a] for w in Wt], [v[a] for v in b], x, False)
        assert np.allclose(oracle.mlp(act, a, x), ref, rtol=1e-5, atol=1e-6)


# ---------------------------------------------------------------- Philox

M0, M1 = 0xD2511F53, 0xCD9E8D57
W0, W1 = 0x9E3779B9, 0xBB67AE85
MASK = 0xFFFFFFFF


def _philox_inverse(y, key):
    """Undo ten Philox4x32 rounds.  A round maps (x0,x1,x2,x3) to
    (hi(M1*x2)^x1^k0, lo(M1*x2), hi(M0*x0)^x3^k1, lo(M0*x0)); the low
    products are invertible mod 2^32 because M0, M1 are odd."""
    inv0, inv1 = pow(M0, -1, 2 ** 32), pow(M1, -1, 2 ** 32)
    keys = [((key[0] + r * W0) & MASK, (key[1] + r * W1) & MASK) for r in range(10)]
    y0, y1, y2, y3 = (int(v) for v in y)
    for k0, k1 in reversed(keys):
        x2 = (y1 * inv1) & MASK
        x0 = (y3 * inv0) & MASK
        x1 = y0 ^ ((M1 * x2) >> 32) ^ k0
        x3 = y2 ^ ((M0 * x0) >> 32) ^ k1
        y0, y1, y2, y3 = x0, x1, x2, x3
    return [y0, y1, y2, y3]


ROCRAND_HEADER = "/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"


@pytest.fixture(scope="module")
def rocrand_philox(tmp_path_factory):
    """Philox4x32-10 words from rocRAND's host engine, for lists of
    (ctr, key) pairs (four and two 32-bit words)."""
    import os
    import shutil
    import subprocess
    if not os.path.exists(ROCRAND_HEADER) or shutil.which("g++") is None:
        pytest.skip("rocRAND headers or g++ not available")
    src = os.path.join(os.path.dirname(__file__), "philox_rocrand.cpp")
    exe = str(tmp_path_factory.mktemp("philox") / "philox_rocrand")
    subprocess.run(["g++", "-O1", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    src, "-o", exe], check=True, capture_output=True)

    def run(cases):
        lines = "".join(f"{k[0] | k[1] << 32} {c[0] | c[1] << 32} {c[2] | c[3] << 32}\n"
                        for c, k in cases)
        out = subprocess.run([exe], input=lines, check=True, capture_output=True, text=True)
        return [[int(w) for w in ln.split()] for ln in out.stdout.splitlines()]
    return run


def test_philox_matches_rocrand(rocrand_philox):
    rng = np.random.default_rng(11)
    edge = [0, 1, 0x7FFFFFFF, 0x80000000, 0xFFFFFFFE, MASK]
    cases = []
    for _ in range(1500):
        ctr = [int(v) for v in rng.integers(0, 2 ** 32, 4, dtype=np.uint64)]
        key = [int(v) for v in rng.integers(0, 2 ** 32, 2, dtype=np.uint64)]
        cases.append((ctr, key))
    for _ in range(300):
        cases.append(([int(rng.choice(edge)) for _ in range(4)],
                      [int(rng.choice(edge)) for _ in range(2)]))
    # the counter patterns of the action noise (i/4, env, step, agent) and of
    # the minibatch draws (i/4, counter, agent, 0x4D42), key = the seed's halves
    seed = 0x0123456789ABCDEF
    key = [seed & MASK, seed >> 32]
    for q in range(0, 25, 6):
        for env in (0, 4095, 65535):
            cases.append(([q, env, 389, 15], key))
    for q in (0, 255):
        cases.append(([q, 12479, 3, 0x4D42], key))
    want = rocrand_philox(cases)
    got = [[int(w) for w in oracle.philox(c, k)] for c, k in cases]
    assert got == want


def test_philox_inverse_recovers_counter():
    rng = np.random.default_rng(7)
    for _ in range(300):
        ctr = [int(v) for v in rng.integers(0, 2 ** 32, 4, dtype=np.uint64)]
        key = [int(v) for v in rng.integers(0, 2 ** 32, 2, dtype=np.uint64)]
        y = oracle.philox(ctr, key)
        assert _philox_inverse(y, key) == ctr


def test_philox_statistics():
    # byte histogram of 4 * 20000 output words is uniform; single-bit counter
    # changes flip about half of the 128 output bits
    key = [0x1234567, 0x89ABCDE]
    words = np.array([oracle.philox([i, 3, 5, 0], key) for i in range(20000)],
                     dtype=np.uint32).ravel()
    counts = np.bincount(words.view(np.uint8), minlength=256)
    chi2 = st.chisquare(counts)
    assert chi2.pvalue > 1e-4
    flips = []
    for i in range(200):
        base = oracle.philox([i, 7, 9, 11], key)
        for bit in (0, 13, 31):
            alt = oracle.philox([i ^ (1 << bit), 7, 9, 11], key)
            flips.append(sum(bin(int(a) ^ int(b)).count("1") for a, b in zip(base, alt)))
    assert abs(np.mean(flips) - 64) < 2.0


def test_uniform_mapping_exact_and_open_interval():
    assert oracle.uniform(0) == 0.5 * 2 ** -23
    assert oracle.uniform(0xFFFFFFFF) == 1 - 0.5 * 2 ** -23
    for w in (1 << 9, 12345 << 9, 0xABCDEF01):
        assert oracle.uniform(w) == ((w >> 9) + 0.5) * 2.0 ** -23


# ------------------------------------------------------------- normals

def test_box_muller_normals_distribution():
    z = np.concatenate([oracle.normals(99, s, e, 0, 100)
                        for s in range(40) for e in range(50)])
    assert z.size == 200000
    assert abs(z.mean()) < 0.01 and abs(z.var() - 1) < 0.015
    assert st.kstest(z, "norm").pvalue > 1e-3
    # different counters (env, step, agent, seed) give uncorrelated streams
    a = oracle.normals(99, 3, 4, 0, 4000)
    for other in (oracle.normals(99, 3, 5, 0, 4000), oracle.normals(99, 4, 4, 0, 4000),
                  oracle.normals(99, 3, 4, 1, 4000), oracle.normals(98, 3, 4, 0, 4000)):
        assert abs(np.corrcoef(a, other)[0, 1]) < 0.06


def test_box_muller_pair_members_independent():
    # the two normals of one Box-Muller pair (cos and sin branch) and the two
    # pairs of one Philox counter are independent N(0,1) draws
    z = np.stack([oracle.normals(3, s, e, 0, 4)
                  for s in range(100) for e in range(200)])
    for i, j in ((0, 1), (2, 3), (0, 2), (1, 3)):
        assert abs(np.corrcoef(z[:, i], z[:, j])[0, 1]) < 0.02
        both = np.mean((z[:, i] > 0) & (z[:, j] > 0))
        assert abs(both - 0.25) < 0.01
        assert abs(np.mean(z[:, i] * z[:, j] * z[:, j])) < 0.03


def test_normals_prefix_consistent():
    # stock i's normal does not depend on n (counter i/4, word i%4)
    a = oracle.normals(5, 1, 2, 3, 7)
    b = oracle.normals(5, 1, 2, 3, 100)
    assert np.array_equal(a, b[:7])


# ------------------------------------------------------------- sampling

def _tiny_rollout(log_std_value, teacher=False, L=3):
    cfg = W.get_config("tiny")
    mk = W.make_market(cfg)
    m = oracle.market(mk.price, mk.ind)
    Wt, b, ls = W.make_actor(cfg)
    ls = np.full_like(ls, log_std_value)
    act = oracle.actor(Wt, b, ls, cfg.dims, False, cfg.E)
    c = oracle.env_cfg(cfg)
    cash, sh, t = oracle.env_reset(c, np.zeros(8, np.int64), cfg.n)
    out = oracle.rollout(m, c, act, cash, sh, t, 77, 0, L, cfg.K_pad)
    return cfg, out, ls


def test_sigma_to_zero_gives_mean_action():
    cfg, out, _ = _tiny_rollout(-200.0)     # exp(-200) underflows to 0 in fp32
    assert np.array_equal(out["act"], out["mu"])


def test_logp_is_gaussian_log_density():
    cfg, out, ls = _tiny_rollout(-0.5)
    a, mu = out["act"].astype(np.float64), out["mu"].astype(np.float64)
    sigma = np.exp(ls[0].astype(np.float64))
    ref = st.norm.logpdf(a, loc=mu, scale=sigma).sum(axis=-1)
    assert np.allclose(out["logp"], ref, rtol=1e-5, atol=1e-4)


def test_done_flag_marks_episode_end():
    cfg = W.get_config("tiny")
    mk = W.make_market(cfg)
    m = oracle.market(mk.price, mk.ind)
    Wt, b, ls = W.make_actor(cfg)
    act = oracle.actor(Wt, b, ls, cfg.dims, False, cfg.E)
    c = oracle.env_cfg(cfg, horizon=10)
    cash, sh, t = oracle.env_reset(c, np.zeros(4, np.int64), cfg.n)
    out = oracle.rollout(m, c, act, cash, sh, t, 1, 0, 10, cfg.K_pad)
    assert out["done"][:9].sum() == 0 and out["done"][9].all()
