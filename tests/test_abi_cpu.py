"""C-ABI contract checks that need no GPU: every function declared in
include/tp.h is exported by libtp.so, and host-side argument checks return
the documented status codes before anything is launched."""

import ctypes as C
import os
import re
import subprocess

import pytest

from paper_2111_05188_amd import tp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tp.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tp_[a-z_0-9]+)\s*\(", src)))


def test_header_declares_the_abi():
    assert set(declared_functions()) == set(tp.EXPORTS)


def test_library_exports_every_declared_symbol():
    out = subprocess.check_output(["nm", "-D", "--defined-only", tp.LIB_PATH]).decode()
    exported = {l.split()[-1] for l in out.splitlines() if " T " in l}
    missing = [f for f in declared_functions() if f not in exported]
    assert not missing, missing
    L = tp.load()
    for f in declared_functions():
        assert hasattr(L, f)
    assert L.tp_version() == 2


PROBE_HEADER = os.path.join(ROOT, "include", "tp_probe.h")
PROBE_LIB = os.path.join(ROOT, "paper_2111_05188_amd", "libtpprobe.so")


def test_probe_library_exports_every_declared_symbol():
    """include/tp_probe.h (the measurement probes) against libtpprobe.so."""
    src = re.sub(r"/\*.*?\*/", "", open(PROBE_HEADER).read(), flags=re.S)
    declared = sorted(set(re.findall(r"\b(tpp_[a-z_0-9]+)\s*\(", src)))
    assert declared, "no probe declared"
    out = subprocess.check_output(["nm", "-D", "--defined-only", PROBE_LIB]).decode()
    exported = {l.split()[-1] for l in out.splitlines() if " T " in l}
    missing = [f for f in declared if f not in exported]
    assert not missing, missing
    L = C.CDLL(PROBE_LIB)
    for f in declared:
        assert hasattr(L, f)
    # argument checks return -1 before anything is launched
    L.tpp_copy.argtypes = [C.c_void_p, C.c_void_p, C.c_size_t, C.c_int, C.c_void_p]
    assert L.tpp_copy(None, None, 16, 1, None) == -1
    assert L.tpp_copy(0x1000, 0x2000, 15, 1, None) == -1


def _nasdaq_actor(dtype=tp.TP_BF16, dims=(1001, 512, 512, 100), A=1):
    a = tp.Actor()
    a.n_agents, a.envs_per_agent, a.dtype = A, 4096, dtype
    for i, d in enumerate(dims):
        a.dims[i] = d
    for l in range(3):
        a.W[l] = 0x1000
        a.b[l] = 0x2000
    a.log_std = 0x3000
    return a


def test_packed_bytes_host_only():
    L = tp.load()
    a = _nasdaq_actor()
    nb = L.tp_actor_packed_bytes(C.byref(a))
    # 3 layers of bf16 fragments + guards + biases + log_std
    frag = (32 * 32 + 32 * 16 + 7 * 16) * 1024
    assert frag < nb < frag + 64 * 1024
    a16 = _nasdaq_actor(A=16)
    assert L.tp_actor_packed_bytes(C.byref(a16)) == 16 * nb
    bad = _nasdaq_actor(dims=(1001, 500, 512, 100))
    assert L.tp_actor_packed_bytes(C.byref(bad)) == 0
    assert "multiples of 128" in tp.last_error()


def test_rollout_path_host_only():
    """Which rollout kernel a market and actor shape get, decided on the
    host: the role-split kernel for 100 stocks with 4, 8 or 10 indicators
    each and two equal bf16 hidden layers of 256 to 1024 (multiples of 256),
    the generic one otherwise."""
    L = tp.load()
    x = 0x100000
    m = tp.Market(x, x, 100, 100, 8)
    for H in (256, 512, 768, 1024):
        assert L.tp_rollout_path(C.byref(m), C.byref(_nasdaq_actor(dims=(1001, H, H, 100)))) == 1
    for dims in ((1001, 384, 384, 100), (1001, 512, 256, 100), (1001, 1280, 1280, 100)):
        assert L.tp_rollout_path(C.byref(m), C.byref(_nasdaq_actor(dims=dims))) == 0
    assert L.tp_rollout_path(C.byref(m), C.byref(_nasdaq_actor(dtype=tp.TP_F32))) == 0
    for I in (4, 10):
        mI = tp.Market(x, x, 100, 100, I)
        for H in (256, 512, 768, 1024):
            a = _nasdaq_actor(dims=(201 + 100 * I, H, H, 100))
            assert L.tp_rollout_path(C.byref(mI), C.byref(a)) == 1
    m6 = tp.Market(x, x, 100, 100, 6)
    assert L.tp_rollout_path(C.byref(m6), C.byref(_nasdaq_actor(dims=(801, 512, 512, 100)))) == 0
    m30 = tp.Market(x, x, 100, 32, 8)
    assert L.tp_rollout_path(C.byref(m30), C.byref(_nasdaq_actor(dims=(321, 512, 512, 32)))) == 0
    assert L.tp_rollout_path(C.byref(m), C.byref(_nasdaq_actor(dims=(1001, 500, 512, 100)))) < 0


def test_argument_errors_without_gpu():
    L = tp.load()
    assert L.tp_gae(None, None, None, 1, 1, 0.99, 0.95, None, None, None) == tp.TP_EINVAL
    assert "NULL" in tp.last_error()
    x = 0x100000
    assert L.tp_gae(x, x, x, 0, 4, 0.99, 0.95, x, x, None) == tp.TP_EINVAL
    assert L.tp_gae(x, x, x, 4, 4, 1.5, 0.95, x, x, None) == tp.TP_EINVAL
    assert L.tp_gae(x, x, x, 4, 4, 0.99, -0.1, x, x, None) == tp.TP_EINVAL
    m = tp.Market(x, x, 100, 200, 8)
    assert L.tp_env_step(C.byref(m), None, None, None, None, None, 0, 0, None) == tp.TP_EINVAL
    assert "market.n" in tp.last_error()
    m = tp.Market(x, x, 100, 10, 8)
    cfg = tp.env_cfg(100, 10, 1e-3, 1e6, 2 ** -12, 2 ** -20, 2 ** -7, 2 ** -7)
    bad_cfg = tp.env_cfg(0, 10, 1e-3, 1e6, 2 ** -12, 2 ** -20, 2 ** -7, 2 ** -7)
    st = tp.EnvState(x, x, x, 4)
    assert L.tp_env_step(C.byref(m), C.byref(bad_cfg), C.byref(st), x, x, None, 0, 0, None) == tp.TP_EINVAL
    assert "hmax" in tp.last_error()
    # obs stride must cover K_pad and be a multiple of 8
    assert L.tp_env_reset(C.byref(m), C.byref(cfg), C.byref(st), x, x, 100, 1, None) == tp.TP_EINVAL
    assert "ld_obs" in tp.last_error()
    # rollout: horizon exceeded -> TP_ERANGE; unpacked buffer -> TP_EINVAL
    a = _nasdaq_actor(dims=(1 + 20 + 80, 128, 128, 10))
    a.envs_per_agent = 4
    tr = tp.Traj(None, 0, x, x, x, x, None, None, None)
    assert L.tp_rollout(C.byref(m), C.byref(cfg), C.byref(st), C.byref(a), x, 1 << 30,
                        1, 5, 10, C.byref(tr), None) == tp.TP_ERANGE
    assert L.tp_rollout(C.byref(m), C.byref(cfg), C.byref(st), C.byref(a), x, 1 << 30,
                        1, 0, 10, C.byref(tr), None) == tp.TP_EINVAL
    assert "tp_actor_pack" in tp.last_error()
    # actor that does not match the market
    a2 = _nasdaq_actor(dims=(999, 128, 128, 10))
    a2.envs_per_agent = 4
    assert L.tp_rollout(C.byref(m), C.byref(cfg), C.byref(st), C.byref(a2), x, 1 << 30,
                        1, 0, 10, C.byref(tr), None) == tp.TP_EINVAL
    assert "match the market" in tp.last_error()
    # empty inputs: no envs, or a rollout of no steps
    st0 = tp.EnvState(x, x, x, 0)
    assert L.tp_rollout(C.byref(m), C.byref(cfg), C.byref(st0), C.byref(a), x, 1 << 30,
                        1, 0, 10, C.byref(tr), None) == tp.TP_EINVAL
    assert "state.E" in tp.last_error()
    assert L.tp_env_step(C.byref(m), C.byref(cfg), C.byref(st0), x, x, None, 0, 0, None) == tp.TP_EINVAL
    assert L.tp_rollout(C.byref(m), C.byref(cfg), C.byref(st), C.byref(a), x, 1 << 30,
                        1, 0, 0, C.byref(tr), None) == tp.TP_EINVAL
    assert "L = 0" in tp.last_error()
    # the largest market: n * n_ind = 1024 accepted, 1025 refused
    big = tp.Market(x, x, 100, 128, 8)
    too_big = tp.Market(x, x, 100, 125, 9)
    ab = _nasdaq_actor(dims=(1 + 256 + 1024, 128, 128, 128))
    assert L.tp_rollout_path(C.byref(big), C.byref(ab)) == 0
    assert L.tp_rollout_path(C.byref(too_big), C.byref(ab)) == tp.TP_EUNSUPPORTED


def _critic(dims=(1001, 512, 512), dtype=tp.TP_BF16, A=1, epa=4096):
    c = tp.Critic()
    c.n_agents, c.envs_per_agent, c.dtype = A, epa, dtype
    for i, d in enumerate(dims):
        c.dims[i] = d
    for l in range(3):
        c.W[l] = 0x1000
        c.b[l] = 0x2000
    return c


def test_critic_packed_bytes_host_only():
    L = tp.load()
    # MFMA layout: two layers of bf16 fragments, w3 and biases in fp32
    nb = L.tp_critic_packed_bytes(C.byref(_critic()))
    frag = (32 * 32 + 32 * 16) * 1024
    assert frag < nb < frag + 16 * 1024
    assert L.tp_critic_packed_bytes(C.byref(_critic(A=3))) == 3 * nb
    # generic layout (fp32 transposes): K_pad x H1 + H1 x H2 floats
    nb32 = L.tp_critic_packed_bytes(C.byref(_critic(dims=(301, 256, 256), dtype=tp.TP_F32)))
    assert (320 * 256 + 256 * 256) * 4 < nb32 < (320 * 256 + 256 * 256) * 4 + 8 * 1024
    assert L.tp_critic_packed_bytes(C.byref(_critic(dims=(301, 250, 256)))) == 0
    assert "multiples of 4" in tp.last_error()


def test_critic_argument_errors_without_gpu():
    L = tp.load()
    x = 0x100000
    c = _critic(A=2, epa=8)
    # E must equal n_agents * envs_per_agent
    assert L.tp_critic_value(C.byref(c), x, 1 << 30, x, 1024, 3, 15, x, None) == tp.TP_EINVAL
    assert "envs_per_agent" in tp.last_error()
    # observation pitch must cover K_pad
    assert L.tp_critic_value(C.byref(c), x, 1 << 30, x, 1000, 3, 16, x, None) == tp.TP_EINVAL
    assert "ld_obs" in tp.last_error()
    # a buffer that tp_critic_pack did not fill
    assert L.tp_critic_value(C.byref(c), x, 1 << 30, x, 1024, 3, 16, x, None) == tp.TP_EINVAL
    assert "tp_critic_pack" in tp.last_error()
    assert L.tp_critic_value(None, x, 1 << 30, x, 1024, 3, 16, x, None) == tp.TP_EINVAL
    assert L.tp_critic_value(C.byref(c), x, 1 << 30, x, 1024, 0, 16, x, None) == tp.TP_EINVAL


def test_evolution_argument_errors_without_gpu():
    L = tp.load()
    x = 0x100000
    assert L.tp_ensemble_fuse(None, 2, 2, 10, None) == tp.TP_EINVAL
    assert L.tp_ensemble_fuse(x, 2, 0, 10, None) == tp.TP_EINVAL
    # envs must split evenly over agents
    assert L.tp_fitness(x, 10, 15, 2, 0.99, x, x, None) == tp.TP_EINVAL
    assert "multiple" in tp.last_error()
    assert L.tp_fitness(x, 10, 16, 2, 1.5, x, x, None) == tp.TP_EINVAL
    assert L.tp_fitness(x, 10, 16, 2, 0.99, None, x, None) == tp.TP_EINVAL
    assert L.tp_keep_best(x, x, x, x, None, 4, 10, None) == tp.TP_EINVAL
    assert L.tp_keep_best(x, x, x, x, x, 0, 10, None) == tp.TP_EINVAL
    # the selector ranks at most 1024 agents and keeps 1..N of them
    assert L.tp_select(x, x, 1025, 10, 1, x, None) == tp.TP_EINVAL
    assert L.tp_select(x, x, 8, 10, 0, x, None) == tp.TP_EINVAL
    assert L.tp_select(x, x, 8, 10, 9, x, None) == tp.TP_EINVAL
    assert "keep" in tp.last_error()


def test_ppo_sizes_and_argument_errors_without_gpu():
    from oracle import ppo
    L = tp.load()
    dims = (1001, 512, 512, 100, 512, 512)
    c = tp.ppo_cfg(dims, tp.TP_BF16, 1024)
    assert tp.ppo_param_count(c) == ppo.param_count(*dims)
    # workspace: at least the operand copies and the fp32 gradient
    nb = L.tp_ppo_workspace_bytes(C.byref(c))
    assert nb > 4 * ppo.param_count(*dims) + 2 * (1024 * 1024 * 2)
    for bad, msg in ((tp.ppo_cfg((1001, 500, 512, 100, 512, 512), tp.TP_BF16, 1024), "multiples"),
                     (tp.ppo_cfg(dims, tp.TP_BF16, 1000), "batch"),
                     (tp.ppo_cfg((1001, 512, 512, 129, 512, 512), tp.TP_BF16, 1024), "n <= 128"),
                     (tp.ppo_cfg(dims, tp.TP_BF16, 1024, clip=1.5), "clip")):
        assert L.tp_ppo_param_count(C.byref(bad)) == 0
        assert msg in tp.last_error()
    x = 0x100000
    args = [C.byref(c), x, x, x, 1, 1, x, 1024, x, x, x, x, 4096, x, None, None, x, nb, None]
    a = list(args)
    a[1] = None
    assert L.tp_ppo_update(*a) == tp.TP_EINVAL and "NULL" in tp.last_error()
    a = list(args)
    a[17] = nb - 1
    assert L.tp_ppo_update(*a) == tp.TP_EINVAL and "workspace" in tp.last_error()
    a = list(args)
    a[4] = 0
    assert L.tp_ppo_update(*a) == tp.TP_EINVAL and "step0" in tp.last_error()
    a = list(args)
    a[7] = 1000
    assert L.tp_ppo_update(*a) == tp.TP_EINVAL and "ld_obs" in tp.last_error()


def test_ppo_agents_argument_errors_without_gpu():
    L = tp.load()
    dims = (1001, 512, 512, 100, 512, 512)
    c = tp.ppo_cfg(dims, tp.TP_BF16, 1024)
    P = tp.ppo_param_count(c)
    nb = L.tp_ppo_workspace_bytes(C.byref(c))
    x = 0x100000
    # cfg, n_agents, agent_stride, params, m, v, step0, n_updates, obs, ld_obs, action, logp,
    # adv, ret, rows, idx, grad, stats, workspace, workspace_bytes, stream
    args = [C.byref(c), 4, P, x, x, x, 1, 1, x, 1024, x, x, x, x, 4096, x, None, None, x, 4 * nb,
            None]
    for i, v, msg in ((1, 0, "n_agents"), (1, 1025, "n_agents"), (2, P - 1, "overlap"),
                      (19, 4 * nb - 1, "workspace"), (3, None, "NULL"), (6, 0, "step0")):
        a = list(args)
        a[i] = v
        assert L.tp_ppo_update_agents(*a) == tp.TP_EINVAL, (i, v)
        assert msg in tp.last_error(), tp.last_error()


def test_boundary_hygiene_without_gpu():
    """Host-only parts of the boundary: the start-row check (TP_ERANGE with
    the first offending env), the packed-buffer registry's release, the
    indicator-count limit and the alignment of the invalid-env counter."""
    import numpy as np
    L = tp.load()
    t0 = np.array([0, 10, 390 * 5, 42], np.int64)
    tp.check_starts(t0, 390 * 6 + 1, 390)           # every start has 390 rows
    with pytest.raises(tp.TPError) as ei:
        tp.check_starts(t0, 390 * 6, 390)           # env 2 is one row short
    assert ei.value.code == tp.TP_ERANGE and "env 2" in str(ei.value)
    bad = np.array([5, -1], np.int64)
    with pytest.raises(tp.TPError) as ei:
        tp.check_starts(bad, 1000, 10)
    assert ei.value.code == tp.TP_ERANGE and "env 1" in str(ei.value)
    assert L.tp_check_starts(None, 4, 100, 10) == tp.TP_EINVAL
    assert L.tp_check_starts(t0.ctypes.data, 4, 100, 0) == tp.TP_EINVAL
    # release of a buffer that was never packed
    assert L.tp_actor_release(0x123400) == tp.TP_EINVAL
    assert "not a packed actor" in tp.last_error()
    assert L.tp_critic_release(0x123400) == tp.TP_EINVAL
    # more indicator values than the kernels hold: TP_EUNSUPPORTED
    x = 0x100000
    cfg = tp.env_cfg(100, 10, 1e-3, 1e6, 2 ** -12, 2 ** -20, 2 ** -7, 2 ** -7)
    st = tp.EnvState(x, x, x, 4, None)
    m = tp.Market(x, x, 100, 100, 11)
    assert L.tp_env_step(C.byref(m), C.byref(cfg), C.byref(st), x, x, None, 0, 0,
                         None) == tp.TP_EUNSUPPORTED
    assert "1024" in tp.last_error()
    # a misaligned invalid-env counter
    m = tp.Market(x, x, 100, 10, 8)
    st = tp.EnvState(x, x, x, 4, x + 2)
    assert L.tp_env_step(C.byref(m), C.byref(cfg), C.byref(st), x, x, None, 0, 0,
                         None) == tp.TP_EINVAL
    assert "aligned" in tp.last_error()
