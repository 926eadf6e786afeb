"""Per-kernel bandwidth benchmark of the standalone HBM-bound kernels.

    python -m paper_2111_05188_amd.kbench [--envs 65536] [--iters 20]

Times, with HIP events on the launch stream:
  * env_step: one teacher-forced transition of every env of the 100-stock
    minute workload (bf16 observation written), at the 65,536-env stress
    shape by default, where the rows touched per launch exceed the 256 MB
    last-level cache;
  * gae: the GAE scan over a 390 x E rollout;
  * critic: the critic forward (1001-512-512-1 bf16) over a 100-stock
    minute trajectory, 391 x 4,096 observation rows, against the bf16 MFMA
    peak (algorithmic FLOPs 2 (S H1 + H1 H2 + H2) per row);
  * metrics: the backtest metrics of total-asset series, for 4,096 envs
    over one 390-minute day and for 16 agents over a year of minute bars
    (98,280 steps); algorithmic bytes T E 8 (series) + 8 E (V_0) + 40 E
    (five metrics);
  * evolution: ensemble fusion of 16 pods (4 agents x 4 pods) over the
    actor and critic parameters of the 100-stock minute workload (P floats
    per pod, N K P 4 bytes in and out), the fitness of a 390 x 16,384
    reward block (L E 4 + 8 E + 8 A bytes), keep-best over 16 agents all
    improving (A P 4 in and out) and the selector keeping 4 of 16 (12 P 4
    in and out);
  * learner: PPO updates of the 1001-512-512-100 actor and 1001-512-512-1
    critic (bf16 operands, fp32 masters and Adam), batch 2^10, 16 updates
    per call on a 390 x 4,096 trajectory; algorithmic FLOPs per update
    2B (2 S H1 + 3 H1 H2 + 3 H2 n + 2 S C1 + 3 C1 C2 + 3 C2) (forward of
    both networks, weight gradients, and input gradients except layer 1's);
    then the same for 16 agents per call (tp_ppo_update_agents);
  * rollout_shapes (only with --only rollout_shapes): the fused rollout
    step (reset, rollout with observations stored, GAE) of 4,096 envs x 390
    steps on each shape the role-split kernel takes: 100 stocks with 4, 8
    or 10 indicators, hidden widths 256, 512, 768 and 1024, on a 60-day
    minute market (the start rows, not the market's length, decide what
    the kernel does); FLOPs 2 (S H + H H + H n) per env-step;
  * train (only with --only train): one generation of the ensemble
    workload (4 agents x 4 pods of 1,024 envs, L = 390): rollout, critic,
    GAE, the learners' 8 L envs / B updates each in one agent-batched call,
    fusion, fitness, keep-best and selection;
  * probes: the device ceilings the roofline figures are read against,
    from libtpprobe.so: the dense bf16 MFMA issue rate (back-to-back
    v_mfma_f32_16x16x32_bf16 or v_mfma_f32_32x32x16_bf16 on register
    operands, 4 workgroups of four waves per CU) and the L2 -> CU stream one CU can pull in the rollout's
    weight-stream pattern (256 workgroups, one per CU, and 8 workgroups);
  * mfma_sweep (only with --only mfma_sweep): the issue rate of both bf16
    MFMA shapes over 1-8 accumulators per wave, operands shared or one pair
    per accumulator, and 1-4 waves per SIMD, with the shader clock the
    loops ran at;
  * copy: a plain device-to-device copy of 1 GiB (the reference kernel used
    to calibrate HBM byte counters: FETCH_SIZE and WRITE_SIZE of this copy
    should each read 1 GiB per launch).

Algorithmic bytes per env (env_step): action n*4 in; holdings 2*n*4 and
balance/time 2*(8+8) in and out; prices of rows t and t+1 2*n*4; indicators
of row t+1 n*I*4; observation S*2 out; reward 4 out.
GAE per env-step: reward, value, done in; advantage, return out (17 B).
Prints one JSON line.
"""

from __future__ import annotations

import argparse
import json
import sys

import numpy as np
import torch

from . import problem, tp

PEAK_HBM_GBS = 8000.0
PEAK_BF16_TFLOPS = 2500.0


def _time(fn, iters, stream):
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    fn()
    torch.cuda.synchronize()
    ev[0].record(stream)
    for _ in range(iters):
        fn()
    ev[1].record(stream)
    torch.cuda.synchronize()
    return ev[0].elapsed_time(ev[1]) / iters * 1e-3


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--envs", type=int, default=65536)
    ap.add_argument("--iters", type=int, default=20)
    ap.add_argument("--only", default=None,
                    choices=["env_step", "gae", "critic", "metrics", "evolution", "learner",
                             "train", "probes", "copy", "mfma_sweep", "sync", "rollout_shapes"])
    args = ap.parse_args()
    sys.path.insert(0, __file__.rsplit("/", 2)[0])
    import workloads as W

    tp.load()
    dev = "cuda"
    stream = torch.cuda.current_stream()
    cfg = W.get_config("stress").with_(E=args.envs)
    out = {"kernel_bench": "standalone kernels", "envs": cfg.E}
    E, n, I = cfg.E, cfg.n, cfg.n_ind

    if args.only in (None, "env_step"):
        print("[kbench] env_step: generating the 100-stock minute market", file=sys.stderr, flush=True)
        mk = W.make_market(cfg)
        mkt = tp.MarketT(torch.from_numpy(mk.price).to(dev), torch.from_numpy(mk.ind).to(dev))
        ecfg = problem.env_cfg(cfg)
        rng = np.random.default_rng(1)
        t0 = torch.from_numpy(rng.integers(0, cfg.T1 - 1 - 2 * (args.iters + 2), E)).to(dev)
        st = tp.StateT.empty(E, n)
        tp.env_reset(mkt, ecfg, st, t0)
        act = torch.from_numpy(W.make_actions(2, E, n, special=False)).to(dev)
        rew = torch.empty(E, device=dev)
        obs = torch.empty(E, cfg.K_pad, dtype=torch.bfloat16, device=dev)
        sec = _time(lambda: tp.env_step(mkt, ecfg, st, act, rew, obs), args.iters, stream)
        per_env = 4 * n + 2 * 4 * n + 2 * 16 + 2 * 4 * n + 4 * n * I + 2 * cfg.S + 4
        gbs = per_env * E / sec / 1e9
        out["env_step"] = {"launch_ms": sec * 1e3, "bytes_per_launch": per_env * E,
                           "GBs": gbs, "hbm_frac": gbs / PEAK_HBM_GBS}
        del mkt, st, act, rew, obs
        torch.cuda.empty_cache()

    if args.only in (None, "gae"):
        L = cfg.L
        print(f"[kbench] gae L={L} E={E}", file=sys.stderr, flush=True)
        r = torch.randn(L, E, device=dev)
        v = torch.randn(L + 1, E, device=dev)
        d = (torch.rand(L, E, device=dev) < 0.01).to(torch.uint8)
        adv = torch.empty(L, E, device=dev)
        ret = torch.empty(L, E, device=dev)
        sec = _time(lambda: tp.gae(r, v, d, cfg.gamma, cfg.lam, adv, ret), args.iters, stream)
        nbytes = 17 * L * E
        out["gae"] = {"launch_ms": sec * 1e3, "bytes_per_launch": nbytes,
                      "GBs": nbytes / sec / 1e9, "hbm_frac": nbytes / sec / 1e9 / PEAK_HBM_GBS}

    if args.only in (None, "critic"):
        # critic forward over a 100-stock minute trajectory: (L+1) x 4096 rows
        # of bf16 observations, 1001-512-512-1
        cc = W.get_config("nasdaq100")
        T, Ec = cc.L + 1, cc.E
        print(f"[kbench] critic T={T} E={Ec}", file=sys.stderr, flush=True)
        g = torch.Generator(device=dev).manual_seed(3)
        obs = torch.randn(T, Ec, cc.K_pad, device=dev, generator=g).to(torch.bfloat16)
        obs[:, :, cc.S:] = 0
        Wc, bc = W.make_critic(cc)
        crit = tp.CriticT([torch.from_numpy(w).to(dev) for w in Wc],
                          [torch.from_numpy(x).to(dev) for x in bc], cc.dims[:3],
                          tp.TP_BF16, cc.envs_per_agent)
        crit.pack()
        val = torch.empty(T, Ec, dtype=torch.float32, device=dev)
        sec = _time(lambda: tp.critic_value(crit, obs, val), args.iters, stream)
        S, H1, H2 = cc.dims[:3]
        flops = 2.0 * (S * H1 + H1 * H2 + H2) * T * Ec
        out["critic"] = {"launch_ms": sec * 1e3, "rows": T * Ec, "flops_per_launch": flops,
                         "TFLOPs": flops / sec / 1e12,
                         "mfma_frac": flops / sec / 1e12 / PEAK_BF16_TFLOPS,
                         "obs_GBs": obs.numel() * 2 / sec / 1e9}
        del obs, crit, val
        torch.cuda.empty_cache()

    if args.only in (None, "metrics"):
        out["metrics"] = {}
        for T, Em in ((390, 4096), (98280, 16)):
            print(f"[kbench] metrics T={T} E={Em}", file=sys.stderr, flush=True)
            g = torch.Generator(device=dev).manual_seed(T)
            v0 = torch.full((Em,), 1e6, dtype=torch.float64, device=dev)
            steps = 1.0 + 1e-3 * torch.randn(T, Em, dtype=torch.float64, device=dev, generator=g)
            v = v0 * torch.cumprod(steps, dim=0)
            met = torch.empty(Em, 5, dtype=torch.float64, device=dev)
            wk = tp.backtest_metrics_workspace(T, Em, dev)
            sec = _time(lambda: tp.backtest_metrics(v0, v, 252.0 * 390, 0.02, out=met, work=wk),
                        args.iters, stream)
            nbytes = 8 * T * Em + 8 * Em + 40 * Em
            out["metrics"][f"T{T}_E{Em}"] = {
                "launch_ms": sec * 1e3, "bytes_per_launch": nbytes, "GBs": nbytes / sec / 1e9,
                "hbm_frac": nbytes / sec / 1e9 / PEAK_HBM_GBS}
            del v0, steps, v, met, wk
        torch.cuda.empty_cache()

    if args.only in (None, "evolution"):
        cc = W.get_config("nasdaq100")
        S, H1, H2, A_ = cc.dims
        P = (S * H1 + H1 + H1 * H2 + H2 + H2 * A_ + 2 * A_) + (S * H1 + H1 + H1 * H2 + H2 + H2 + 1)
        N, K = 4, 4
        print(f"[kbench] evolution P={P}", file=sys.stderr, flush=True)
        ev = {}
        g = torch.Generator(device=dev).manual_seed(7)
        pods = torch.randn(N, K, P, device=dev, generator=g)
        sec = _time(lambda: tp.ensemble_fuse(pods), args.iters, stream)
        nb = 2 * N * K * P * 4
        ev["fuse"] = {"launch_ms": sec * 1e3, "bytes_per_launch": nb, "GBs": nb / sec / 1e9,
                      "hbm_frac": nb / sec / 1e9 / PEAK_HBM_GBS}
        del pods
        L, Ef, Af = 390, 16384, 16
        rew = 2.0 ** -8 * torch.randn(L, Ef, device=dev, generator=g)
        ret = torch.empty(Ef, dtype=torch.float64, device=dev)
        fit = torch.empty(Af, dtype=torch.float64, device=dev)
        sec = _time(lambda: tp.fitness(rew, Af, 0.99, env_return=ret, out=fit), args.iters, stream)
        nb = L * Ef * 4 + 8 * Ef + 8 * Af
        ev["fitness"] = {"launch_ms": sec * 1e3, "bytes_per_launch": nb, "GBs": nb / sec / 1e9,
                         "hbm_frac": nb / sec / 1e9 / PEAK_HBM_GBS}
        params = torch.randn(Af, P, device=dev, generator=g)
        bestp = torch.empty_like(params)
        fit = torch.arange(Af, dtype=torch.float64, device=dev)
        best = torch.full((Af,), float("nan"), dtype=torch.float64, device=dev)
        stall = torch.zeros(Af, dtype=torch.int32, device=dev)

        def kb():
            best.fill_(float("nan"))          # every agent improves: the full copy
            tp.keep_best(fit, best, stall, params, bestp)
        sec = _time(kb, args.iters, stream)
        nb = 2 * Af * P * 4
        ev["keep_best"] = {"launch_ms": sec * 1e3, "bytes_per_launch": nb, "GBs": nb / sec / 1e9,
                           "hbm_frac": nb / sec / 1e9 / PEAK_HBM_GBS,
                           "note": "includes a 16-element fill"}
        rank = torch.empty(Af, dtype=torch.int32, device=dev)
        sec = _time(lambda: tp.select(fit, params, 4, rank=rank), args.iters, stream)
        nb = 2 * (Af - 4) * P * 4
        ev["select"] = {"launch_ms": sec * 1e3, "bytes_per_launch": nb, "GBs": nb / sec / 1e9,
                        "hbm_frac": nb / sec / 1e9 / PEAK_HBM_GBS}
        out["evolution"] = {"P": P, **ev}
        del rew, ret, fit, params, bestp, best, stall, rank
        torch.cuda.empty_cache()

    if args.only in (None, "learner"):
        cc = W.get_config("nasdaq100")
        S, H1, H2, n = cc.dims
        C1, C2 = H1, H2
        B, NU, rows = 1024, 16, cc.L * cc.E
        print(f"[kbench] learner B={B} updates={NU}", file=sys.stderr, flush=True)
        c = tp.ppo_cfg((S, H1, H2, n, C1, C2), tp.TP_BF16, B)
        P = tp.ppo_param_count(c)
        g = torch.Generator(device=dev).manual_seed(11)
        obs = (0.5 * torch.randn(rows, cc.K_pad, device=dev, generator=g)).to(torch.bfloat16)
        obs[:, S:] = 0
        act = 0.6 * torch.randn(rows, n, device=dev, generator=g)
        logp = torch.full((rows,), -60.0, device=dev)
        adv = torch.randn(rows, device=dev, generator=g)
        ret = torch.randn(rows, device=dev, generator=g)
        params = torch.from_numpy(W.make_flat_params(cc)).to(dev)
        m = torch.zeros(P, device=dev)
        v = torch.zeros(P, device=dev)
        idx = torch.randint(0, rows, (NU, B), device=dev, generator=g)
        ws = tp.ppo_workspace(c)
        step = [1]

        def upd():
            tp.ppo_update(c, params, m, v, step[0], obs, act, logp, adv, ret, idx, ws)
            step[0] += NU
        sec = _time(upd, max(1, args.iters // 4), stream) / NU
        flops = 2.0 * B * (2 * S * H1 + 3 * H1 * H2 + 3 * H2 * n + 2 * S * C1 + 3 * C1 * C2
                           + 3 * C2)
        out["learner"] = {"update_ms": sec * 1e3, "flops_per_update": flops,
                          "TFLOPs": flops / sec / 1e12,
                          "mfma_frac": flops / sec / 1e12 / PEAK_BF16_TFLOPS, "P": P}
        del params, m, v, idx, ws
        torch.cuda.empty_cache()
        # the same updates for 16 agents in one call (tp_ppo_update_agents)
        A = 16
        print(f"[kbench] learner agents={A} B={B} updates={NU}", file=sys.stderr, flush=True)
        params = torch.from_numpy(np.stack([W.make_flat_params(cc, agent=a)
                                            for a in range(A)])).to(dev)
        m = torch.zeros(A, P, device=dev)
        v = torch.zeros(A, P, device=dev)
        idx = torch.randint(0, rows, (A, NU, B), device=dev, generator=g)
        ws = tp.ppo_workspace(c, n_agents=A)
        step = [1]

        def upd_agents():
            tp.ppo_update_agents(c, params, m, v, step[0], obs, act, logp, adv, ret, idx, ws)
            step[0] += NU
        sec = _time(upd_agents, max(1, args.iters // 4), stream) / NU
        out["learner"]["agents16"] = {"update_ms": sec * 1e3, "agent_update_ms": sec * 1e3 / A,
                                      "TFLOPs": A * flops / sec / 1e12,
                                      "mfma_frac": A * flops / sec / 1e12 / PEAK_BF16_TFLOPS}
        del obs, act, logp, adv, ret, params, m, v, idx, ws
        torch.cuda.empty_cache()

    if args.only == "rollout_shapes":
        shapes = {}
        for ni in (4, 8, 10):
            base = W.get_config("nasdaq100").with_(n_ind=ni, N=60 * W.MINUTES_PER_DAY)
            print(f"[kbench] rollout shapes: {base.n} stocks x {ni} indicators", file=sys.stderr,
                  flush=True)
            mk = W.make_market(base)
            t0 = W.make_t0(base)
            for H in (256, 512, 768, 1024):
                c = base.with_(hidden=(H, H))
                pb = problem.Problem(c, mk, W.make_actor(c), t0, store_obs=True, taps=False)
                pb.set_values(W.make_values(c))
                k = [0]

                def step():
                    pb.step(1000 + k[0], stream)
                    k[0] += 1
                sec = _time(step, max(2, args.iters // 4), stream)
                es = c.E * c.L / sec
                fl = es * c.flops_per_env_step()
                shapes[f"I{ni}_H{H}"] = {"S": c.S, "path": tp.rollout_path(pb.mkt, pb.actor),
                                         "step_ms": sec * 1e3, "env_steps_per_s": es,
                                         "us_per_lockstep_step": sec * 1e6 / c.L,
                                         "TFLOPs": fl / 1e12, "mfma_frac": fl / 1e12 / PEAK_BF16_TFLOPS}
                print(f"[kbench]   I={ni} H={H}: {es / 1e6:.1f} M env-steps/s", file=sys.stderr,
                      flush=True)
                del pb
                torch.cuda.empty_cache()
            del mk
        out["rollout_shapes"] = shapes

    if args.only == "train":   # opt-in: one generation is ~50,000 launches
        # one generation of the ensemble workload: 4 agents x 4 pods (16
        # learners of 1,024 envs), rollout, critic, GAE, 8 L envs / B
        # updates per learner in one agent-batched call, fusion, fitness,
        # keep-best and selection
        from paper_2111_05188_amd.train import Trainer
        ce = W.get_config("ensemble")
        NA, KP = 4, 4
        print(f"[kbench] train: {NA} agents x {KP} pods, E={ce.E}, L={ce.L}", file=sys.stderr,
              flush=True)
        mk = W.make_market(ce)
        flat = np.stack([W.make_flat_params(ce, agent=a) for a in range(NA * KP)])
        tr = Trainer(ce, mk, W.make_t0(ce), flat, NA, KP, device=dev)
        del mk, flat
        sec = _time(lambda: tr.epoch(stream), 1, stream)
        L16 = NA * KP
        out["train"] = {"generation_ms": sec * 1e3, "learners": L16,
                        "updates_per_learner": tr.updates, "env_steps": ce.E * ce.L,
                        "agent_updates_per_s": L16 * tr.updates / sec,
                        "learner_TFLOPs": L16 * tr.updates * 2.0 * 1024 * (
                            2 * 1001 * 512 + 3 * 512 * 512 + 3 * 512 * 100 + 2 * 1001 * 512
                            + 3 * 512 * 512 + 3 * 512) / sec / 1e12}
        del tr
        torch.cuda.empty_cache()

    if args.only in (None, "probes"):
        import ctypes as C
        import os
        pl = C.CDLL(os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtpprobe.so"))
        pl.tpp_mfma_issue.argtypes = [C.c_int, C.c_int, C.c_void_p, C.c_void_p]
        pl.tpp_mfma_issue_flops.restype = C.c_double
        pl.tpp_mfma_issue_flops.argtypes = [C.c_int, C.c_int]
        pl.tpp_l2_stream.argtypes = [C.c_void_p, C.c_size_t, C.c_int, C.c_int, C.c_int,
                                     C.c_void_p, C.c_void_p]
        sp = stream.cuda_stream
        blocks, iters = 1024, 4096
        sink = torch.empty(blocks * 256, device=dev)
        sec = _time(lambda: pl.tpp_mfma_issue(blocks, iters, sink.data_ptr(), sp), 5, stream)
        fl = pl.tpp_mfma_issue_flops(blocks, iters)
        probes = {"mfma_16x16x32_bf16_TFLOPs": fl / sec / 1e12,
                  "mfma_16x16x32_frac_of_2500": fl / sec / 1e12 / PEAK_BF16_TFLOPS}
        pl.tpp_mfma32_issue.argtypes = [C.c_int, C.c_int, C.c_void_p, C.c_void_p]
        pl.tpp_mfma32_issue_flops.restype = C.c_double
        pl.tpp_mfma32_issue_flops.argtypes = [C.c_int, C.c_int]
        sec = _time(lambda: pl.tpp_mfma32_issue(blocks, iters // 2, sink.data_ptr(), sp), 5,
                    stream)
        fl = pl.tpp_mfma32_issue_flops(blocks, iters // 2)
        probes["mfma_32x32x16_bf16_TFLOPs"] = fl / sec / 1e12
        probes["mfma_32x32x16_frac_of_2500"] = fl / sec / 1e12 / PEAK_BF16_TFLOPS
        fpw, reps = 200, 20
        buf = torch.ones(8 * fpw * 1024 // 4 + 16384, dtype=torch.int32, device=dev)
        for nb in (256, 8):
            so = torch.empty(nb * 512 * 4, dtype=torch.int32, device=dev)
            sec = _time(lambda: pl.tpp_l2_stream(buf.data_ptr(), buf.numel() * 4, fpw, reps, nb,
                                                 so.data_ptr(), sp), 5, stream)
            per_cu = 8 * fpw * 1024 * reps / sec / 1e9
            probes[f"l2_stream_GBs_per_CU_{nb}wg"] = per_cu
        out["probes"] = probes

    if args.only == "mfma_sweep":
        # issue rate of the two bf16 MFMA shapes over accumulators per wave,
        # shared or per-accumulator operands and waves per SIMD, with the
        # shader clock the loops ran at (s_memtime ticks over s_memrealtime's
        # 100 MHz ticks)
        import ctypes as C
        import os
        pl = C.CDLL(os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtpprobe.so"))
        pl.tpp_mfma_sweep.argtypes = [C.c_int] * 6 + [C.c_void_p, C.c_void_p, C.c_void_p]
        pl.tpp_mfma_sweep_flops.restype = C.c_double
        pl.tpp_mfma_sweep_flops.argtypes = [C.c_int] * 5
        sp = stream.cuda_stream
        clk = torch.zeros(2, dtype=torch.int64, device=dev)
        rows = []
        for m in (16, 32):
            for distinct in (0, 1):
                for nacc in (1, 2, 4, 8):
                    for blocks, waves in ((256, 4), (512, 4), (1024, 4), (2048, 4)):
                        # 2^28 (16x16x32) or 2^27 (32x32x16) instructions per launch
                        total = (1 << 28) if m == 16 else (1 << 27)
                        iters = max(1, total // (blocks * waves * nacc))
                        sink = torch.empty(blocks * waves * 64, device=dev)
                        fn = lambda: pl.tpp_mfma_sweep(m, nacc, distinct, blocks, waves, iters,
                                                       sink.data_ptr(), clk.data_ptr(), sp)
                        assert fn() == 0
                        sec = _time(fn, 3, stream)
                        c = clk.cpu().tolist()
                        tf = pl.tpp_mfma_sweep_flops(m, nacc, blocks, waves, iters) / sec / 1e12
                        rows.append({"shape": f"{m}x{m}x{512 // m}", "acc_per_wave": nacc,
                                     "operands": "per accumulator" if distinct else "shared",
                                     "waves_per_simd": blocks * waves // 1024,
                                     "TFLOPs": round(tf, 1),
                                     "frac_of_2500": round(tf / PEAK_BF16_TFLOPS, 3),
                                     "clock_GHz": round(0.1 * c[0] / max(c[1], 1), 3)})
                        print(f"[kbench] mfma sweep {rows[-1]}", file=sys.stderr, flush=True)
        out["mfma_sweep"] = rows

    if args.only == "sync":
        # workgroup handoff latency through one flag word (agent-scope
        # release/acquire, or relaxed agent-scope atomics), partners 8 apart
        # (the same XCD under round-robin dispatch) or 1 apart; and what
        # agent-scope fences cost a concurrent L2 weight stream
        import ctypes as C
        import os
        pl = C.CDLL(os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtpprobe.so"))
        pl.tpp_pingpong.argtypes = [C.c_int] * 5 + [C.c_void_p, C.c_void_p, C.c_void_p]
        pl.tpp_l2_stream_fence.argtypes = [C.c_void_p, C.c_size_t, C.c_int, C.c_int, C.c_int,
                                           C.c_int, C.c_int, C.c_void_p, C.c_void_p]
        sp = stream.cuda_stream
        res = []
        pairs, rounds = 128, 2000
        for mode in (0, 1):
            for stride in (8, 1):
                flags = torch.zeros(pairs * 32, dtype=torch.int32, device=dev)
                rec = torch.zeros(2 * pairs, 2, dtype=torch.int64, device=dev)
                assert pl.tpp_pingpong(mode, pairs, stride, rounds, 1 << 20, flags.data_ptr(),
                                       rec.data_ptr(), sp) == 0
                torch.cuda.synchronize()
                r = rec.cpu().numpy()
                xcc = (r[:, 0] & 0xFFFFFFFF).astype(np.int64)
                tmo = (r[:, 0] >> 32).astype(np.int64)
                ticks = r[:, 1].astype(np.float64)
                b = np.arange(2 * pairs)
                same = float(np.mean(xcc == xcc[b ^ stride]))
                rt_us = ticks / rounds * 0.01     # 100 MHz ticks -> us per round trip
                res.append({"mode": "release/acquire" if mode == 0 else "relaxed",
                            "partner_stride": stride, "same_xcd_frac": same,
                            "timeouts": int(tmo.sum()),
                            "round_trip_us_median": float(np.median(rt_us)),
                            "round_trip_us_max": float(rt_us.max()),
                            "xcc_of_first_16": xcc[:16].tolist()})
                print(f"[kbench] sync {res[-1]}", file=sys.stderr, flush=True)
        pl.tpp_pingpong_data.argtypes = [C.c_int] * 5 + [C.c_void_p] * 4
        for mode in (0, 1):
            for stride in (8, 1):
                flags = torch.zeros(pairs * 32, dtype=torch.int32, device=dev)
                data = torch.zeros(pairs * 2 * 1024 * 4, dtype=torch.int32, device=dev)
                rec = torch.zeros(2 * pairs, 6, dtype=torch.int32, device=dev)
                assert pl.tpp_pingpong_data(mode, pairs, stride, 500, 1 << 20, flags.data_ptr(),
                                            data.data_ptr(), rec.data_ptr(), sp) == 0
                torch.cuda.synchronize()
                r = rec.cpu().numpy().astype(np.int64)
                xcc, tmo = r[:, 0], r[:, 1]
                ticks = (r[:, 2] & 0xFFFFFFFF) + (r[:, 3] << 32)
                b = np.arange(2 * pairs)
                rt_us = ticks / 500 * 0.01
                res.append({"payload": "16 KiB", "mode": "plain store + sc0 load" if mode == 0
                            else "sc1 store + sc1 load", "partner_stride": stride,
                            "same_xcd_frac": float(np.mean(xcc == xcc[b ^ stride])),
                            "timeouts": int(tmo.sum()), "stale_words": int(r[:, 4].sum()),
                            "round_trip_us_median": float(np.median(rt_us)),
                            "round_trip_us_max": float(rt_us.max())})
                print(f"[kbench] sync {res[-1]}", file=sys.stderr, flush=True)
        fpw, reps = 200, 20
        buf = torch.ones(8 * fpw * 1024 // 4 + 16384, dtype=torch.int32, device=dev)
        so = torch.empty(256 * 512 * 4, dtype=torch.int32, device=dev)
        fence = []
        for mode, every in ((0, 1), (1, 64), (1, 16), (2, 64), (2, 16)):
            sec = _time(lambda: pl.tpp_l2_stream_fence(buf.data_ptr(), buf.numel() * 4, fpw,
                                                       reps, 256, mode, every, so.data_ptr(), sp),
                        5, stream)
            fence.append({"fence": ["none", "acquire", "release"][mode], "every_frags": every,
                          "GBs_per_CU": 8 * fpw * 1024 * reps / sec / 1e9})
            print(f"[kbench] stream {fence[-1]}", file=sys.stderr, flush=True)
        out["sync"] = {"pingpong": res, "l2_stream_with_fences": fence}

    if args.only in (None, "copy"):
        a = torch.empty(1 << 28, dtype=torch.float32, device=dev)   # 1 GiB
        b = torch.empty_like(a)
        a.fill_(1.0)
        sec = _time(lambda: b.copy_(a), args.iters, stream)
        out["copy_1GiB"] = {"launch_ms": sec * 1e3, "GBs": 2 * a.numel() * 4 / sec / 1e9}
        # the probe library's plain copy (16 bytes per lane, four loads in
        # flight, non-temporal) over a few grid sizes
        import ctypes as C
        import os
        pl = C.CDLL(os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtpprobe.so"))
        pl.tpp_copy.argtypes = [C.c_void_p, C.c_void_p, C.c_size_t, C.c_int, C.c_void_p]
        sp = stream.cuda_stream
        nbytes = a.numel() * 4
        probe = {}
        for nb in (2048, 8192, 16384, 32768, 65536):
            assert pl.tpp_copy(a.data_ptr(), b.data_ptr(), nbytes, nb, sp) == 0
            sec = _time(lambda: pl.tpp_copy(a.data_ptr(), b.data_ptr(), nbytes, nb, sp),
                        args.iters, stream)
            probe[f"{nb}wg_GBs"] = 2 * nbytes / sec / 1e9
        out["copy_1GiB_probe"] = probe

    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
