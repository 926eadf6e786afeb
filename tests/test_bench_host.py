"""Host-side logic of bench.py (no GPU): the single-GPU refusal, the per
env-step work figures the roofline divides by, the counter lookup's source
gate and the oracle samples (all cores, one thread, fp32 actor)."""

import json
import os
import subprocess
import sys

import numpy as np

import bench
import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_work_per_env_step_at_the_100_stock_minute_shape():
    cfg = W.get_config("nasdaq100")
    # market row n(1+I)*4, bf16 observation 2S, action 4n, logp, reward, done
    assert bench.algorithmic_bytes_rollout(cfg) == 4 * 100 * 9 + 2 * 1001 + 4 * 100 + 9
    # reward, value, done in; advantage, return out
    assert bench.algorithmic_bytes_gae() == 17
    assert bench.algorithmic_bytes_rollout(cfg) + bench.algorithmic_bytes_gae() == 6028
    # 2 * sum(in * out) over the 1001-512-512-100 actor
    assert cfg.flops_per_env_step() == 2 * (1001 * 512 + 512 * 512 + 512 * 100) == 1651712


def test_counter_traffic_is_gated_by_the_kernel_sources():
    text = open(os.path.join(ROOT, "profiles", "hbm_counters.md")).read()
    data = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
    key = "rollout_rs_kernel nasdaq100"
    got = bench.counter_traffic(key)
    if data["source_sha256"] == bench.kernel_source_hash():
        assert got == data["kernels"][key]["traffic_bytes"] and got > 0
    else:
        assert got is None
    # other kernels' counters are not the rollout kernel's traffic
    assert bench.counter_traffic("gae_kernel nasdaq100") is None
    assert bench.counter_traffic("no_such_kernel x") is None


def test_oracle_samples_name_the_host_and_the_threads():
    import oracle
    cfg = W.get_config("tiny")
    mk, t0, params = W.make_market(cfg), W.make_t0(cfg), W.make_actor(cfg)
    r = bench.cpu_baseline(cfg, mk, params, t0, 24, all_core_envs=40)
    assert r["kind"] == "oracle" and r["unit"] == "env-steps/s"
    assert r["cores"] == oracle.threads(True) >= 1
    assert r["value"] > 0 and np.isfinite(r["value"]) and r["seconds"] > 0
    assert r["cpu_model"] and r["host_cpus"] >= 1
    assert "40 envs" in r["sample"] and "OpenMP" in r["sample"]
    one = r["single_thread"]
    assert one["cores"] == 1 and one["value"] > 0 and "24 envs" in one["sample"]
    f32 = r["single_thread_fp32_actor"]
    assert f32["cores"] == 1 and f32["value"] > 0 and "12 envs" in f32["sample"]
