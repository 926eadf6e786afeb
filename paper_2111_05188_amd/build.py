"""Build libtp.so (the HIP library behind include/tp.h) for gfx950 only."""

from __future__ import annotations

import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libtp.so")
SOURCES = ["api.cpp", "rollout.hip", "rollout_rs.hip", "rollout_rs_i4.hip", "rollout_rs_i10.hip",
           "rollout_rs_i10_wide.hip", "critic.hip", "metrics.hip", "evolution.hip", "learner.hip",
           "env_kernels.hip", "gae.hip", "pack.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # no implicit fma contraction: the env step's rounding is spelled out
    "-ffp-contract=off",
    # packed fp32 instructions stay off (not trusted on this hardware)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-Wall",
]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    subprocess.check_call([HIPCC, "-x", "hip", *FLAGS, "-c",
                           os.path.join(CSRC, src), "-o", obj])
    return obj


PROBE_LIB = os.path.join(HERE, "libtpprobe.so")


def _link(objs, lib):
    tmp = lib + ".tmp"
    subprocess.check_call([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC",
                           "-o", tmp, *objs])
    os.replace(tmp, lib)


def build() -> str:
    """Compile every source and link libtp.so and the probe library
    libtpprobe.so (always rebuilds)."""
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(len(SOURCES) + 1) as ex:
        objs = list(ex.map(_compile, SOURCES + ["probe.hip"]))
    _link(objs[:-1], LIB)
    _link(objs[-1:], PROBE_LIB)
    return LIB


if __name__ == "__main__":
    print(build())
