"""Sanitizer runs of the host code (CPU only): the C oracle and the C-ABI
layer's host-side argument checks, built with AddressSanitizer and
UndefinedBehaviorSanitizer and exercised by the existing CPU tests in a
subprocess that preloads the sanitizer runtime.

- oracle.c: gcc -fsanitize=address,undefined, loaded through ORACLE_LIB by
  the oracle pin tests (env step, GAE, metrics, evolution, actor).
- api.cpp: the host pass only (hipcc -Xarch_host -fsanitize=...), linked
  with the library's other objects, loaded through TP_LIB_PATH by the ABI
  contract tests (argument checks, registry, start-row check).
A planted heap overflow in a scratch C file shows that the harness reports
what it should."""

import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2111_05188_amd", "csrc")
BUILD = os.path.join(ROOT, "_build")

GCC_SAN = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined"]


def _gcc_runtime():
    libs = [subprocess.check_output(["gcc", f"-print-file-name={n}"]).decode().strip()
            for n in ("libasan.so", "libubsan.so")]
    return ":".join(libs)


def _env(**kw):
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=0"   # the interpreter itself is not instrumented
    env["UBSAN_OPTIONS"] = "print_stacktrace=1"
    env.update(kw)
    return env


@pytest.mark.parametrize("body,call,report", [
    ("#include <stdlib.h>\nint poke(int i) { int *p = malloc(4 * sizeof(int));"
     " p[i] = 1; int v = p[0]; free(p); return v; }\n", "poke(4)", "heap-buffer-overflow"),
    ("int bump(int x) { return x + 1; }\n", "bump(2147483647)", "signed integer overflow")])
def test_the_harness_reports_a_planted_mistake(tmp_path, body, call, report):
    src = tmp_path / "bad.c"
    src.write_text(body)
    lib = tmp_path / "libbad.so"
    subprocess.check_call(["gcc", *GCC_SAN, "-fno-sanitize=object-size", "-fPIC", "-shared",
                           "-o", str(lib), str(src)])
    code = f"import ctypes; ctypes.CDLL({str(lib)!r}).{call}"
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=120,
                       env=_env(LD_PRELOAD=_gcc_runtime()))
    assert r.returncode != 0 and report in r.stderr, r.stderr[-2000:]


def test_oracle_pins_under_address_and_ub_sanitizers(tmp_path):
    lib = tmp_path / "liboracle_san.so"
    subprocess.check_call(["gcc", *GCC_SAN, "-std=c11", "-ffp-contract=off", "-fno-fast-math",
                           "-fPIC", "-shared", "-Wno-unknown-pragmas", "-o", str(lib),
                           os.path.join(ROOT, "oracle", "oracle.c"), "-lm"])
    files = [os.path.join(ROOT, "tests", f) for f in
             ("test_oracle_env.py", "test_oracle_gae.py", "test_oracle_metrics.py",
              "test_oracle_evolution.py", "test_oracle_actor.py")]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        "-k", "not openmp", *files], capture_output=True, text=True,
                       timeout=900, cwd=ROOT,
                       env=_env(LD_PRELOAD=_gcc_runtime(), ORACLE_LIB=str(lib)))
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "passed" in r.stdout


def _clang_asan_runtime():
    hits = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    if not hits:
        pytest.skip("clang's ASan runtime is not installed")
    return hits[0]


def test_abi_host_checks_under_address_and_ub_sanitizers(tmp_path):
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    objs = [o for o in glob.glob(os.path.join(BUILD, "*.o"))
            if os.path.basename(o) not in ("api.o", "probe.o")]
    if len(objs) < 9:
        from paper_2111_05188_amd import build as hip_build
        hip_build.build()
        objs = [o for o in glob.glob(os.path.join(BUILD, "*.o"))
                if os.path.basename(o) not in ("api.o", "probe.o")]
    host_san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-omit-frame-pointer", "-shared-libsan"]
    api = tmp_path / "api_san.o"
    subprocess.check_call([hipcc, "-x", "hip", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
                           "-fPIC", "-ffp-contract=off", *host_san, "-I",
                           os.path.join(ROOT, "include"), "-I", CSRC, "-c",
                           os.path.join(CSRC, "api.cpp"), "-o", str(api)],
                          stderr=subprocess.DEVNULL)
    lib = tmp_path / "libtp_san.so"
    subprocess.check_call([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", *host_san,
                           "-o", str(lib), str(api), *objs], stderr=subprocess.DEVNULL)
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_cpu.py")], capture_output=True,
                       text=True, timeout=600, cwd=ROOT,
                       env=_env(LD_PRELOAD=_clang_asan_runtime(), TP_LIB_PATH=str(lib)))
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "passed" in r.stdout
