"""The oracle and the library's host-side code under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only).

Each test builds an instrumented copy in a temporary directory and runs the
existing CPU tests against it in a child process with the sanitizer runtime
preloaded (the Python interpreter itself is not instrumented):

  * the oracle (plain C, gcc) under its oracle pins;
  * libga.so with its host code instrumented (hipcc; the device code is built
    as usual) under the C-ABI argument checks, which exercise every host-side
    validation path and the workspace layouts.

A canary library with a planted heap overflow and a planted signed overflow,
built and loaded the same way, shows that each setup reports errors.
"""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2306_01926_amd", "csrc")

CANARY = r"""
#include <stdlib.h>
int canary_heap(int n, int i) { int *p = (int *)malloc(n * sizeof(int)); p[0] = 1; int v = p[i]; free(p); return v; }
int canary_overflow(int x) { return x + 1; }
"""


def _child(env_extra, code=None, pytest_args=None, timeout=900):
    env = dict(os.environ, **env_extra)
    env.pop("PYTEST_ADDOPTS", None)
    if pytest_args is not None:
        cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", *pytest_args]
    else:
        cmd = [sys.executable, "-c", code]
    return subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=timeout)


def _canary_checks(build, env):
    """The canary built by `build(src, out)` must make the child fail with the
    sanitizer's report: a heap overflow, then a signed overflow."""
    heap = _child(env, "import ctypes; L = ctypes.CDLL(%r); L.canary_heap(4, 9)" % build)
    assert heap.returncode != 0 and "heap-buffer-overflow" in heap.stderr, heap.stderr[-2000:]
    ovf = _child(env, "import ctypes; L = ctypes.CDLL(%r); L.canary_overflow(2147483647)" % build)
    assert ovf.returncode != 0 and "signed integer overflow" in ovf.stderr, ovf.stderr[-2000:]


def test_oracle_pins_under_asan_ubsan(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not found")
    runtime = subprocess.run([gcc, "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(runtime) or not os.path.exists(runtime):
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    flags = ["-O1", "-g", "-fPIC", "-shared", "-fno-omit-frame-pointer",
             "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined"]
    env = {"LD_PRELOAD": runtime, "ASAN_OPTIONS": "detect_leaks=0", "UBSAN_OPTIONS": "print_stacktrace=1"}
    canary_src, canary = tmp_path / "canary.c", str(tmp_path / "libcanary.so")
    canary_src.write_text(CANARY)
    subprocess.run([gcc, *flags, "-o", canary, str(canary_src)], check=True)
    _canary_checks(canary, env)
    lib = str(tmp_path / "libga_oracle_san.so")
    subprocess.run([gcc, *flags, "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-o", lib,
                    os.path.join(ROOT, "oracle", "ga_oracle.c"), "-lm"], check=True)
    r = _child(dict(env, GA_ORACLE_LIB=lib), pytest_args=["-m", "not gpu", "tests/test_oracle_pins.py"])
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert "passed" in r.stdout and "Sanitizer" not in r.stderr


def test_host_checks_under_asan_ubsan(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    runtimes = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not os.path.exists(hipcc) or not runtimes:
        pytest.skip("hipcc or clang's AddressSanitizer runtime not found")
    # the sanitizers instrument the host code only (each -fsanitize behind -Xarch_host)
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
           "-shared-libasan"]
    env = {"LD_PRELOAD": runtimes[-1], "ASAN_OPTIONS": "detect_leaks=0", "UBSAN_OPTIONS": "print_stacktrace=1"}
    canary_src, canary = tmp_path / "canary.cpp", str(tmp_path / "libcanary.so")
    canary_src.write_text('extern "C" {\n' + CANARY + "}\n")
    subprocess.run([hipcc, "-O1", "-g", "-fPIC", "-shared", *san, "-o", canary, str(canary_src)], check=True,
                   capture_output=True)
    _canary_checks(canary, env)
    sys.path.insert(0, os.path.join(ROOT, "paper_2306_01926_amd"))
    from build import SOURCES  # the library's sources, the same list the product build compiles

    lib = str(tmp_path / "libga_san.so")
    r = subprocess.run([hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-shared",
                        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *san,
                        "-I", os.path.join(ROOT, "include"), *SOURCES, "-o", lib], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    r = _child(dict(env, GA_LIB=lib), pytest_args=["-m", "not gpu", "tests/test_abi_cpu.py"])
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert "passed" in r.stdout and "Sanitizer" not in r.stderr
