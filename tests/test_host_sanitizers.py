"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

1. The C ABI layer (csrc/api.hip: validation, workspace sizing and layout,
   dispatch) is compiled for the host alone with both sanitizers, linked with
   stand-in launchers that report a failed launch, and driven over the
   workloads' configurations and 20000 random and extreme parameter sets
   (tests/sanitize/abi_host_driver.cpp).
2. The oracle is compiled with both sanitizers and the oracle's own tests
   (tests/test_oracle_*.py) run against that build in a child process.

Any sanitizer report aborts the child and fails the test."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OUT = os.path.join(ROOT, "_build", "sanitize")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/llvm/bin/clang++"
# hipcc: each sanitizer flag applies to the host compilation only
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]


def run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout[-4000:]}\n{r.stderr[-4000:]}"
    return r


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)), reason="ROCm compilers not installed")
def test_abi_host_code_under_sanitizers():
    os.makedirs(OUT, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include")]
    host_only = [HIPCC, "-O1", "-g", "-std=c++17", "-x", "hip", "--offload-host-only", *HOST_SAN, *inc, "-c"]
    api = os.path.join(OUT, "api.o")
    stubs = os.path.join(OUT, "launch_stubs.o")
    drv = os.path.join(OUT, "abi_host_driver.o")
    exe = os.path.join(OUT, "abi_host_driver")
    run(host_only + [os.path.join(ROOT, "paper_2601_02819_amd", "csrc", "api.hip"), "-o", api])
    run(host_only + [os.path.join(ROOT, "tests", "sanitize", "launch_stubs.cpp"), "-o", stubs])
    run([CLANG, "-O1", "-g", "-std=c++17", *SAN, *inc, "-c",
         os.path.join(ROOT, "tests", "sanitize", "abi_host_driver.cpp"), "-o", drv])
    run([CLANG, *SAN, api, stubs, drv, "-o", exe])
    r = run([exe], env={**os.environ, "ASAN_OPTIONS": "detect_leaks=1:abort_on_error=1",
                        "UBSAN_OPTIONS": "print_stacktrace=1"})
    assert " 0 failed" in r.stdout, r.stdout


def test_oracle_under_sanitizers():
    libasan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(libasan):
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    os.makedirs(OUT, exist_ok=True)
    lib = os.path.join(OUT, "libphsa_oracle_san.so")
    run(["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-fPIC", "-shared", *SAN,
         os.path.join(ROOT, "oracle", "phsa_oracle.c"), "-o", lib, "-lm"])
    tests = sorted(glob.glob(os.path.join(ROOT, "tests", "test_oracle_*.py")))
    pre = os.environ.get("LD_PRELOAD", "")
    env = {**os.environ, "PHSA_ORACLE_LIB": lib,
           # the runtime must come first; anything already preloaded stays
           "LD_PRELOAD": libasan + (":" + pre if pre else ""),
           "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1", "UBSAN_OPTIONS": "print_stacktrace=1",
           "OMP_NUM_THREADS": "4"}
    r = run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu", "-p", "no:cacheprovider", *tests],
            env=env, cwd=ROOT)
    assert " passed" in r.stdout and "failed" not in r.stdout, r.stdout[-2000:]
