"""Builds libphsa.so (the HIP kernels + C ABI) in-tree for gfx950.

    python -m paper_2601_02819_amd.build

Each ``csrc/*.hip`` file is compiled separately (in parallel) with hipcc and
linked into ``paper_2601_02819_amd/libphsa.so``, which exports only the C ABI
of ``include/phsa.h``.  The same objects plus ``csrc/prof/kernel_timing.hip``
make ``libphsa_prof.so``, the profiling build that records a pair of HIP
events around every kernel launch (``include/phsa_prof.h``).  Packed-fp32
instructions are disabled for device code; hipcc's host pass warns that it
does not know the feature, which is expected.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libphsa.so")
OUT_PROF = os.path.join(HERE, "libphsa_prof.so")
BUILD_DIR = os.path.join(ROOT, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

CFLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fvisibility=hidden", "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
    "-I", os.path.join(ROOT, "include"),
]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    cmd = [HIPCC, *CFLAGS, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{err}")
    if err.strip():
        sys.stderr.write(err + "\n")
    return obj


def _link(objs, out: str) -> None:
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, out)


def build(verbose: bool = True) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    prof_src = os.path.join(CSRC, "prof", "kernel_timing.hip")
    workers = min(len(srcs) + 1, max(1, (os.cpu_count() or 4)))
    with cf.ThreadPoolExecutor(workers) as ex:
        objs = list(ex.map(_compile, srcs + [prof_src]))
    prof_obj = objs.pop()
    _link(objs, OUT)
    _link(objs + [prof_obj], OUT_PROF)
    if verbose:
        print(f"built {OUT} from {len(srcs)} sources, and {OUT_PROF}")
    return OUT


if __name__ == "__main__":
    build()
