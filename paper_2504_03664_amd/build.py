"""Build the gfx950 shared library (libpipo.so) and the CPU-only schedule
library (libpipo_sched.so) in-tree.

    python -m paper_2504_03664_amd.build

Every HIP source is compiled with hipcc for gfx950 only, with packed fp32
instructions disabled; objects go to ``_build/`` and the libraries next to
this file.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libpipo.so")
SCHED_LIB = os.path.join(PKG, "libpipo_sched.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-I", INCLUDE, "-I", CSRC,
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-Wall",
             "-Wno-unused-result"]
SOURCES = ["gemm.hip", "attention.hip", "kvcache.hip", "elementwise.hip", "engine.cpp", "config.cpp", "pack.cpp", "ops_api.cpp",
           "schedule.cpp", "sched_capi.cpp"]
SCHED_SOURCES = ["schedule.cpp", "sched_capi.cpp"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines()
                    if "packed-fp32-ops" not in l and l.strip())
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, src + ".o")
    cmd = [HIPCC, *HIP_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd = [HIPCC, "-x", "hip", *HIP_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    _run(cmd)
    return obj


def build_gpu(jobs: int = 8) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + f".tmp{os.getpid()}"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    return LIB


def build_sched_cpu() -> str:
    tmp = SCHED_LIB + f".tmp{os.getpid()}"
    _run(["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-Wall", "-I", INCLUDE, "-I", CSRC,
          "-o", tmp, *[os.path.join(CSRC, s) for s in SCHED_SOURCES]])
    os.replace(tmp, SCHED_LIB)
    return SCHED_LIB


def build_all() -> None:
    build_sched_cpu()
    build_gpu()


if __name__ == "__main__":
    build_all()
    print(LIB)
    print(SCHED_LIB)
    sys.exit(0)
