"""Host-side AddressSanitizer builds of the libraries, for CPU tests.

    python -m paper_2504_03664_amd.build_asan

libpipo_asan.so is libpipo.so with every host-side function instrumented
(the device code is compiled as usual and is not run by the CPU tests);
libpipo_sched_asan.so is the schedule library, instrumented.  Both are
linked without the sanitizer runtime: a process loads them after
preloading clang's shared ASan runtime (asan_runtime()), and the bindings
pick them up through PIPO_LIB / PIPO_SCHED_LIB.  tests/test_asan_cpu.py
runs the host-logic tests (schedule, configuration, packing, disk probe)
that way.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import sys

from .build import (ARCH, BUILD, CSRC, HIP_FLAGS, HIPCC, INCLUDE, PKG, SCHED_SOURCES, SOURCES,
                    _run)

ASAN_BUILD = BUILD + "_asan"
LIB = os.path.join(PKG, "libpipo_asan.so")
SCHED_LIB = os.path.join(PKG, "libpipo_sched_asan.so")
CLANG = os.path.join(os.path.dirname(os.path.realpath(HIPCC)), "..", "llvm", "bin", "clang++")
# host compilation only: each sanitizer flag applies to the host side
HOST_ASAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]


def asan_runtime() -> str:
    """clang's shared ASan runtime (to preload)."""
    hits = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    if not hits:
        raise FileNotFoundError("libclang_rt.asan-x86_64.so not found under /opt/rocm/llvm")
    return sorted(hits)[-1]


def _compile(src: str) -> str:
    obj = os.path.join(ASAN_BUILD, src + ".o")
    lang = ["-x", "hip"] if src.endswith(".cpp") else []
    _run([HIPCC, *lang, *HIP_FLAGS, *HOST_ASAN, "-c", os.path.join(CSRC, src), "-o", obj])
    return obj


def build_asan(jobs: int = 8) -> tuple:
    os.makedirs(ASAN_BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + f".tmp{os.getpid()}"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    tmp = SCHED_LIB + f".tmp{os.getpid()}"
    _run([CLANG, "-O1", "-g", "-std=c++17", "-fPIC", "-shared", *HOST_ASAN[1::2],
          "-I", INCLUDE, "-I", CSRC, "-o", tmp, *[os.path.join(CSRC, s) for s in SCHED_SOURCES]])
    os.replace(tmp, SCHED_LIB)
    return LIB, SCHED_LIB


if __name__ == "__main__":
    for p in build_asan():
        print(p)
    sys.exit(0)
