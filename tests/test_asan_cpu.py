"""The host-side logic of the libraries under AddressSanitizer, on the CPU:
the schedule (Algorithm 1 as stream operations), the configuration and
memory plan (Eq. (1)), the weight packers and the disk probe, run by their
CPU tests against libpipo_asan.so / libpipo_sched_asan.so
(paper_2504_03664_amd/build_asan.py) with clang's ASan runtime preloaded.
Any report of the sanitizer fails the run."""
import os
import subprocess
import sys

import pytest

from paper_2504_03664_amd import build_asan

pytestmark = pytest.mark.asan

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2504_03664_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
HOST_TESTS = ["tests/test_schedule_cpu.py", "tests/test_configure_cpu.py",
              "tests/test_abi_cpu.py"]


def _stale(lib):
    if not os.path.exists(lib):
        return True
    t = os.path.getmtime(lib)
    srcs = [os.path.join(d, f) for d in (CSRC, INCLUDE) for f in os.listdir(d)]
    return any(os.path.getmtime(s) > t for s in srcs)


@pytest.fixture(scope="module")
def asan_libs():
    if _stale(build_asan.LIB) or _stale(build_asan.SCHED_LIB):
        build_asan.build_asan()
    return build_asan.LIB, build_asan.SCHED_LIB


def test_libraries_are_instrumented(asan_libs):
    for lib in asan_libs:
        out = subprocess.run(["nm", "-D", lib], stdout=subprocess.PIPE, text=True,
                             check=True).stdout
        assert "__asan_report_load" in out and "__asan_report_store" in out, lib


def test_host_logic_clean_under_asan(asan_libs):
    lib, sched = asan_libs
    env = dict(os.environ, LD_PRELOAD=build_asan.asan_runtime(), PIPO_LIB=lib,
               PIPO_SCHED_LIB=sched,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0:exitcode=86")
    probe = ("import ctypes, sys; from paper_2504_03664_amd import binding as B; "
             "B.lib(); B.sched_lib(); maps = open('/proc/self/maps').read(); "
             "assert 'libclang_rt.asan' in maps and B.LIB_PATH in maps "
             "and B.SCHED_LIB_PATH in maps, 'ASan builds not loaded'")
    r = subprocess.run([sys.executable, "-c", probe], cwd=ROOT, env=env,
                       stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert r.returncode == 0, r.stdout[-3000:]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        "-m", "not gpu", *HOST_TESTS], cwd=ROOT, env=env,
                       stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert "AddressSanitizer" not in r.stdout, r.stdout[-5000:]
    assert r.returncode == 0, r.stdout[-3000:]
