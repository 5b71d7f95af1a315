"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

A copy of libkara.so is built with the host side of every source sanitized
(paper_2607_01237_amd/build_sanitized.py; the gfx950 code is unchanged), and
the CPU tests that drive host code -- the scheduler runtime (test_sched.py)
and the C ABI's exports and argument checks (test_abi_cpu.py) -- run against
it in a child process that loads clang's shared ASan runtime first.  Any
memory error or undefined behaviour aborts that process, and the test fails.
"""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_host_code_under_asan_and_ubsan():
    from paper_2607_01237_amd import build_sanitized
    lib = build_sanitized.build()
    env = dict(os.environ, KARA_LIBRARY=lib, LD_PRELOAD=build_sanitized.runtime(),
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    probe = ("import ctypes; from paper_2607_01237_amd import kara; l = kara.load(); "
             "assert l._name == kara.LIB_PATH and kara.LIB_PATH.endswith('libkara_san.so'); "
             "ctypes.CDLL(None).__asan_report_load1; print('sanitized library loaded')")
    r = subprocess.run([sys.executable, "-c", probe], env=env, cwd=ROOT, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and "sanitized library loaded" in r.stdout, r.stdout[-2000:] + r.stderr[-4000:]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
                        "tests/test_sched.py", "tests/test_abi_cpu.py"],
                       env=env, cwd=ROOT, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-6000:]
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-6000:]
    assert " passed" in r.stdout
