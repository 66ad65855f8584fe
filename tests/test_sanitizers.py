"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

* The oracle: oracle/oracle.c and the driver tests/sanitize/oracle_main.c,
  which calls every entry point on small inputs (both layouts, all
  precisions, k = 1 / 3 / 5, residual networks), built with gcc
  -fsanitize=address,undefined and leak checks; any finding aborts it.
* The library's host side (argument checks, planning, the C ABI): the
  host-only tests run against libpredecoder_san.so (`python
  paper_2604_12841_amd/build.py --sanitize`, a build of a few minutes, so
  this part is skipped unless that library exists) with the sanitizer
  runtime preloaded and PD_LIBRARY pointing at it.
"""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_oracle_under_asan_and_ubsan(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("no gcc")
    exe = str(tmp_path / "oracle_san")
    cmd = ["gcc", "-O1", "-g", "-fopenmp", "-std=c11", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
           os.path.join(ROOT, "oracle", "oracle.c"), os.path.join(ROOT, "tests", "sanitize", "oracle_main.c"),
           "-o", exe, "-lm"]
    subprocess.check_call(cmd)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", OMP_NUM_THREADS="2")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr


def test_library_host_side_under_asan_and_ubsan():
    lib = os.path.join(ROOT, "paper_2604_12841_amd", "libpredecoder_san.so")
    if not os.path.exists(lib):
        pytest.skip("libpredecoder_san.so not built (python paper_2604_12841_amd/build.py --sanitize)")
    rt = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    if not rt:
        pytest.skip("no clang AddressSanitizer runtime")
    env = dict(os.environ, LD_PRELOAD=rt[0], ASAN_OPTIONS="detect_leaks=0", PD_LIBRARY=lib,
               UBSAN_OPTIONS="print_stacktrace=1")
    tests = [os.path.join(ROOT, "tests", t) for t in ("test_abi_host.py", "test_stream_host.py",
                                                      "test_binding_checks.py")]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu"] + tests,
                       capture_output=True, text=True, env=env, cwd=ROOT, timeout=900)
    assert r.returncode == 0, r.stdout[-4000:] + r.stderr[-4000:]
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, r.stderr[-4000:]
