"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer.

The generator, the planner's tables and the MINIROCKET fit (plain C++ with no
HIP code) are built with g++ -fsanitize=address,undefined into a host-only
library, and the oracle's C library with gcc and the same sanitizers.  The
CPU tests that exercise them then run again in a child process with those
builds loaded in place of the regular ones and the sanitizer runtimes
preloaded: an out-of-bounds access, a use after free, an integer overflow or
any other undefined behaviour aborts the child and fails this test.  The
child also forces the generator's allocation failure (ROCKET_ERR_OOM), which
the sanitizer's allocator reports by returning NULL."""
import os
import shutil
import subprocess
import sys

import pytest

pytestmark = pytest.mark.sanitize

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2601_17091_amd", "csrc")
HOST_SOURCES = [os.path.join(CSRC, f) for f in ("generate.cpp", "plan.cpp", "minirocket.cpp")]
ORACLE_SOURCES = [os.path.join(ROOT, "oracle", f) for f in ("rocket_oracle.c", "minirocket_oracle.c")]
HOST_TESTS = ["tests/test_plan_host.py", "tests/test_oracle_examples.py", "tests/test_oracle_generator.py",
              "tests/test_oracle_invariants.py", "tests/test_oracle_multivariate.py",
              "tests/test_oracle_minirocket.py", "tests/test_abi.py"]
# tests of test_abi.py that load the full HIP library (exports, plan and
# transform entry points) stay with the regular build
NEEDS_FULL_LIBRARY = ["test_header_declares", "test_library_exports", "test_plan_validation",
                      "test_transform_validation", "test_minirocket_plan_rejects",
                      "test_product_build_is_unchecked", "test_checked_build_exports"]
SAN_FLAGS = ["-O1", "-g", "-fPIC", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=undefined"]


def _runtime(cc, name):
    path = subprocess.run([cc, "-print-file-name=" + name], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_host_code_under_sanitizers(tmp_path):
    gxx, gcc = shutil.which("g++"), shutil.which("gcc")
    if not gxx or not gcc:
        pytest.skip("g++ and gcc are needed for the sanitized builds")
    asan, ubsan = _runtime(gcc, "libasan.so"), _runtime(gcc, "libubsan.so")
    if not asan or not ubsan:
        pytest.skip("the compiler's sanitizer runtimes are not installed")
    host = str(tmp_path / "librocket_host_san.so")
    subprocess.run([gxx, "-std=c++17", "-shared"] + SAN_FLAGS
                   + ["-I", os.path.join(ROOT, "include"), "-I", CSRC] + HOST_SOURCES + ["-o", host], check=True)
    orc = str(tmp_path / "librocket_oracle_san.so")
    subprocess.run([gcc, "-std=c11", "-shared", "-fopenmp", "-ffp-contract=off", "-fno-fast-math"] + SAN_FLAGS
                   + ORACLE_SOURCES + ["-lm", "-o", orc], check=True)
    env = dict(os.environ,
               LD_PRELOAD=asan + ":" + ubsan,
               ASAN_OPTIONS="detect_leaks=0:allocator_may_return_null=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
               ROCKET_TEST_HOST_LIB=host, ROCKET_TEST_ORACLE_LIB=orc, OMP_NUM_THREADS="4")
    kexpr = "not (" + " or ".join(NEEDS_FULL_LIBRARY) + ")"
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-s", "-p", "no:cacheprovider", "-m", "not gpu and not sanitize",
           "-k", kexpr] + HOST_TESTS
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=1200)
    tail = (r.stdout[-6000:] + "\n" + r.stderr[-6000:])
    assert r.returncode == 0, tail
    assert " passed" in r.stdout, tail
    # the child ran against the sanitized builds
    assert "[sanitized builds] host=%s oracle=%s" % (host, orc) in r.stdout, tail
    print(r.stdout.strip().splitlines()[-1])
