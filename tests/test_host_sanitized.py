"""The host-only C++ of the library (descriptor checks, launch plan, cohort
former, online compactor, cohort feed: csrc/rc_host.cpp and csrc/rc_pack.cpp)
built with AddressSanitizer and UndefinedBehaviorSanitizer, and the CPU tests
of those entry points run against that build in a child process.  Any
sanitizer report aborts the child, which fails this test.  CPU only."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_12123_amd", "csrc")
SOURCES = [os.path.join(CSRC, "rc_host.cpp"), os.path.join(CSRC, "rc_pack.cpp")]
# the CPU tests that reach only host-side entry points
TESTS = ["tests/test_plan.py", "tests/test_pack_native.py", "tests/test_online_native.py",
         "tests/test_abi.py::test_status_strings",
         "tests/test_abi.py::test_invalid_descriptor_rejected_by_plan_inspection"]


def _runtime(name):
    gcc = shutil.which("gcc")
    if not gcc:
        return None
    p = subprocess.run([gcc, "-print-file-name=" + name], capture_output=True, text=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else None


@pytest.fixture(scope="module")
def sanitized_lib(tmp_path_factory):
    gxx = shutil.which("g++")
    if not gxx or not _runtime("libasan.so"):
        pytest.skip("g++ with the ASan runtime is not available")
    out = str(tmp_path_factory.mktemp("asan") / "librc_host_asan.so")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fPIC", "-shared",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-Wall", "-Wextra",
           "-I", os.path.join(ROOT, "include"), "-o", out] + SOURCES
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stdout + res.stderr
    return out


def test_host_code_under_asan_and_ubsan(sanitized_lib):
    env = dict(os.environ)
    env["RC_COHORT_LIB"] = sanitized_lib
    # the ASan runtime first, anything already preloaded kept after it
    prev = env.get("LD_PRELOAD", "")
    env["LD_PRELOAD"] = _runtime("libasan.so") + (":" + prev if prev else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:verify_asan_link_order=0"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu"] + TESTS
    res = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (res.stdout + res.stderr)[-4000:]
    assert res.returncode == 0, tail
    assert "passed" in res.stdout, tail
    assert "ERROR: AddressSanitizer" not in res.stderr and "runtime error:" not in res.stderr, tail
