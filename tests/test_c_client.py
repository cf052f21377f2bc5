"""The C ABI from plain C (CPU only): tests/abi_client.c is compiled as C99
with every warning an error against include/rc_cohort.h, linked against the
built library, and run; it calls only the entry points that need no GPU and
checks their results (see the file's header)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2608_12123_amd")
LIB = os.path.join(PKG, "librc_cohort.so")
ROCM_LIB = "/opt/rocm/lib"


def test_c_client(tmp_path):
    gcc = shutil.which("gcc")
    if not gcc:
        pytest.skip("gcc is not available")
    if not os.path.exists(LIB):
        pytest.fail("librc_cohort.so is not built (run __graft_entry__.build())")
    exe = str(tmp_path / "abi_client")
    cmd = [gcc, "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", "-O1",
           "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "abi_client.c"),
           "-o", exe, "-L", PKG, "-lrc_cohort", "-Wl,-rpath," + PKG,
           "-Wl,-rpath-link," + ROCM_LIB]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stdout + res.stderr
    run = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, run.stdout + run.stderr
    assert run.stdout.strip().endswith("ok"), run.stdout
