"""The C ABI from plain C.

CPU: tests/abi_client.c is compiled as C99 with every warning an error
against include/rc_cohort.h, linked against the built library, and run; it
calls only the entry points that need no GPU and checks their results.

GPU (needs an MI355X): tests/abi_client_gpu.c drives the library with device
memory from hipMalloc -- no Python, no torch -- in every kernel form and
entry mode, and compares every output with the oracle's C entry point bit
for bit (see each file's header)."""
import os
import shutil
import subprocess
import sys

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


@pytest.mark.gpu
def test_c_client_on_the_gpu(tmp_path):
    import oracle
    gcc = shutil.which("gcc")
    if not gcc:
        pytest.skip("gcc is not available")
    if not os.path.exists(LIB):
        pytest.fail("librc_cohort.so is not built (run __graft_entry__.build())")
    orc_lib = oracle.build(force=False)
    exe = str(tmp_path / "abi_client_gpu")
    cmd = [gcc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-O1", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
           os.path.join(ROOT, "tests", "abi_client_gpu.c"), "-o", exe,
           "-L", PKG, "-lrc_cohort", "-L", os.path.dirname(orc_lib), "-lrc_oracle",
           "-L", ROCM_LIB, "-lamdhip64", "-lm",
           "-Wl,-rpath," + PKG, "-Wl,-rpath," + os.path.dirname(orc_lib), "-Wl,-rpath," + ROCM_LIB]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stdout + res.stderr
    print("C client on the GPU: four shapes, five entry modes each", flush=True)
    sys.stdout.flush()
    run = subprocess.run([exe], capture_output=True, text=True, timeout=100)
    assert run.returncode == 0, run.stdout + run.stderr
    assert run.stdout.strip().endswith("ok"), run.stdout
