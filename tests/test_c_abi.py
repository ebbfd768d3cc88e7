"""The C ABI from a plain C99 caller: tests/c_abi/abi_check.c, compiled with gcc against
include/pace.h alone and linked to libpace.so, runs the host-only helpers and the argument
checks that return before any launch (no GPU needed)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_c_caller(tmp_path):
    gcc = shutil.which("gcc")
    rocm_inc = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "include")
    if gcc is None or not os.path.isdir(rocm_inc):
        pytest.skip("gcc or the ROCm headers are not available")
    from paper_2608_27206_amd import pace
    lib = pace.LIB_PATH
    assert os.path.exists(lib), "build the library first (python -m paper_2608_27206_amd.build)"
    exe = str(tmp_path / "abi_check")
    cmd = [gcc, "-std=c99", "-Wall", "-Wextra", "-Werror=implicit-function-declaration", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", rocm_inc, os.path.join(ROOT, "tests", "c_abi", "abi_check.c"),
           "-o", exe, lib, "-lm", "-Wl,-rpath," + os.path.dirname(lib)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    run = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert run.returncode == 0 and "c abi ok" in run.stdout, run.stdout + run.stderr
