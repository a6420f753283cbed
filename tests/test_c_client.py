"""The interface from plain C (CPU only).

tests/c_api/host_calls.c includes include/kb.h as C11 with every warning an
error, links libkb.so, and makes the calls that need no GPU: the policy gate,
the verdicts of host records, the rung survival table, the workspace size,
an argument error and its text, the version."""
import os
import shutil
import subprocess

import pytest

from tests.helpers import ensure_built

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2608_02611_amd")
ROCM_INCLUDE = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "include")


def test_c_client(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None or not os.path.isdir(ROCM_INCLUDE):
        pytest.skip("needs gcc and the ROCm headers")
    ensure_built()
    exe = str(tmp_path / "host_calls")
    # (HIP's runtime header needs the platform named when a plain C compiler
    # reads it)
    cmd = [gcc, "-std=c11", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", ROCM_INCLUDE,
           os.path.join(ROOT, "tests", "c_api", "host_calls.c"), "-o", exe,
           "-L", PKG, "-lkb", "-Wl,-rpath," + PKG, "-lm"]
    subprocess.run(cmd, check=True)
    out = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.strip().endswith("PASSED"), out.stdout
