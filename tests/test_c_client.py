"""The interface from plain C.

tests/c_api/host_calls.c (CPU) includes include/kb.h as C11 with every
warning an error, links libkb.so, and makes the calls that need no GPU: the
policy gate, the verdicts of host records, the rung survival table, the
workspace size, an argument error and its text, the version.

tests/c_api/screen_from_c.c (GPU) runs the screening path from C with no
Python and no torch: hipMalloc'd buffers, a seeded reference from
kb_gen_inputs, three candidates with exact expectations by construction,
kb_screen, kb_screen_stats and kb_screen_locate."""
import os
import shutil
import subprocess

import pytest

from tests.helpers import ensure_built

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2608_02611_amd")
ROCM_INCLUDE = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "include")


ROCM_LIB = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "lib")


def build_and_run(tmp_path, name, hip_runtime=False):
    gcc = shutil.which("gcc")
    if gcc is None or not os.path.isdir(ROCM_INCLUDE):
        pytest.skip("needs gcc and the ROCm headers")
    ensure_built()
    exe = str(tmp_path / name)
    # (HIP's runtime header needs the platform named when a plain C compiler
    # reads it)
    cmd = [gcc, "-std=c11", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", ROCM_INCLUDE,
           os.path.join(ROOT, "tests", "c_api", name + ".c"), "-o", exe,
           "-L", PKG, "-lkb", "-Wl,-rpath," + PKG]
    if hip_runtime:
        cmd += ["-L", ROCM_LIB, "-lamdhip64", "-Wl,-rpath," + ROCM_LIB]
    subprocess.run(cmd + ["-lm"], check=True)
    print("running", name, flush=True)
    out = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    print(out.stdout, flush=True)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.strip().endswith("PASSED"), out.stdout


def test_c_client(tmp_path):
    build_and_run(tmp_path, "host_calls")


@pytest.mark.gpu
def test_c_client_screens_on_the_gpu(tmp_path):
    build_and_run(tmp_path, "screen_from_c", hip_runtime=True)
