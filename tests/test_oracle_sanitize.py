"""The CPU oracle under AddressSanitizer and UndefinedBehaviorSanitizer.

tests/sanitize_oracle.c calls every oracle entry point (screening, merge,
positions, the maps and the generator, the rung statistics and the
promotion decision, the derived inputs) on special values, empty and ragged sizes and random
inputs, with every buffer allocated at its exact size; built here with both
sanitizers and no recovery, any out-of-bounds access, use of freed memory,
signed overflow or invalid shift ends the run with a report."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_clean_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "sanitize_oracle")
    srcs = [os.path.join(ROOT, "tests", "sanitize_oracle.c"), os.path.join(ROOT, "oracle", "kbo.c"),
            os.path.join(ROOT, "oracle", "kbo_rung.c"), os.path.join(ROOT, "oracle", "kbo_derived.c")]
    cmd = ["gcc", "-std=c11", "-O1", "-g", "-ffp-contract=off", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "oracle"),
           *srcs, "-o", exe, "-lm"]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    res = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert res.returncode == 0, res.stderr[-4000:]
    assert res.stdout.strip() == "ok", res.stdout
