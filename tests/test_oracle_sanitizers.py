"""The CPU oracle under AddressSanitizer and UndefinedBehaviorSanitizer: a
small ragged problem through every entry point (probe, the three selection
modes, both budget recurrences, sparse and dense attention).  Any
out-of-bounds access, leak or undefined operation aborts the program."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
MAIN = os.path.join(ROOT, "tests", "native", "oracle_sanitize_main.c")


def test_oracle_is_clean_under_asan_and_ubsan(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc is not available")
    exe = str(tmp_path / "oracle_sanitized")
    build = subprocess.run(
        [gcc, "-O1", "-g", "-std=c11", "-fopenmp", "-ffp-contract=off",
         "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
         MAIN, "-o", exe, "-lm"], capture_output=True, text=True)
    if build.returncode != 0 and "sanitize" in build.stderr:
        pytest.skip("gcc here has no sanitizer runtimes")
    assert build.returncode == 0, build.stderr
    env = dict(os.environ, OMP_NUM_THREADS="2")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "oracle sanitized run: ok" in run.stdout
