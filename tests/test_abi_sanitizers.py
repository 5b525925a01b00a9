"""The host side of the C ABI (argument checks, size helpers over extreme and
invalid sizes, status strings) built with AddressSanitizer and
UndefinedBehaviorSanitizer on host code only, linked with the library's
kernel objects.  Every call in the driver is rejected (or empty) before any
launch, so this runs without a GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
MAIN = os.path.join(ROOT, "tests", "native", "abi_sanitize_main.cpp")
API = os.path.join(ROOT, "paper_2606_09508_amd", "csrc", "ei_api.hip")
NOALLOC = os.path.join(ROOT, "paper_2606_09508_amd", "csrc", "ei_noalloc.hip")
OBJS = [os.path.join(ROOT, "paper_2606_09508_amd", "_build", f"{n}.o")
        for n in ("ei_probe", "ei_select", "ei_attn")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"]


def test_abi_host_code_is_clean_under_asan_and_ubsan(tmp_path):
    if not (os.path.exists(HIPCC) or shutil.which("hipcc")):
        pytest.skip("hipcc is not available")
    if not all(os.path.exists(o) for o in OBJS):
        pytest.skip("the library's kernel objects are not built")
    common = ["-O1", "-g", "-std=c++17", "-I", os.path.join(ROOT, "include")]
    api_o, na_o, main_o, exe = (str(tmp_path / n)
                                for n in ("api.o", "noalloc.o", "main.o", "abi_sanitized"))
    host = [HIPCC, "--offload-arch=gfx950", *common, "-fPIC", "-Xclang", "-target-feature",
            "-Xclang", "-packed-fp32-ops", *SAN, "-Xarch_host", "-fno-sanitize-recover=all"]
    steps = [
        [*host, "-c", API, "-o", api_o],
        [*host, "-c", NOALLOC, "-o", na_o],
        [HIPCC, *common, *SAN, "-Xarch_host", "-fno-sanitize-recover=all", "-x", "c++", "-c",
         MAIN, "-o", main_o],
        [HIPCC, "--offload-arch=gfx950", *SAN, main_o, api_o, na_o, *OBJS, "-o", exe],
    ]
    for cmd in steps:
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert run.returncode == 0, run.stdout + run.stderr[-3000:]
    assert "abi sanitized run: ok" in run.stdout
