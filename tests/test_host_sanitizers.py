"""The library's host code (DualRadixTree, decode plan, C-ABI checks) built with AddressSanitizer
and UndefinedBehaviorSanitizer and driven by tests/sanitize_host.cpp (random tree operations,
plans for every head layout, rank and RoPE setting, table validation, error paths).  Host
sources only: the GPU code is not part of this build."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2604_06370_amd", "csrc")
HOST_SOURCES = ["tree.cpp", "plan.cpp", "capi.cpp"]


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_code_is_clean_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "sanitize_host")
    srcs = [os.path.join(ROOT, "tests", "sanitize_host.cpp")] + [os.path.join(CSRC, s) for s in HOST_SOURCES]
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-o", exe] + srcs
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert "sanitized host run: ok" in r.stdout
