"""The library's host-side planning code (packed-weight and workspace
layouts, GEMM launch plans, sizing) built with g++ under AddressSanitizer and
UndefinedBehaviorSanitizer and run over every batch and token count a call
admits at the benchmarked shapes: every launch's split-K partials and
attention partials lie inside the workspace the call validated, requests no
call admits are refused at once, and extreme config values cause no
undefined arithmetic. CPU only."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = [os.path.join(ROOT, "tests", "native", "plan_check.cpp"),
       os.path.join(ROOT, "paper_2302_01318_amd", "csrc", "plan.cpp")]


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_plan_under_sanitizers(tmp_path):
    exe = str(tmp_path / "plan_check")
    flags = ["-std=c++17", "-O1", "-g", "-Wall", "-fno-omit-frame-pointer",
             "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
    r = subprocess.run(["g++"] + flags + ["-I" + os.path.join(ROOT, "include")] + SRC + ["-o", exe],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert "plan check ok" in r.stdout
