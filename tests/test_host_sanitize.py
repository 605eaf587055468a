"""The host planner (plan.cpp: scales, rectangles, stitching, conv5 windows) built with
AddressSanitizer and UndefinedBehaviorSanitizer on the CPU and driven over a grid of image sizes,
recipes, batches and invalid arguments (tests/host_sanitize_plan.cpp).  A memory error, undefined
behaviour or a violated plan invariant fails the test.  Host code only: no device code is built."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

pytestmark = pytest.mark.slow


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not found")
def test_planner_under_asan_and_ubsan(tmp_path):
    exe = tmp_path / "plan_sanitized"
    cmd = [HIPCC, "-O1", "-g", "-fno-omit-frame-pointer",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_1404_1869_amd", "csrc"),
           os.path.join(ROOT, "tests", "host_sanitize_plan.cpp"),
           os.path.join(ROOT, "paper_1404_1869_amd", "csrc", "plan.cpp"), "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, (r.stdout + r.stderr)[-3000:]
    assert "errors 0" in r.stdout
