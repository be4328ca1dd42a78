"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer.

tests/sanitize_schedule_driver.cpp drives seedq_plan_schedule and
seedq_derive_schedule with random descriptors, valid and broken;
tests/sanitize_frontend_driver.cpp the front end's Gauss-Hermite rule, channel
sort and outlier selection. Built here with the sanitizers on host code only,
any out-of-bounds access, leak or undefined operation makes a driver exit
non-zero."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")


def _build_and_run(tmp_path, source, driver, args):
    exe = str(tmp_path / driver)
    cmd = [HIPCC, "-O1", "-g", "-std=c++17", "-D__HIP_PLATFORM_AMD__",
           "-I" + os.path.join(ROOT, "include"),
           "-I" + os.path.join(ROOT, "paper_2609_38477_amd", "csrc"),
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-fno-gpu-sanitize",
           os.path.join(ROOT, "paper_2609_38477_amd", "csrc", source),
           os.path.join(ROOT, "tests", driver + ".cpp"), "-o", exe]
    b = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert b.returncode == 0, b.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe, *args], capture_output=True, text=True, timeout=600, env=env)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "failures 0" in r.stdout


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not found")
def test_planner_under_sanitizers(tmp_path):
    _build_and_run(tmp_path, "seedq_schedule.cpp", "sanitize_schedule_driver", ["3000"])


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not found")
def test_frontend_host_code_under_sanitizers(tmp_path):
    _build_and_run(tmp_path, "seedq_frontend_host.cpp", "sanitize_frontend_driver", [])
