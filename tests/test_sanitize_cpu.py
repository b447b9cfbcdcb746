"""Host sanitizers over the C-ABI layer and the planner's host mirror.

api.cpp is built with AddressSanitizer and UndefinedBehaviorSanitizer on the
host side only (-Xarch_host before each -fsanitize=), linked against a
test-only stub of the kernel launchers, and driven over random shapes by
tests/sanitize/plan_fuzz.cpp: splash_mla_plan_host with every buffer at
exactly its documented size, coverage of each plan, and the argument checks.
No GPU is used.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_37626_amd", "csrc")


@pytest.mark.timeout(600)
def test_planner_and_abi_under_host_sanitizers(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not found")
    exe = tmp_path / "plan_fuzz"
    cmd = [hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(CSRC, "api.cpp"), os.path.join(ROOT, "tests", "sanitize", "launch_stubs.cpp"),
           os.path.join(ROOT, "tests", "sanitize", "plan_fuzz.cpp"), "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe), "400"], capture_output=True, text=True, env=env, timeout=500)
    print(r.stdout[-2000:], r.stderr[-4000:])
    assert r.returncode == 0, r.stderr[-4000:]
    assert r.stdout.startswith("ok ") and int(r.stdout.split()[1]) > 100
