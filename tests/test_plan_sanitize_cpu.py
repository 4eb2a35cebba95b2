"""The plan builder (host C++) under AddressSanitizer and UndefinedBehaviorSanitizer:
tests/plan_fuzz.cpp, built with g++ together with plan.cpp (no HIP code), feeds it
random valid and invalid descriptors and checks the structure of every plan it
accepts.  Any sanitizer report or failed check fails the test."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ is not installed")
def test_plan_builder_fuzz_under_sanitizers(tmp_path):
    exe = str(tmp_path / "plan_fuzz")
    build = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=undefined", "-I", os.path.join(ROOT, "include"),
             "-I", os.path.join(ROOT, "paper_2607_17715_amd", "csrc"),
             os.path.join(ROOT, "tests", "plan_fuzz.cpp"),
             os.path.join(ROOT, "paper_2607_17715_amd", "csrc", "plan.cpp"), "-o", exe]
    r = subprocess.run(build, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    for seed in (1, 2):
        r = subprocess.run([exe, "6000", str(seed)], capture_output=True, text=True,
                           timeout=300, env=env)
        assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
        assert "ERROR" not in r.stderr and "runtime error" not in r.stderr, r.stderr[-4000:]
        ok, rejected = int(r.stdout.split()[1]), int(r.stdout.split()[3])
        assert ok > 500 and rejected > 500, r.stdout
