"""The library's host code (KV block allocator, batch builder, shared-prefix
grouping, attention work planners, mode switch) built with g++ under
AddressSanitizer and UndefinedBehaviorSanitizer and driven by randomised
operation sequences (tests/sanitize/host_fuzz.cpp), every invariant checked
after every step.  CPU only: no HIP code is compiled."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2609_37062_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_host_code_under_address_and_ub_sanitizers(tmp_path):
    exe = str(tmp_path / "host_fuzz")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"),
           os.path.join(HERE, "sanitize", "host_fuzz.cpp"),
           os.path.join(CSRC, "alloc.cpp"), os.path.join(CSRC, "mode.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe, "300"], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert "passed" in r.stdout
    print(r.stdout.strip())
    # the random sequences reach every planner
    counts = [int(t) for t in r.stdout.replace(",", " ").replace(";", " ").split() if t.isdigit()]
    assert all(c > 0 for c in counts[:5]), r.stdout
