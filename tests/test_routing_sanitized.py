"""The host routing library (route.cpp) under AddressSanitizer and
UndefinedBehaviorSanitizer: a randomized driver (routing_fuzz.cpp) calls every
entry point of include/eldr_route.h on random shapes and edge values; any
sanitizer report fails the test.  CPU only (g++)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_routing_library_under_sanitizers(tmp_path):
    exe = tmp_path / "routing_fuzz"
    build = subprocess.run(
        ["g++", "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
         "-fno-omit-frame-pointer", "-I", os.path.join(ROOT, "include"),
         os.path.join(ROOT, "tests", "routing_fuzz.cpp"),
         os.path.join(ROOT, "paper_2607_00466_amd", "csrc", "route.cpp"), "-o", str(exe)],
        capture_output=True, text=True, timeout=300)
    assert build.returncode == 0, build.stderr[-2000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    out = run.stdout + run.stderr
    assert run.returncode == 0, out[-3000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-3000:]
    assert "calls" in run.stdout
