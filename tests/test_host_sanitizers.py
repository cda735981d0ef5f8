"""Host-side schedule builders under AddressSanitizer and UBSan.

Builds tests/host_schedule_fuzz.cpp together with the library's host-only
schedule source with g++ (-fsanitize=address,undefined; no GPU code is
compiled with a sanitizer) and runs it: random valid shapes of both kinds
of schedule and of block-sparse lists, one-word-short output buffers, and
malformed inputs (decreasing cu_seqlens, out-of-range or unsorted k-tile
indices, inconsistent list offsets, bad scalars).  Any sanitizer report
fails the test.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_schedule_builders_under_sanitizers(tmp_path):
    exe = tmp_path / "host_schedule_fuzz"
    build = subprocess.run(
        ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
         "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
         "-I", os.path.join(ROOT, "include"), "-o", str(exe),
         os.path.join(ROOT, "tests", "host_schedule_fuzz.cpp"),
         os.path.join(ROOT, "paper_2507_21526_amd", "csrc", "triattn_schedule.cpp")],
        capture_output=True, text=True, timeout=300)
    assert build.returncode == 0, build.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    assert run.returncode == 0, (run.stdout + run.stderr)[-4000:]
    assert "runtime error" not in run.stderr and "AddressSanitizer" not in run.stderr
    assert "ok " in run.stdout and "malformed: rejected" in run.stdout
