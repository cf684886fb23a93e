"""The library's host code (fit, Cholesky and inverse, likelihood search,
forest training, EHVI boxes, forest packing and the shared thread pool) run
under AddressSanitizer with UndefinedBehaviorSanitizer, and under
ThreadSanitizer, through the CPU-only driver tests/host_sanitize.cpp: both
builds must exit cleanly with no sanitizer report.  Searches and forest
training run from several threads at once on the shared pool."""
import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2408_04323_amd", "csrc")

BUILDS = {
    "address,undefined": ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"],
    "thread": ["-fsanitize=thread"],
}


@pytest.mark.parametrize("which", list(BUILDS))
def test_host_code_under_sanitizers(tmp_path, which):
    cxx = shutil.which("g++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    exe = str(tmp_path / "host_sanitize")
    srcs = sorted(glob.glob(os.path.join(CSRC, "host_*.cpp")))
    cmd = [cxx, "-O1", "-g", "-std=c++17", "-fopenmp-simd", *BUILDS[which], "-I", os.path.join(ROOT, "include"),
           "-I", CSRC, os.path.join(ROOT, "tests", "host_sanitize.cpp"), *srcs, "-o", exe, "-lpthread"]
    subprocess.run(cmd, check=True)
    env = dict(os.environ, SCOOT_HOST_THREADS="6", ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1", TSAN_OPTIONS="halt_on_error=1 second_deadlock_stack=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    for marker in ("ERROR: AddressSanitizer", "ERROR: LeakSanitizer", "runtime error:", "WARNING: ThreadSanitizer"):
        assert marker not in out, out[-4000:]
    assert "OK: 0 failure(s)" in r.stdout
