"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer: the CPU
oracle (oracle/oracle.c) and the adaptive batcher (csrc/batcher.cpp), each
linked with a driver that exercises every entry point on small inputs held in
exactly sized heap buffers.  Any sanitizer report fails the run."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
       "-fno-sanitize-recover=all"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1", OMP_NUM_THREADS="2")


def _build_and_run(tmp_path, compiler, srcs, extra):
    exe = str(tmp_path / "driver")
    r = subprocess.run([compiler, *SAN, *srcs, *extra, "-o", exe], capture_output=True,
                       text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=120)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out
    assert "runtime error" not in out and "ERROR: AddressSanitizer" not in out, out
    return out


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not installed")
def test_oracle_under_sanitizers(tmp_path):
    out = _build_and_run(tmp_path, "gcc",
                         [os.path.join(ROOT, "oracle", "oracle.c"),
                          os.path.join(ROOT, "tests", "sanitize", "oracle_driver.c")],
                         ["-std=c11", "-fopenmp", "-lm"])
    assert "values checked" in out


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not installed")
def test_batcher_under_sanitizers(tmp_path):
    out = _build_and_run(tmp_path, "g++",
                         [os.path.join(ROOT, "paper_2507_18748_amd", "csrc", "batcher.cpp"),
                          os.path.join(ROOT, "tests", "sanitize", "batcher_driver.cpp")],
                         ["-std=c++17", "-I", os.path.join(ROOT, "include")])
    assert "0 overlaps" in out
