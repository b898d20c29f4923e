"""The projection thread pool of libarctopk (host code) against its own
single-threaded generator, built and run under ThreadSanitizer on the CPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2510_26709_amd", "csrc")


@pytest.mark.skipif(shutil.which("hipcc") is None, reason="hipcc not found")
def test_projection_pool_matches_single_thread_under_tsan(tmp_path):
    exe = tmp_path / "projection_pool_check"
    # host code only: the sanitizer applies to the host compilation
    cmd = ["hipcc", "-std=c++17", "-O1", "-g", "-Xarch_host", "-fsanitize=thread",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "projection_pool_check.cpp"),
           os.path.join(CSRC, "arc_projection.cpp"), "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True, timeout=300)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300,
                       env=dict(os.environ, TSAN_OPTIONS="halt_on_error=1"))
    assert r.returncode == 0, r.stdout + r.stderr[-3000:]
    assert r.stdout.strip().endswith("ok")
    assert "ThreadSanitizer" not in r.stderr, r.stderr[-3000:]
