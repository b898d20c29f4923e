"""The oracle's C code under AddressSanitizer and UBSan: a copy built with
both runs a set of the oracle's own pin tests in a child process (the
instrumented library is loaded only there)."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    r = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
def test_oracle_pins_pass_under_asan_and_ubsan(tmp_path):
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if asan is None or ubsan is None:
        pytest.skip("sanitizer runtimes not found")
    lib = tmp_path / "liboracle.so"
    subprocess.run(["gcc", "-std=c11", "-O1", "-g", "-fPIC", "-shared", "-fopenmp",
                    "-ffp-contract=off", "-fno-fast-math", "-mfma",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                    os.path.join(ROOT, "oracle", "arc_oracle.c"), "-o", str(lib), "-lm"],
                   check=True, capture_output=True, timeout=300)
    log = tmp_path / "sanitizer"
    env = dict(os.environ, LD_PRELOAD=f"{asan} {ubsan}", ARC_ORACLE_LIB=str(lib),
               ASAN_OPTIONS=f"detect_leaks=0:log_path={log}", UBSAN_OPTIONS=f"log_path={log}")
    tests = [os.path.join(ROOT, "tests", t) for t in
             ("test_oracle_select.py", "test_oracle_stages.py", "test_oracle_step.py",
              "test_oracle_tensors.py", "test_oracle_compare.py", "test_oracle_model.py")]
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        *tests], cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    reports = "".join(p.read_text() for p in tmp_path.glob("sanitizer*"))
    assert r.returncode == 0 and not reports, reports[:3000] + r.stdout[-2000:]
