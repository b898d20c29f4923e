"""libarctopk's host code under AddressSanitizer (with leak checking) on the
CPU: a copy of the library whose host compilation carries the sanitizer
(device code is built as usual) is driven through the C ABI paths that need
no device by tests/abi_asan_check.c: every configuration rejection, the
create-time planning of valid layouts, the host projection and the
NULL-context paths."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLANG = "/opt/rocm/llvm/bin/clang"


@pytest.mark.skipif(shutil.which("hipcc") is None or not os.path.exists(CLANG),
                    reason="hipcc / ROCm clang not found")
def test_host_code_under_asan(tmp_path):
    import __graft_entry__ as ge
    lb = ge._load_by_path("_arc_lib_build_asan", "paper_2510_26709_amd/build.py")
    lib = tmp_path / "libarctopk.so"
    # each -fsanitize= right after -Xarch_host: host compilation only
    lb.build_lib(extra_flags=["-g", "-fno-omit-frame-pointer", "-Xarch_host",
                              "-fsanitize=address"],
                 out=str(lib), obj_dir=str(tmp_path / "obj"))
    exe = tmp_path / "abi_asan_check"
    subprocess.run([CLANG, "-g", "-fsanitize=address", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "abi_asan_check.c"), f"-L{tmp_path}",
                    "-larctopk", f"-Wl,-rpath,{tmp_path}", "-o", str(exe)],
                   check=True, capture_output=True, timeout=300)
    out = subprocess.run(["nm", "-D", str(lib)], capture_output=True, text=True,
                         check=True).stdout
    assert "__asan_report" in out, "the library copy is not instrumented"
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout + r.stderr[-4000:]
    assert r.stdout.strip().endswith("ok")
    assert "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
