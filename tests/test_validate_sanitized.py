"""The C ABI's host-side argument checks (e2s_validate.cpp: every entry point runs
them before it touches the HIP runtime) built with AddressSanitizer and
UndefinedBehaviorSanitizer (g++, CPU only) and driven by randomized, often
extreme, arguments (tests/native/validate_fuzz.cpp): no out-of-bounds access,
signed overflow or other undefined behaviour, and the fixed cases give their
status codes."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_23253_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_validation_under_asan_and_ubsan(tmp_path):
    exe = tmp_path / "validate_fuzz"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}",
           os.path.join(ROOT, "tests", "native", "validate_fuzz.cpp"),
           os.path.join(CSRC, "e2s_validate.cpp"), "-o", str(exe)]
    build = subprocess.run(cmd, capture_output=True, text=True)
    assert build.returncode == 0, build.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    run = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    print(run.stdout)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "0 failures" in run.stdout
