"""The CPU oracle built with AddressSanitizer and UndefinedBehaviorSanitizer
(g++, host code only) and driven through every entry point by
tests/oracle_asan_driver.cpp: random small cases, the method's edge cases and
invalid inputs.  Any out-of-bounds access, use of uninitialised heap memory
the sanitizers can see, leak or undefined operation fails the test."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_oracle_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    build = ["g++", "-O1", "-g", "-std=c++17", "-fno-omit-frame-pointer",
             "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
             os.path.join(ROOT, "oracle", "oracle.cpp"),
             os.path.join(HERE, "oracle_asan_driver.cpp"), "-o", exe]
    r = subprocess.run(build, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-6000:])
    assert "runtime error" not in r.stderr, r.stderr[-6000:]
    assert "all cases ran clean" in r.stdout
