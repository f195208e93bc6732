"""The library's host code (C-ABI argument checks, workspace layout
arithmetic) built with AddressSanitizer and UndefinedBehaviorSanitizer on the
host side only, and driven by tests/lib_asan_driver.cpp.  Every call in the
driver fails an argument check, so nothing reaches a GPU; the device pointers
are dummies.  It runs only where no GPU is visible, so that a call that wrongly
passed its checks could not launch a kernel on them."""
import glob
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
PKG = os.path.join(ROOT, "paper_2005_04680_amd")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _gpu_visible():
    return os.path.exists("/dev/kfd")


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="needs hipcc")
@pytest.mark.skipif(_gpu_visible(), reason="host-only driver: run where no GPU is visible")
def test_library_host_code_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "lib_driver")
    # Sanitizers on the host side only (-Xarch_host before each), device code as built.
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-ffp-contract=off",
             "-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "csrc")]
    srcs = sorted(glob.glob(os.path.join(PKG, "csrc", "*.hip")))
    objs = []
    procs = []
    for src in srcs:
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        objs.append(obj)
        procs.append(subprocess.Popen([HIPCC, *flags, *san, "-c", src, "-o", obj],
                                      stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True))
    for p in procs:
        out, err = p.communicate(timeout=600)
        assert p.returncode == 0, err[-4000:]
    drv = os.path.join(HERE, "lib_asan_driver.cpp")
    r = subprocess.run([HIPCC, *flags, *san, "-x", "hip", drv, "-x", "none", *objs, "-o", exe],
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="print_stacktrace=1")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-6000:])
    assert "runtime error" not in r.stderr, r.stderr[-6000:]
    assert "all cases ran clean" in r.stdout
