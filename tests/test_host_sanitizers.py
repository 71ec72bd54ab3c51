"""The host side of libmkv (argument validation, arena layout, KV-memory accounting, the
configuration choice, the codebook fit) built with AddressSanitizer and UndefinedBehaviorSanitizer
on host code only, and run on the CPU through a small native driver (tests/native/host_checks.cpp)
whose kernel launchers are stubs: no path it takes reaches a device."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not found")
def test_host_library_under_asan_and_ubsan(tmp_path):
    csrc = os.path.join(ROOT, "paper_2609_07966_amd", "csrc")
    srcs = [os.path.join(csrc, f) for f in ("mkv_api.cpp", "calib.cpp", "select.cpp")]
    srcs.append(os.path.join(ROOT, "tests", "native", "host_checks.cpp"))
    exe = str(tmp_path / "host_checks")
    cmd = [HIPCC, "-O1", "-g", "-std=c++17", "-fno-omit-frame-pointer",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-fno-sanitize-recover=undefined",
           "-I", os.path.join(ROOT, "include"), "-I", csrc] + srcs + ["-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "ok (0 failures)" in r.stdout
