"""The host geometry (Pareto front, box decomposition) built on its own with
AddressSanitizer and UndefinedBehaviorSanitizer and checked against brute
force (tests/host_geom_check.cpp). CPU only: host compiler, no device code."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="no host C++ compiler")
def test_host_geometry_under_sanitizers(tmp_path):
    exe = tmp_path / "host_geom_check"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
           "-I", "/opt/rocm/include",
           os.path.join(ROOT, "tests", "host_geom_check.cpp"),
           os.path.join(ROOT, "paper_2602_10729_amd", "csrc", "host_geom.cpp"),
           "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    # the sanitizer runtime need not be first among preloaded libraries here
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert "host geometry ok" in r.stdout
