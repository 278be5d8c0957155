"""The host-only library (cache plan, expert packers, error reporting) built with
AddressSanitizer and UndefinedBehaviorSanitizer and driven over random and invalid inputs
(tests/native/host_sanitized.cpp): no access outside the buffers apex.h declares and no
undefined behaviour."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_host_library_under_sanitizers(tmp_path):
    from paper_2608_11688_amd import build
    cxx = shutil.which("g++")
    if cxx is None:
        pytest.skip("no g++")
    exe = str(tmp_path / "host_sanitized")
    srcs = [os.path.join(build.CSRC, s) for s in build.HOST_SOURCES]
    cmd = [cxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"), "-I", build.CSRC,
           "-I", "/opt/rocm/include",
           os.path.join(ROOT, "tests", "native", "host_sanitized.cpp"), *srcs, "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), (r.stdout[-2000:],
                                                                   r.stderr[-4000:])
