"""AddressSanitizer and UndefinedBehaviorSanitizer builds of the CPU oracle
and of the library's host code (CPU only).

tests/sanitize/oracle_driver.c runs every oracle entry point on seeded random
inputs of several shapes (1 device up to 256 devices x 255 blocks);
tests/sanitize/lib_driver.cpp runs libe2's host-only paths: quantisation
(including overflow), every argument check, and context creation failing at
its first HIP call (the failure injection hook), which must leak nothing.
Each is built with the sanitizers (GPU code of the library untouched: the
host flags only) and must exit 0 with no sanitizer report.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2606_03770_amd", "csrc")
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def _run(exe, timeout):
    r = subprocess.run([exe], env=ENV, capture_output=True, text=True, timeout=timeout)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert "runtime error" not in r.stderr and "ERROR: AddressSanitizer" not in r.stderr
    return r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    subprocess.check_call(["gcc", "-O1", "-g", "-fno-omit-frame-pointer",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                           "-o", exe, os.path.join(SAN, "oracle_driver.c"),
                           os.path.join(ROOT, "oracle", "oracle.c")])
    assert "shapes ok" in _run(exe, 300)


def _hipcc():
    for c in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    return None


@pytest.mark.skipif(_hipcc() is None, reason="needs hipcc")
def test_library_host_code_under_sanitizers(tmp_path):
    exe = str(tmp_path / "lib_driver")
    # the sanitizers apply to host code only (each flag after -Xarch_host)
    cmd = [_hipcc(), "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-fno-omit-frame-pointer", "-o", exe,
           os.path.join(CSRC, "e2_api.hip"), os.path.join(CSRC, "e2_kernels.hip"),
           os.path.join(SAN, "lib_driver.cpp")]
    subprocess.check_call(cmd, stderr=subprocess.DEVNULL)
    assert "library host driver: ok" in _run(exe, 120)
