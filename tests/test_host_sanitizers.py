"""The host side of the library (argument validation, parameter packing, calibration and bit
allocation: abi.cpp, group_abi.cpp and calibrate.cpp) built with the host compiler's AddressSanitizer and
UndefinedBehaviorSanitizer, with the HIP launchers replaced by host stubs
(tests/host_stub/launch_stub.cpp), and driven by the CPU tests of the C ABI."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_14191_amd", "csrc")


def _runtime(name):
    out = subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True, text=True)
    path = out.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.skipif(shutil.which("g++") is None, reason="no host C++ compiler")
def test_abi_and_calibration_under_asan_and_ubsan(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("no AddressSanitizer runtime")
    lib = tmp_path / "libaatc_sanitized.so"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fPIC", "-shared", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(CSRC, "calibrate.cpp"), os.path.join(CSRC, "abi.cpp"),
           os.path.join(CSRC, "group_abi.cpp"),
           os.path.join(ROOT, "tests", "host_stub", "launch_stub.cpp"), "-o", str(lib)]
    build = subprocess.run(cmd, capture_output=True, text=True)
    assert build.returncode == 0, build.stderr
    env = dict(os.environ, AATC_LIBRARY=str(lib), LD_PRELOAD=asan,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    run = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                          os.path.join(ROOT, "tests", "test_lib_cpu.py"),
                          os.path.join(ROOT, "tests", "test_lib_groups_cpu.py")],
                         capture_output=True, text=True, env=env, cwd=ROOT, timeout=600)
    tail = (run.stdout + run.stderr)[-3000:]
    assert run.returncode == 0, tail
    assert "passed" in run.stdout and "ERROR: AddressSanitizer" not in tail
    assert "runtime error" not in tail
