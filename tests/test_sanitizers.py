"""The oracle and the library's host code built with AddressSanitizer and
UndefinedBehaviorSanitizer (plain gcc/g++, CPU only) and driven on small
inputs: tests/sanitize/oracle_driver.c runs the oracle's step, rotary step
and prefill over NaN-poisoned caches; tests/sanitize/host_driver.cpp runs map
construction, argument validation, planning and workspace sizing of every
entry point, with the device side replaced by host stand-ins
(tests/sanitize/kernel_stubs.cpp) that refuse launches."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-g", "-O1", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
       "-fno-omit-frame-pointer"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", OMP_NUM_THREADS="2")


def _run(exe):
    r = subprocess.run([exe], env=ENV, capture_output=True, text=True, timeout=300)
    report = r.stdout + r.stderr
    assert r.returncode == 0, report
    assert "runtime error" not in report and "AddressSanitizer" not in report, report
    assert "0 failure(s)" in r.stdout, report


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    subprocess.check_call(["gcc", "-std=c11", *SAN, "-fopenmp",
                           os.path.join(ROOT, "oracle", "oracle.c"),
                           os.path.join(ROOT, "tests", "sanitize", "oracle_driver.c"),
                           "-lm", "-o", exe], timeout=300)
    _run(exe)


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include"),
                    reason="needs g++ and the ROCm headers")
def test_host_code_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    exe = str(tmp_path / "host_driver")
    csrc = os.path.join(ROOT, "paper_2406_09297_amd", "csrc")
    subprocess.check_call(["g++", "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__",
                           "-I/opt/rocm/include", "-I", os.path.join(ROOT, "include"), "-I", csrc,
                           os.path.join(csrc, "mlkv.cpp"),
                           os.path.join(ROOT, "tests", "sanitize", "kernel_stubs.cpp"),
                           os.path.join(ROOT, "tests", "sanitize", "host_driver.cpp"),
                           "-L/opt/rocm/lib", "-lamdhip64", "-lrocblas",
                           "-Wl,-rpath,/opt/rocm/lib", "-o", exe], timeout=600)
    _run(exe)
