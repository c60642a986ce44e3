"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer, on the CPU: the oracle (gcc) and
the library's host side (hipcc, sanitizers on the host pass only: each sanitizer flag sits right
after -Xarch_host, so no GPU code is built with them) are compiled with both sanitizers, and driver
programs in tests/sanitize/ run every host entry point on seeded random inputs.  A sanitizer report
or a wrong return code fails the test."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2609_38706_amd", "csrc")
SANITIZERS = ["address", "undefined"]


def _run(exe, env_extra):
    env = dict(os.environ)
    env.update(env_extra)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    report = r.stdout + r.stderr
    assert r.returncode == 0, report[-4000:]
    assert "runtime error" not in report and "AddressSanitizer" not in report, report[-4000:]


def test_oracle_under_sanitizers(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    exe = str(tmp_path / "oracle_san")
    cmd = [gcc, "-std=c11", "-O1", "-g", "-fno-omit-frame-pointer", "-fno-sanitize-recover=undefined"]
    cmd += ["-fsanitize=" + s for s in SANITIZERS]
    cmd += ["-o", exe, os.path.join(SAN, "oracle_driver.c"), os.path.join(ROOT, "oracle", "pkv_oracle.c"), "-lpthread"]
    subprocess.run(cmd, check=True, timeout=600)
    _run(exe, {"ASAN_OPTIONS": "detect_leaks=1:abort_on_error=0", "UBSAN_OPTIONS": "print_stacktrace=1"})


def test_library_host_code_under_sanitizers(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    exe = str(tmp_path / "host_san")
    cmd = [hipcc, "-std=c++17", "-O1", "-g", "--offload-arch=gfx950",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
    for s in SANITIZERS:
        cmd += ["-Xarch_host", "-fsanitize=" + s]
    cmd += ["-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]
    cmd += ["-I", os.path.join(ROOT, "include"), "-I", CSRC, "-o", exe, os.path.join(SAN, "host_driver.cpp")]
    cmd += [os.path.join(CSRC, f) for f in ("api.hip", "k_derive.hip", "k_table.hip", "k_tree.hip")]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    # the HIP runtime's own start-up allocations are not this library's: leak checking stays off here
    _run(exe, {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=0", "UBSAN_OPTIONS": "print_stacktrace=1"})
