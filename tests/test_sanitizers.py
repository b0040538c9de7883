"""Host code under sanitizers (CPU only).

The float64 oracle and the host trajectory record are built with gcc / g++ together with small
drivers (tests/sanitize/) that call every entry point on edge-case inputs: AddressSanitizer and
UndefinedBehaviorSanitizer for both, ThreadSanitizer for the record store, which four threads
use at once.  The drivers allocate each buffer at exactly the size a call may touch, so a read
or write past it fails the build's run.  No GPU code is built here.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
ROCM_INCLUDE = "/opt/rocm/include"  # stride.h names hipStream_t from the HIP runtime API header


def _run(cmd, env=None, timeout=300):
    r = subprocess.run(cmd, capture_output=True, text=True, env=env, timeout=timeout)
    return r.returncode, r.stdout + r.stderr


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_address_and_undefined_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    rc, out = _run(["gcc", "-std=c11", "-O1", "-g", "-fopenmp", "-ffp-contract=off",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    "-fno-omit-frame-pointer", os.path.join(ROOT, "oracle", "oracle.c"),
                    os.path.join(SAN, "oracle_driver.c"), "-o", exe, "-lm"])
    assert rc == 0, out
    env = dict(os.environ, OMP_NUM_THREADS="4", ASAN_OPTIONS="detect_leaks=1")
    rc, out = _run([exe], env=env)
    assert rc == 0 and "oracle driver ok" in out, out


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir(ROCM_INCLUDE),
                    reason="g++ or the HIP headers not available")
@pytest.mark.parametrize("sanitizer", ["address,undefined", "thread"])
def test_record_store_under_sanitizers(tmp_path, sanitizer):
    exe = str(tmp_path / "records_driver")
    rc, out = _run(["g++", "-std=c++17", "-O1", "-g", "-D__HIP_PLATFORM_AMD__", "-I", ROCM_INCLUDE,
                    f"-fsanitize={sanitizer}", "-fno-sanitize-recover=all",
                    "-fno-omit-frame-pointer",
                    os.path.join(ROOT, "paper_2609_14636_amd", "csrc", "record.cpp"),
                    os.path.join(SAN, "records_driver.cpp"), "-o", exe, "-pthread"])
    assert rc == 0, out
    rc, out = _run([exe])
    assert rc == 0 and "records driver ok" in out, out
