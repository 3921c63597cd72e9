"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only): tests/native/host_structures_fuzz.cpp built with placement.cpp,
glt.cpp and bounce.cpp; tests/native/file_io_test.cpp built with fileio.cpp
(the storage tier's plan, worker threads and files); tests/native/placement_fuzz.cpp driving
placement-only pools through the C ABI of the host-sanitized library;
tests/native/alloc_failure.cpp failing host allocations inside place, extend
and release; and the oracle itself (tests/native/oracle_fuzz.c)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_14779_amd", "csrc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_structures_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "host_structures_fuzz")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-isystem", os.path.join(ROCM, "include"),
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "native", "host_structures_fuzz.cpp"),
           os.path.join(CSRC, "placement.cpp"), os.path.join(CSRC, "glt.cpp"), os.path.join(CSRC, "bounce.cpp"),
           "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_file_tier_host_side_under_asan_ubsan(tmp_path):
    """plan_file's batches on random inputs, the per-region worker threads on O_DIRECT files, and the
    file-region life cycle (tests/native/file_io_test.cpp)."""
    exe = str(tmp_path / "file_io_test")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-pthread", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-isystem", os.path.join(ROCM, "include"),
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "native", "file_io_test.cpp"), os.path.join(CSRC, "fileio.cpp"),
           os.path.join(CSRC, "placement.cpp"), "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout


SAN_LIB = os.path.join(ROOT, "tests", "abi_client", "asan", "libkvpool.so")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_placement_through_the_abi_under_asan_ubsan(tmp_path):
    """Random place / extend / release / lookup on placement-only pools, through the C ABI of the
    host-sanitized library (built by the package build), with no GPU."""
    if not os.path.exists(SAN_LIB):
        pytest.skip("host-sanitized library not built (run the package build first)")
    exe = str(tmp_path / "placement_fuzz")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "native", "placement_fuzz.cpp"),
           "-o", exe, "-L", os.path.dirname(SAN_LIB), "-lkvpool", "-Wl,-rpath," + os.path.dirname(SAN_LIB),
           "-L", os.path.join(ROCM, "lib"), "-Wl,-rpath-link," + os.path.join(ROCM, "lib")]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_allocation_failures_change_nothing(tmp_path):
    """Every place, extend and release retried with each of its host allocations failing in turn:
    each failed try returns KVP_ERR_NOMEM and leaves the pool as it was, checked against a twin pool
    that never fails (tests/native/alloc_failure.cpp), with leak checking."""
    if not os.path.exists(SAN_LIB):
        pytest.skip("host-sanitized library not built (run the package build first)")
    exe = str(tmp_path / "alloc_failure")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "native", "alloc_failure.cpp"),
           "-o", exe, "-L", os.path.dirname(SAN_LIB), "-lkvpool", "-Wl,-rpath," + os.path.dirname(SAN_LIB),
           "-L", os.path.join(ROCM, "lib"), "-Wl,-rpath-link," + os.path.join(ROCM, "lib")]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_asan_ubsan(tmp_path):
    """The oracle itself under the sanitizers, with leak checking: place / extend / release and store /
    gather round trips into exactly-sized buffers (tests/native/oracle_fuzz.c)."""
    exe = str(tmp_path / "oracle_fuzz")
    cmd = ["gcc", "-std=c11", "-O1", "-g", "-Wall", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           os.path.join(ROOT, "tests", "native", "oracle_fuzz.c"), os.path.join(ROOT, "oracle", "oracle.c"),
           "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout
