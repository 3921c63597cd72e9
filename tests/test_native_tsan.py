"""The library's host code under ThreadSanitizer (CPU only): several threads
place, extend, look up and release requests on one placement-only pool at
once through the C ABI while others read it (tests/native/placement_threads.cpp);
and the storage tier's worker threads, fed by one and by two submitting
threads (tests/native/file_io_test.cpp with fileio.cpp).

The library's C++ sources are compiled here with g++ -fsanitize=thread and
linked with the kernels object of the package build (GPU code, never called
by a placement-only pool)."""
import concurrent.futures as cf
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2606_14779_amd")
CSRC = os.path.join(PKG, "csrc")
KERNELS_OBJ = os.path.join(PKG, "_build", "kernels.hip.o")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
FLAGS = ["-std=c++17", "-O1", "-g", "-fsanitize=thread", "-D__HIP_PLATFORM_AMD__", "-isystem",
         os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, " ".join(cmd) + "\n" + r.stdout + r.stderr


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_placement_from_many_threads_under_tsan(tmp_path):
    if not os.path.exists(KERNELS_OBJ):
        pytest.skip("kernels object not built (run the package build first)")
    srcs = sorted(os.path.join(CSRC, n) for n in os.listdir(CSRC) if n.endswith(".cpp"))
    srcs.append(os.path.join(ROOT, "tests", "native", "placement_threads.cpp"))
    objs = [str(tmp_path / (os.path.basename(s) + ".o")) for s in srcs]
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        list(ex.map(lambda so: _run(["g++"] + FLAGS + ["-c", so[0], "-o", so[1]]), zip(srcs, objs)))
    exe = str(tmp_path / "placement_threads")
    _run(["g++", "-fsanitize=thread", "-o", exe] + objs + [KERNELS_OBJ, "-L" + os.path.join(ROCM, "lib"),
         "-lamdhip64", "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-pthread"])
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1 second_deadlock_stack=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout
    assert "ThreadSanitizer" not in r.stderr, r.stderr


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_file_workers_under_tsan(tmp_path):
    exe = str(tmp_path / "file_io_test")
    _run(["g++"] + FLAGS + ["-pthread", os.path.join(ROOT, "tests", "native", "file_io_test.cpp"),
                            os.path.join(CSRC, "fileio.cpp"), os.path.join(CSRC, "placement.cpp"), "-o", exe])
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1 second_deadlock_stack=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout
    assert "ThreadSanitizer" not in r.stderr, r.stderr
