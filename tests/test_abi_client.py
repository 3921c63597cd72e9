"""The C ABI from a plain C++ program (no Python in the data path, no torch)."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXE = os.path.join(ROOT, "tests", "abi_client", "abi_client")

pytestmark = pytest.mark.gpu


def test_cpp_client_round_trip():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    assert os.path.exists(EXE), "abi_client is built by paper_2606_14779_amd.build"
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "retrieved exactly" in r.stdout


def test_cpp_client_under_host_sanitizers():
    """The same client over a build of the library whose host code runs under AddressSanitizer and
    UndefinedBehaviorSanitizer (GPU code uninstrumented): every host-side path it takes -- create,
    place, store, retrieve by id, the copy-engine ring, release, destroy -- without a finding.
    Leak checking is off: the ROCm runtime keeps allocations until exit."""
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    exe = os.path.join(ROOT, "tests", "abi_client", "abi_client_asan")
    assert os.path.exists(exe), "abi_client_asan is built by paper_2606_14779_amd.build"
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:verify_asan_link_order=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "retrieved exactly" in r.stdout
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr


def test_cpp_client_exits_with_a_pool_open():
    """A C++ caller that returns from main with its pool open and a retrieve enqueued (no
    kv_pool_destroy): the process ends with status 0.  The library has no exit-time handler or
    static destructor that calls the HIP runtime, so nothing of it runs after the runtime's own
    teardown."""
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    r = subprocess.run([EXE, "exit-open"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "exiting with the pool open" in r.stdout
