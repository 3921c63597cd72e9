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
