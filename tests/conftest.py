import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU; run with -m gpu")


@pytest.fixture(scope="session", autouse=True)
def _built_host_libs():
    """The oracle and the input generator are plain C; build them if absent."""
    import kvgen
    import oracle
    kvgen.build(force=False)
    oracle.build(force=False)
