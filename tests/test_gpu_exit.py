"""A Python process that ends with pools still open.

The binding closes every pool still open from an exit hook registered after
torch's import (exit hooks run last-registered first), so kv_pool_destroy
waits for the pool's work and frees its memory while the HIP runtime is
whole, before the runtime's own exit-time teardown.  Each case runs in a
fresh interpreter and must end with status 0.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.gpu

SCRIPT = r"""
import sys
import torch
from kvgen import workloads
from paper_2606_14779_amd import kvpool as K
from paper_2606_14779_amd.runner import WorkloadRun

wl = workloads.make(3, max_blocks=200)
run = WorkloadRun(wl, 0)
run.setup()
run.pool.set_launch(K.CLASS_HOST, K.OP_RETRIEVE, 0, K.LAUNCH_SDMA)   # the copy-engine ring is live too
side = torch.cuda.Stream()
side.wait_stream(torch.cuda.current_stream())
run.retrieve(wl.requests[0], side)             # may still run when the interpreter exits
print("exiting with the pool open", flush=True)
if sys.argv[1] == "sys_exit":
    sys.exit(0)
"""


@pytest.mark.parametrize("how", ["end_of_script", "sys_exit"])
def test_interpreter_exit_with_a_pool_open(how):
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    env = dict(os.environ, PYTHONPATH=ROOT + os.pathsep + os.environ.get("PYTHONPATH", ""))
    r = subprocess.run([sys.executable, "-c", SCRIPT, how], capture_output=True, text=True, timeout=180,
                       env=env, cwd=ROOT)
    assert r.returncode == 0, "status %d\n%s%s" % (r.returncode, r.stdout, r.stderr[-3000:])
    assert "exiting with the pool open" in r.stdout
