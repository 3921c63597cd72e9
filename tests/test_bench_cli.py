"""bench.py's command line, checked without a GPU: more than one GPU is
refused with a message and exit status 2, every mode flag parses, and the
PMC summary it reads is parsed only for the kernels.hip it was taken with."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*args, timeout=120):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=timeout, cwd=ROOT)


@pytest.mark.parametrize("n", ["2", "8"])
def test_more_than_one_gpu_is_refused(n):
    r = _bench("--gpus", n)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_help_lists_every_mode():
    r = _bench("--help")
    assert r.returncode == 0
    for flag in ("--gpus", "--steps", "--warmup", "--config", "--layout", "--sdma", "--copy-ring-mib", "--flush",
                 "--pipeline", "--latency", "--duplex", "--ablation", "--layerwise", "--no-cpu-baseline",
                 "--no-probes", "--no-copy-engine", "--host-grid", "--staging-grid", "--store-grid", "--stand-in",
                 "--batch", "--context", "--upload", "--store-flags", "--decode"):
        assert flag in r.stdout, flag


def test_pmc_summary_matches_current_kernels():
    """The committed PMC summary names the kernels.hip it was taken with, and bench reads
    the host-class gather's traffic from it only while that source is unchanged."""
    sys.path.insert(0, ROOT)
    import hashlib

    import bench
    path = os.path.join(ROOT, "profiles", "retrieve_llama3.1-8b-kv-128k-6region_pmc.txt")
    text = open(path).read()
    sha = hashlib.sha256(open(os.path.join(ROOT, "paper_2606_14779_amd", "csrc", "kernels.hip"), "rb").read()).hexdigest()
    recorded = [l.split(":", 1)[1].strip() for l in text.splitlines() if l.startswith("kernels_hip_sha256:")]
    assert recorded, "no sha recorded"
    rec = bench.pmc_traffic("llama3.1-8b-kv-128k-6region", "host_region_copy<true, 0,")
    if recorded[0] == sha:
        assert rec is not None and rec["fetch_bytes"] > 0 and rec["write_bytes"] > 0
    else:
        assert rec is None
