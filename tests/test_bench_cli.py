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
                 "--batch", "--context", "--upload", "--store-flags", "--decode", "--measured-weights",
                 "--summarize-pmc", "--summarize-trace", "--weights", "--file-regions", "--file-dir",
                 "--host-staged", "--store-staging-grid", "--store-staging-flags"):
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


def test_pmc_summary_from_counter_passes(tmp_path):
    """The summary step on synthetic rocprofv3 counter files: FETCH_SIZE / WRITE_SIZE are scaled so
    that the 4 GiB probe copy reads and writes 4 GiB (the derived FETCH_SIZE prices 128-byte reads
    at 64 bytes on gfx950, so its scale comes out 2), the per-destination 32-byte counters become
    bytes unscaled, and bench reads the figures back for the current kernels.hip."""
    sys.path.insert(0, ROOT)
    import csv
    import bench
    hdr = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id", "Grid_Size",
           "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size", "Scratch_Size", "VGPR_Count",
           "Accum_VGPR_Count", "SGPR_Count", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]
    probe = "void kvp::probe_copy_kernel<4, true, false>(HIP_vector_type<unsigned int, 4u> const*, ...)"
    host = "void kvp::host_region_copy<true, 0, 8, false, false>(kvp::CopyArgs)"
    four_gib_kib = 4 * 2 ** 20
    rows = {                       # pass -> [(kernel, grid threads, counter, value)]
        "fetch": [(probe, 65536 * 256, "FETCH_SIZE", four_gib_kib / 2), (host, 12 * 256, "FETCH_SIZE", 1000.0)],
        "write": [(probe, 65536 * 256, "WRITE_SIZE", four_gib_kib), (host, 12 * 256, "WRITE_SIZE", 3000.0)],
        "rd": [(probe, 65536 * 256, "TCC_EA0_RDREQ_DRAM_32B_sum", (4 << 30) / 32),
               (host, 12 * 256, "TCC_EA0_RDREQ_IO_32B_sum", 1e6), (host, 12 * 256, "TCC_EA0_RDREQ_DRAM_32B_sum", 5)],
    }
    for name, rs in rows.items():
        os.makedirs(tmp_path / "pmc" / name)
        with open(tmp_path / "pmc" / name / (name + "_counter_collection.csv"), "w", newline="") as f:
            w = csv.writer(f)
            w.writerow(hdr)
            for i, (k, grid, c, v) in enumerate(rs):
                w.writerow([i, i, "Agent 1", 0, 1, 1, grid, 1, k, 256, 0, 0, 8, 0, 16, c, v, 0, 1])
    out = tmp_path / "profiles"
    os.makedirs(out)
    bench.summarize_pmc(str(tmp_path / "pmc"), "synthetic", "--steps 2", out_dir=str(out))
    text = open(out / "retrieve_synthetic_pmc.txt").read()
    assert "fetch_scale: 2.000000" in text and "write_scale: 1.000000" in text
    rec = bench.pmc_traffic("synthetic", "host_region_copy<true, 0,", profiles_dir=str(out))
    assert rec is not None
    assert rec["workgroups"] == 12
    assert rec["fetch_bytes"] == 1000.0 * 1024 * 2 and rec["write_bytes"] == 3000.0 * 1024
    assert rec["rd_io_bytes"] == 32e6 and rec["rd_dram_bytes"] == 160
    p = bench.pmc_traffic("synthetic", "probe_copy_kernel<4,", profiles_dir=str(out))
    assert p["rd_dram_bytes"] == 4 << 30
