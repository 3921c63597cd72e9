"""Benchmark of KV-cache retrieval from a bandwidth-striped KV pool on one MI355X.

One step = one ``kv_pool_retrieve`` of a whole 128K-token LLaMA-3.1-8B-shaped
request (8192 blocks of 16 tokens, 32 layers, 8 KV heads, head_dim 128, bf16:
16 GiB) striped over 2 pinned host regions (weight 4 each) and 4 HBM staging
regions standing in for SSDs (weight 1 each), gathered into a fragmented
10240-slot paged cache.  Inputs are resident (pool filled by kv_pool_store)
before the timed region starts.

Prints one JSON line: retrieved GB/s (value), ms per retrieve, the two
kernels' durations from HIP events recorded on the streams they run on, the
measured copy peaks (HBM copy kernel / hipMemcpy D2D; host->GPU zero-copy
kernel / hipMemcpy H2D) from the same process, and the CPU oracle timed on
a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PCIE5_X16_GBPS = 64.0       # published per-direction rate of the MI355X host link (PCIe 5.0 x16)
HBM_PEAK_GBPS = 8000.0      # published MI355X HBM3E bandwidth


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _events_ms(torch, fn, iters=3):
    """Best and list of per-iteration ms of fn() on the current stream."""
    out = []
    for _ in range(iters):
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        fn()
        e.record()
        e.synchronize()
        out.append(s.elapsed_time(e))
    return out


HBM_PROBE_GRIDS = (2048, 8192, 32768, 65536, 262144)   # grids of the 4 GiB HBM copy sweep (262144: one
                                                       # 16 KiB tile per workgroup)
SAME_BYTES_GRIDS = (16384, 131072, 1048576)   # grids of the same-bytes copy probe: none of the 4 GiB sweep's


def probes(torch, K, run, nbytes, same_bytes=0):
    """Copy peaks in GB/s (1e9 B/s of copied bytes), measured on this GPU in this process.

    same_bytes: also a contiguous HBM copy of that many bytes (the staging side's bytes of the
    step), since a copy's rate falls as its address span grows; its grids differ from the 4 GiB
    sweep's, so that traces and counters tell the two apart."""
    res = {}
    cur = torch.cuda.current_stream()
    n = same_bytes // 16384 * 16384
    free = torch.cuda.mem_get_info()[0] if same_bytes >= (64 << 20) else 0
    if same_bytes >= (64 << 20) and 2 * n + (1 << 30) > free:
        # two buffers of the staging side's size do not fit beside the caches and regions
        res["hbm_copy_same_bytes_skipped"] = "needs 2 x %d B of HBM, %d B free" % (n, free)
    elif same_bytes >= (64 << 20):
        a = torch.empty(n // 2, dtype=torch.int16, device="cuda")
        b = torch.empty_like(a)
        a.fill_(1)
        best, bgrid, bflags = 0.0, 0, 0
        for grid in SAME_BYTES_GRIDS:
            for fl in (K.LAUNCH_SPLIT2, K.LAUNCH_SPLIT2 | K.LAUNCH_NT_LOAD,
                       K.LAUNCH_SPLIT2 | K.LAUNCH_NT_LOAD | K.LAUNCH_NT_STORE):
                ms = min(_events_ms(torch, lambda: K.probe_copy_kernel(b.data_ptr(), a.data_ptr(), n, grid, fl,
                                                                       cur.cuda_stream)))
                if n / ms / 1e6 > best:
                    best, bgrid, bflags = n / ms / 1e6, grid, fl
        res["hbm_copy_same_bytes"] = {"bytes": n, "gbps": round(best, 1), "grid": bgrid, "flags": bflags}
        del a, b
        torch.cuda.empty_cache()
    a = torch.empty(nbytes // 2, dtype=torch.int16, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1)
    best_k, best_grid, best_flags = 0.0, 0, 0
    for grid in HBM_PROBE_GRIDS:
        for fl in (0, K.LAUNCH_NT_LOAD, K.LAUNCH_SPLIT2, K.LAUNCH_SPLIT2 | K.LAUNCH_NT_LOAD,
                   K.LAUNCH_SPLIT2 | K.LAUNCH_NT_LOAD | K.LAUNCH_NT_STORE):
            ms = min(_events_ms(torch, lambda: K.probe_copy_kernel(b.data_ptr(), a.data_ptr(), nbytes, grid, fl,
                                                                   cur.cuda_stream)))
            gbps = nbytes / ms / 1e6
            if gbps > best_k:
                best_k, best_grid, best_flags = gbps, grid, fl
    ms = min(_events_ms(torch, lambda: K.probe_memcpy(b.data_ptr(), a.data_ptr(), nbytes, cur.cuda_stream)))
    res["hbm_copy_kernel_gbps"] = round(best_k, 1)
    res["hbm_copy_kernel_grid"] = best_grid
    res["hbm_copy_kernel_flags"] = best_flags
    res["hbm_memcpy_d2d_gbps"] = round(nbytes / ms / 1e6, 1)
    res["hbm_copy_peak_gbps"] = max(res["hbm_copy_kernel_gbps"], res["hbm_memcpy_d2d_gbps"])
    # host link: read from each pinned host region of the pool into HBM
    link = []
    for r in range(run.pool.n_regions):
        info = run.pool.region_info(r)
        if info["type"] != K.REGION_HOST:
            continue
        n = min(nbytes, info["capacity_bytes"]) // 4096 * 4096
        src = info["device_ptr"]
        best, bgrid = 0.0, 0
        for grid in (32, 64, 128, 256, 512):
            ms = min(_events_ms(torch, lambda: K.probe_copy_kernel(b.data_ptr(), src, n, grid, 0, cur.cuda_stream),
                                iters=2))
            if n / ms / 1e6 > best:
                best, bgrid = n / ms / 1e6, grid
        ms = min(_events_ms(torch, lambda: K.probe_memcpy(b.data_ptr(), info["host_ptr"], n, cur.cuda_stream),
                            iters=2))
        link.append({"region": r, "numa_node": info["numa_node_actual"], "kernel_gbps": round(best, 2),
                     "kernel_grid": bgrid, "memcpy_h2d_gbps": round(n / ms / 1e6, 2)})
    res["host_link"] = link
    res["host_link_peak_gbps"] = max([max(x["kernel_gbps"], x["memcpy_h2d_gbps"]) for x in link] or [0.0])
    # GPU -> host direction (the store path): writes into a separate pinned buffer
    h = torch.empty(nbytes // 2, dtype=torch.int16, pin_memory=True)
    best, bgrid = 0.0, 0
    for grid in (8, 12, 16, 32):
        ms = min(_events_ms(torch, lambda: K.probe_copy_kernel(h.data_ptr(), b.data_ptr(), nbytes, grid,
                                                               K.LAUNCH_NT_STORE, cur.cuda_stream), iters=2))
        if nbytes / ms / 1e6 > best:
            best, bgrid = nbytes / ms / 1e6, grid
    ms = min(_events_ms(torch, lambda: K.probe_memcpy(h.data_ptr(), b.data_ptr(), nbytes, cur.cuda_stream), iters=2))
    res["d2h"] = {"kernel_gbps": round(best, 2), "kernel_grid": bgrid, "memcpy_d2h_gbps": round(nbytes / ms / 1e6, 2)}
    res["d2h_peak_gbps"] = max(res["d2h"]["kernel_gbps"], res["d2h"]["memcpy_d2h_gbps"])
    del a, b, h
    torch.cuda.empty_cache()
    return res


# rocprofv3 counter passes behind the PMC summaries in profiles/.  Each pass is one run of
#   rocprofv3 --pmc <counters> --output-format csv -d <dir>/<pass> -o <pass> -- python3 bench.py <args>
# (at most 4 TCC counters per pass on gfx950); then `python3 bench.py --summarize-pmc <dir>
# --tag <tag> --bench-args "<args>"` writes profiles/retrieve_<tag>_pmc.txt.
PMC_PASSES = [
    ("fetch", ["FETCH_SIZE"]),
    ("write", ["WRITE_SIZE"]),
    ("rd", ["TCC_EA0_RDREQ_DRAM_32B_sum", "TCC_EA0_RDREQ_IO_32B_sum", "TCC_EA0_RDREQ_GMI_32B_sum"]),
    ("wr", ["TCC_EA0_WRREQ_WRITE_DRAM_32B_sum", "TCC_EA0_WRREQ_WRITE_IO_32B_sum", "TCC_EA0_WRREQ_WRITE_GMI_32B_sum"]),
    ("req", ["TCC_EA0_RDREQ_sum", "TCC_EA0_RDREQ_32B_sum", "TCC_EA0_RDREQ_128B_sum", "TCC_BUBBLE_sum"]),
    ("utcl", ["TCP_UTCL1_TRANSLATION_MISS_sum", "TCP_UTCL1_TRANSLATION_HIT_sum",
              "TCP_UTCL1_STALL_UTCL2_REQ_OUT_OF_CREDITS_sum", "TCP_PENDING_STALL_CYCLES_sum", "GRBM_UTCL2_BUSY",
              "GRBM_GUI_ACTIVE"]),
    ("stall", ["TCC_EA0_WRREQ_STALL_sum", "TCC_EA0_WRREQ_DRAM_CREDIT_STALL_sum",
               "TCC_EA0_RDREQ_DRAM_CREDIT_STALL_sum", "TCC_TAG_STALL_sum"]),
    ("lat", ["TCC_EA0_RDREQ_LEVEL_sum", "TCC_EA0_WRREQ_LEVEL_sum", "TCC_EA0_WRREQ_sum", "GRBM_GUI_ACTIVE"]),
]
PROBE_COPY_BYTES = 4 << 30          # bytes one probe-copy dispatch of the bench reads and writes


def kernels_sha():
    import hashlib
    src = os.path.join(ROOT, "paper_2606_14779_amd", "csrc", "kernels.hip")
    return hashlib.sha256(open(src, "rb").read()).hexdigest()


def summarize_pmc(d, tag, bench_args, out_dir=None):
    """profiles/retrieve_<tag>_pmc.txt from the counter passes under d (one directory per pass).

    Per (kernel, workgroups): the mean per dispatch of every counter, and bytes:
      fetch_bytes / write_bytes  FETCH_SIZE / WRITE_SIZE (KiB) x 1024, each scaled so that the
                                 bench's 4 GiB probe copy reads / writes exactly 4 GiB;
      rd_* / wr_* _bytes         32 x the per-destination 32-byte request counts (dram = HBM,
                                 io = the host link, gmi = another die), unscaled."""
    import csv
    from collections import defaultdict
    vals = defaultdict(lambda: defaultdict(list))
    for name, counters in PMC_PASSES:
        path = os.path.join(d, name, name + "_counter_collection.csv")
        if not os.path.exists(path):
            continue
        for t in csv.DictReader(open(path)):
            k = t["Kernel_Name"].split("(")[0].replace("void ", "")
            if "at::native" in k:
                continue
            wg = int(t["Grid_Size"]) // max(1, int(t["Workgroup_Size"]))
            vals[(k, wg)][t["Counter_Name"]].append(float(t["Counter_Value"]))

    def mean(xs):
        return sum(xs) / len(xs)
    # calibration: the 4 GiB HBM copy sweep only (its grids), not the host-link, device-to-host or
    # same-bytes probes, whose sizes differ
    probe = [v for k, v in vals.items() if "probe_copy_kernel" in k[0] and k[1] in HBM_PROBE_GRIDS
             and "FETCH_SIZE" in v and "WRITE_SIZE" in v]
    fetch_scale = PROBE_COPY_BYTES / 1024 / mean([x for v in probe for x in v["FETCH_SIZE"]]) if probe else None
    write_scale = PROBE_COPY_BYTES / 1024 / mean([x for v in probe for x in v["WRITE_SIZE"]]) if probe else None
    short = {"TCC_EA0_RDREQ_DRAM_32B_sum": "rd_dram", "TCC_EA0_RDREQ_IO_32B_sum": "rd_io",
             "TCC_EA0_RDREQ_GMI_32B_sum": "rd_gmi", "TCC_EA0_WRREQ_WRITE_DRAM_32B_sum": "wr_dram",
             "TCC_EA0_WRREQ_WRITE_IO_32B_sum": "wr_io", "TCC_EA0_WRREQ_WRITE_GMI_32B_sum": "wr_gmi"}
    lines = ["# rocprofv3 PMC summary: KV store / retrieve kernels, %s" % tag,
             "# passes (repository root on the MI355X machine, after `cd /tmp && export TMPDIR=/tmp`), one run each:"]
    dn = os.path.normpath(d)   # the commands name the directory the passes were written to
    for name, counters in PMC_PASSES:
        lines.append("#   rocprofv3 --pmc %s --output-format csv -d %s/%s -o %s -- python3 bench.py %s"
                     % (" ".join(counters), dn, name, name, bench_args))
    lines += ["# then: python3 bench.py --summarize-pmc %s --tag %s --bench-args \"%s\""
              % (dn, tag, bench_args),
              "# Values are means per dispatch.  *_bytes = 32 x the 32-byte request counters, per destination",
              "# (dram: HBM; io: the host link; gmi: another die), unscaled.  fetch_bytes / write_bytes =",
              "# FETCH_SIZE / WRITE_SIZE x 1024 x the scale that makes the 4 GiB probe copy read / write 4 GiB.",
              "kernels_hip_sha256: %s" % kernels_sha(),
              "fetch_scale: %s" % ("%.6f" % fetch_scale if fetch_scale else "none"),
              "write_scale: %s" % ("%.6f" % write_scale if write_scale else "none")]
    for k in sorted(vals, key=lambda k: -mean(vals[k].get("FETCH_SIZE", [0.0]))):
        v = vals[k]
        f = ["workgroups=%d" % k[1], "dispatches=%d" % max(len(x) for x in v.values())]
        if "FETCH_SIZE" in v:
            f.append("fetch_size_kib=%.1f" % mean(v["FETCH_SIZE"]))
            if fetch_scale:
                f.append("fetch_bytes=%.0f" % (mean(v["FETCH_SIZE"]) * 1024 * fetch_scale))
        if "WRITE_SIZE" in v:
            f.append("write_size_kib=%.1f" % mean(v["WRITE_SIZE"]))
            if write_scale:
                f.append("write_bytes=%.0f" % (mean(v["WRITE_SIZE"]) * 1024 * write_scale))
        for c, sname in short.items():
            if c in v:
                f.append("%s_bytes=%.0f" % (sname, 32 * mean(v[c])))
        for c in sorted(v):
            if c not in short and c not in ("FETCH_SIZE", "WRITE_SIZE"):
                f.append("%s=%.0f" % (c.replace("_sum", ""), mean(v[c])))
        lines.append("kernel: %s | %s" % (k[0], " | ".join(f)))
    out = os.path.join(out_dir or os.path.join(ROOT, "profiles"), "retrieve_%s_pmc.txt" % tag)
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_trace(d, tag, bench_args, bench_json):
    """profiles/retrieve_<tag>_kernel_trace.md from a rocprofv3 --kernel-trace --stats run under d
    (output name kt) and the bench line that run printed (file bench_json)."""
    import csv
    from collections import defaultdict
    stats = list(csv.DictReader(open(os.path.join(d, "kt_kernel_stats.csv"))))
    trace = list(csv.DictReader(open(os.path.join(d, "kt_kernel_trace.csv"))))
    per = defaultdict(list)
    for t in trace:
        gx = int(t.get("Grid_Size_X") or t.get("Grid_Size"))
        wx = int(t.get("Workgroup_Size_X") or t.get("Workgroup_Size"))
        per[(t["Kernel_Name"], gx // max(1, wx))].append((int(t["End_Timestamp"]) - int(t["Start_Timestamp"])) / 1e6)
    out = ["# Kernel trace summary: %s" % tag, "",
           "Command (repository root on the MI355X machine, after `cd /tmp && export TMPDIR=/tmp`):", "",
           "    rocprofv3 --kernel-trace%s --stats --output-format csv -d %s -o kt -- python3 bench.py %s"
           % (" --memory-copy-trace" if os.path.exists(os.path.join(d, "kt_memory_copy_stats.csv")) else "",
              os.path.normpath(d), bench_args), "",
           "then `python3 bench.py --summarize-trace %s --tag %s --bench-args \"%s\" --bench-json <its "
           "JSON line>`." % (os.path.normpath(d), tag, bench_args), "",
           "kernels.hip sha256: `%s`" % kernels_sha(), "", "## rocprofv3 --stats", "",
           "| Kernel | Calls | Avg ms | Min ms | Max ms | % |", "|---|---:|---:|---:|---:|---:|"]
    for r in stats[:16]:
        out.append("| `%s` | %s | %.3f | %.3f | %.3f | %.2f |" % (
            r["Name"].split("(")[0].replace("void ", "")[:100], r["Calls"], float(r["AverageNs"]) / 1e6,
            float(r["MinNs"]) / 1e6, float(r["MaxNs"]) / 1e6, float(r["Percentage"])))
    out += ["", "## Per launch shape", "", "| Kernel | Workgroups | Dispatches | Avg ms | Min ms |",
            "|---|---:|---:|---:|---:|"]
    for (name, wg), ds in sorted(per.items(), key=lambda kv: -sum(kv[1]))[:16]:
        out.append("| `%s` | %d | %d | %.3f | %.3f |" % (name.split("(")[0].replace("void ", "")[:90], wg, len(ds),
                                                         sum(ds) / len(ds), min(ds)))
    mc_stats = os.path.join(d, "kt_memory_copy_stats.csv")
    if os.path.exists(mc_stats):   # a run with --memory-copy-trace as well
        out += ["", "## rocprofv3 --stats: memory copies", "", "| Direction | Calls | Avg ms | Min ms | Max ms |",
                "|---|---:|---:|---:|---:|"]
        for r in csv.DictReader(open(mc_stats)):
            out.append("| `%s` | %s | %.3f | %.3f | %.3f |" % (r["Name"], r["Calls"], float(r["AverageNs"]) / 1e6,
                                                           float(r["MinNs"]) / 1e6, float(r["MaxNs"]) / 1e6))
        mc = [(int(t["End_Timestamp"]) - int(t["Start_Timestamp"])) / 1e6
              for t in csv.DictReader(open(os.path.join(d, "kt_memory_copy_trace.csv")))]
        longc = sorted(x for x in mc if x >= 10.0)
        if longc:   # in a copy-engine run these are the whole ring slots (the trace records no sizes)
            out += ["", "Copies of at least 10 ms: %d, median %.3f ms." % (len(longc), longc[len(longc) // 2])]
    if bench_json and os.path.exists(bench_json):
        b = json.loads(open(bench_json).read().strip().splitlines()[-1])
        if "value" in b and "roofline" in b:
            rf = b.get("roofline") or {}
            ms = (rf.get("bytes_per_launch") or 0) / (rf.get("achieved") or 1) / 1e6
            out += ["", "## Bench line of the same run", "",
                    "    value %.2f GB/s, ms_per_step %.3f; dominant kernel %s: %.3f ms per launch (HIP events), "
                    "%s %s = %.4f of %s" % (b["value"], b["ms_per_step"], rf.get("kernel", "?").split(" ")[0], ms,
                                            rf.get("achieved"), rf.get("unit"), rf.get("frac") or 0, rf.get("peak"))]
        else:   # another mode's line (latency, duplex, ...): as printed
            out += ["", "## JSON line of the same run", "", "    " + json.dumps(b)]
    path = os.path.join(ROOT, "profiles", "retrieve_%s_kernel_trace.md" % tag)
    open(path, "w").write("\n".join(out) + "\n")
    print("\n".join(out))


def pmc_traffic(wl_name, kernel_prefix, profiles_dir=None):
    """Counter figures per dispatch of the first kernel matching kernel_prefix in the committed
    rocprofv3 PMC summary of this workload (profiles/retrieve_<workload>_pmc.txt).

    Returns None when there is no summary or when kernels.hip changed since the
    counters were taken (the summary records the source's sha256)."""
    path = os.path.join(profiles_dir or os.path.join(ROOT, "profiles"), "retrieve_%s_pmc.txt" % wl_name)
    if not os.path.exists(path):
        return None
    rec, sha = {}, None
    for line in open(path):
        if line.startswith("kernels_hip_sha256:"):
            sha = line.split(":", 1)[1].strip()
        elif line.startswith("kernel: ") and kernel_prefix in line and not rec:
            for f in line.split("|")[1:]:
                k, v = f.strip().split("=", 1)
                rec[k] = float(v)
    if sha != kernels_sha() or "fetch_bytes" not in rec or "write_bytes" not in rec:
        return None
    rec["source"] = os.path.relpath(path, ROOT) if profiles_dir is None else path
    return rec


def same_bytes_frac(pr, copied_gbps):
    """The HBM kernel's copied rate against the contiguous copy of the same byte count."""
    sb = pr.get("hbm_copy_same_bytes") if pr else None
    if not sb:
        return {}
    return {"measured_copy_peak_same_bytes": sb["gbps"], "frac_measured_same_bytes": round(copied_gbps / sb["gbps"], 4)}


def traffic_detail(tr, alg_read, alg_write):
    """The counter figures of one kernel beside its algorithmic bytes: HBM (DRAM) and host-link (IO)
    bytes read and written per dispatch, and FETCH_SIZE / WRITE_SIZE scaled and unscaled."""
    if not tr:
        return None
    out = {"algorithmic_read_bytes": round(alg_read), "algorithmic_write_bytes": round(alg_write),
           "fetch_bytes": round(tr["fetch_bytes"]), "write_bytes": round(tr["write_bytes"]),
           "fetch_size_kib_unscaled": tr.get("fetch_size_kib"), "write_size_kib_unscaled": tr.get("write_size_kib"),
           "source": tr["source"]}
    for k in ("rd_dram_bytes", "rd_io_bytes", "rd_gmi_bytes", "wr_dram_bytes", "wr_io_bytes", "wr_gmi_bytes"):
        if k in tr:
            out[k] = round(tr[k])
    return out


def measure_weights(torch, K, wl, file_dir=None):
    """Eq. 1 weights measured by the pool organizer: a pool of the workload's region kinds (1 GiB
    each) reads 256 MiB of every region into HBM with its class's kernel (a file region: 256 MiB
    written to a probe file beside it and read back); host regions share one host link, so their
    figure is divided by their count (KVP_MEASURE_SHARED_LINK), and file regions are read all at
    once, as a retrieve reads them (KVP_MEASURE_FILES_TOGETHER).  MB/s."""
    import tempfile
    regions = []
    for i, r in enumerate(wl.regions):
        if r.kind == "file":
            path = os.path.join(file_dir or tempfile.gettempdir(), "kvpool-measure-%d-%d.bin" % (os.getpid(), i))
            regions.append(K.Region("file", 1 << 30, -1, 0, path))
        else:
            regions.append(K.Region("host", 1 << 30, -1) if r.kind == "host" else K.Region("staging", 1 << 30))
    sh = wl.shape
    spec = K.KVSpec(sh.layers, sh.kv_heads, sh.head_dim, sh.block_size, sh.elem_bytes, wl.layout)
    with K.KVPool(regions, [1] * len(regions), spec, 0) as p:
        w = p.measure_bandwidth(256 << 20, K.MEASURE_SHARED_LINK | K.MEASURE_FILES_TOGETHER)
    torch.cuda.synchronize()
    return [int(x) for x in w]


def round_trip_ok(torch, run, wl):
    """Every present block's destination slot equals its source slot in every layer, and every
    slot no block names still holds the fill value (on the GPU, layer by layer)."""
    import numpy as np
    from paper_2606_14779_amd.runner import SENTINEL
    dev = run.dst.device
    touched = np.zeros(wl.dst_num_slots, bool)
    ok = True
    for q in wl.requests:
        ds = torch.from_numpy(q.dst_slots[:q.n_present].astype(np.int64)).to(dev)
        ss = torch.from_numpy(q.src_slots.astype(np.int64)).to(dev)
        touched[q.dst_slots[:q.n_present]] = True
        for l in range(wl.shape.layers):
            ok = ok and bool(torch.equal(run.dst[l].index_select(1, ds), run.src[l].index_select(1, ss)))
    rest = torch.from_numpy(np.flatnonzero(~touched).astype(np.int64)).to(dev)
    sent = int(np.uint16(SENTINEL).view(np.int16))
    if len(rest):
        for l in range(wl.shape.layers):
            ok = ok and bool((run.dst[l].index_select(1, rest) == sent).all())
    return ok


def host_facts():
    """CPU model, usable cores and NUMA layout of the machine the bench runs on."""
    facts = {"cpu_model": None, "cores_available": len(os.sched_getaffinity(0)), "numa_nodes": {}}
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                facts["cpu_model"] = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    base = "/sys/devices/system/node"
    try:
        for d in sorted(os.listdir(base)):
            if d.startswith("node") and d[4:].isdigit():
                cpus = open(os.path.join(base, d, "cpulist")).read().strip()
                mem_kb = None
                for line in open(os.path.join(base, d, "meminfo")):
                    if "MemTotal" in line:
                        mem_kb = int(line.split()[-2])
                facts["numa_nodes"][d[4:]] = {"cpus": cpus, "mem_gib": round(mem_kb / 2**20, 1) if mem_kb else None}
    except OSError:
        pass
    return facts


def cpu_baseline(run, wl, warmup=3, iters=10):
    """The oracle's gather (memcpy per chunk, unmodified) over the whole request on the host cores:
    the host regions are read where they are (pinned host memory), the staging regions (HBM) from a
    host mirror, into a host mirror of the whole paged cache with the request's own block table.
    Median and min of `iters` timed passes after `warmup`, on one thread and on T threads (the same
    function, each thread over its own slice of the blocks)."""
    import threading

    import numpy as np
    import oracle
    sh = wl.shape
    q = wl.requests[0]
    m = run.maps[q.request_id]
    n = q.n_present
    regions = []
    mirrors = []
    for r in range(len(wl.regions)):
        info = run.pool.region_info(r)
        if info["type"] == 0:
            regions.append(info["host_ptr"])
        else:                                    # whole staging region mirrored (its span for this request)
            offs = m["offset"][m["region"] == r]
            hi = int(offs.max()) + sh.block_bytes if len(offs) else 0
            buf = run.pool.region_read(r, 0, hi) if hi else np.zeros(16, np.uint8)
            mirrors.append(buf)
            regions.append(buf.ctypes.data)
    L = sh.layers
    dst = np.zeros((L, 2, wl.dst_num_slots, sh.kv_heads, sh.block_size, sh.head_dim), np.uint16)
    slots = q.dst_slots[:n].astype(np.int32)
    shape = (L, sh.kv_heads, sh.block_size, sh.head_dim, sh.elem_bytes)
    kd, vd = [dst[l, 0] for l in range(L)], [dst[l, 1] for l in range(L)]

    def one_thread():
        oracle.gather(m, slots, regions, kd, vd, shape, wl.layout)

    T = max(1, len(os.sched_getaffinity(0)))
    bounds = np.linspace(0, n, T + 1).astype(int)

    def t_threads():
        ts = [threading.Thread(target=oracle.gather,
                               args=(m[bounds[i]:bounds[i + 1]], slots[bounds[i]:bounds[i + 1]], regions, kd, vd,
                                     shape, wl.layout)) for i in range(T)]
        for t_ in ts:
            t_.start()
        for t_ in ts:
            t_.join()

    def timed(fn):
        for _ in range(warmup):
            fn()
        ms = []
        for _ in range(iters):
            t = time.perf_counter()
            fn()
            ms.append((time.perf_counter() - t) * 1e3)
        return ms

    nbytes = n * sh.block_bytes
    ms1 = timed(one_thread)
    msT = timed(t_threads)
    # the oracle's result is the retrieve's: spot-check it against the GPU destination
    import torch
    for b in (0, n // 2, n - 1):
        got = run.dst[:, :, int(slots[b])].cpu().numpy().view(np.uint16)
        assert np.array_equal(got, dst[:, :, int(slots[b])]), "oracle gather and GPU retrieve differ"
    del dst, mirrors

    def row(ms, cores):
        med = statistics.median(ms)
        return {"cores": cores, "ms_median": round(med, 2), "ms_min": round(min(ms), 2),
                "gbps_median": round(nbytes / med / 1e6, 3), "gbps_max": round(nbytes / min(ms) / 1e6, 3)}
    one, multi = row(ms1, 1), row(msT, T)
    return {"value": one["gbps_median"], "unit": "GB/s", "cores": 1, "kind": "oracle",
            "ms_per_request_median": one["ms_median"], "ms_per_request_min": one["ms_min"],
            "one_thread": one, "threads": multi,
            "sample": "the whole request: %d blocks (%.2f GiB), every host-region block read in place, every "
                      "staging block from a host mirror, into a host mirror of the %d-slot cache; %d warm-up and "
                      "%d timed passes per thread count" % (n, nbytes / 2**30, wl.dst_num_slots, warmup, iters),
            "note": "host-to-host copies: the oracle's destination is host memory, so no host link is crossed",
            "host": host_facts()}


def ablation(args):
    """Retrieval of the same request through differently organised pools (the
    paper's ablation of its orchestrator, Sec. 5.3, restated for this path):
    everything on one host region; striped over the two host regions only;
    all six regions with equal weights; the configured 4:4:1:1:1:1 striping;
    and weights measured by the pool organizer (per-region read probes, host
    regions sharing one link)."""
    import copy

    import torch

    from kvgen import workloads
    from paper_2606_14779_amd import kvpool as K
    from paper_2606_14779_amd.runner import WorkloadRun

    base = workloads.make(args.config)
    n = base.requests[0].n_present

    def variant(name, regions):
        wl = copy.deepcopy(base)
        wl.regions = regions
        workloads._size_regions(wl.regions, [q.n_present for q in wl.requests], wl.shape.block_bytes)
        run = WorkloadRun(wl, device=0)
        run.setup()
        counts = [int(x) for x in np.bincount(run.maps[wl.requests[0].request_id]["region"].astype(np.int64),
                                             minlength=len(regions))]
        ms = []
        for i in range(args.warmup + args.steps):
            torch.cuda.synchronize()
            t = time.perf_counter()
            run.retrieve_all()
            torch.cuda.synchronize()
            if i >= args.warmup:
                ms.append((time.perf_counter() - t) * 1e3)
        out = {"variant": name, "regions": [(r.kind, r.weight) for r in regions], "blocks": counts,
               "ms_median": round(statistics.median(ms), 3),
               "gbps": round(wl.retrieved_bytes / statistics.median(ms) / 1e6, 2)}
        measured = None
        if name.startswith("configured"):
            measured = [int(x) for x in run.pool.measure_bandwidth(256 << 20, K.MEASURE_SHARED_LINK)]
            out["measured_mbps_shared_link"] = measured
        run.close()
        torch.cuda.empty_cache()
        log(json.dumps(out))
        return out, measured

    import numpy as np
    R = workloads.RegionSpec
    res = []
    res.append(variant("single host region", [R("host", 1, 0)])[0])
    res.append(variant("two host regions 1:1", [R("host", 1, 0), R("host", 1, 1)])[0])
    res.append(variant("same regions, equal weights (striping without Eq. 1)",
                       [R(r.kind, 1, r.numa) for r in base.regions])[0])
    conf, measured = variant("configured 4:4:1:1:1:1", copy.deepcopy(base.regions))
    res.append(conf)
    mregions = [R(r.kind, int(w), r.numa) for r, w in zip(base.regions, measured)]
    res.append(variant("measured weights (shared host link)", mregions)[0])
    print(json.dumps({"metric": "retrieval ms of one request by pool organisation (ablation)",
                      "workload": base.name, "blocks": n, "retrieved_bytes": base.retrieved_bytes,
                      "steps": args.steps, "warmup": args.warmup, "variants": res}), flush=True)


def file_ablation(args):
    """The paper's ablation (Sec. 5.3) on the storage tier: the staging regions of the workload become
    file regions, and the same request is retrieved through
      - passthrough only: the whole request on one O_DIRECT file region, no striping;
      - orchestrator only: striped 4:4:1:1:1:1 over the host regions and four file regions that are
        read through the page cache (the file system's path; each file's cached pages are dropped
        before every retrieve, so the reads are cold);
      - full: the same striping over O_DIRECT file regions, with the configured weights and with
        weights the pool measures (files read together).
    Retrieve ms per call, median of --steps after --warmup; all file regions in --file-dir."""
    import copy
    import dataclasses

    import torch

    from kvgen import workloads
    from paper_2606_14779_amd import kvpool as K
    from paper_2606_14779_amd.runner import WorkloadRun

    torch.cuda.set_device(0)
    base = workloads.make(args.config)
    base.regions = [dataclasses.replace(r, kind="file") if r.kind == "staging" else r for r in base.regions]
    R = workloads.RegionSpec

    def drop_cached(paths):
        for path in paths:
            fd = os.open(path, os.O_RDONLY)
            try:
                os.fsync(fd)
                os.posix_fadvise(fd, 0, 0, os.POSIX_FADV_DONTNEED)
            finally:
                os.close(fd)

    def variant(name, regions, file_flags=0):
        wl = copy.deepcopy(base)
        wl.regions = regions
        workloads._size_regions(wl.regions, [q.n_present for q in wl.requests], wl.shape.block_bytes)
        run = WorkloadRun(wl, device=0, file_dir=args.file_dir, file_flags=file_flags)
        try:
            run.setup()
            counts = [int(x) for x in np.bincount(run.maps[wl.requests[0].request_id]["region"].astype(np.int64),
                                                 minlength=len(regions))]
            ms = []
            for i in range(args.warmup + args.steps):
                if file_flags & K.FILE_BUFFERED:
                    drop_cached(run.file_paths)
                torch.cuda.synchronize()
                t = time.perf_counter()
                run.retrieve_all()
                torch.cuda.synchronize()
                if i >= args.warmup:
                    ms.append((time.perf_counter() - t) * 1e3)
            out = {"variant": name, "regions": [(r.kind, r.weight) for r in regions], "blocks": counts,
                   "ms_median": round(statistics.median(ms), 1), "ms_min": round(min(ms), 1),
                   "gbps": round(wl.retrieved_bytes / statistics.median(ms) / 1e6, 2)}
        finally:
            run.close()
            torch.cuda.empty_cache()
        log(json.dumps(out))
        return out

    import numpy as np
    res = [variant("passthrough only: one O_DIRECT file region", [R("file", 1)]),
           variant("orchestrator only: striped, files through the page cache", copy.deepcopy(base.regions),
                   K.FILE_BUFFERED),
           variant("full: striped, O_DIRECT files, configured weights", copy.deepcopy(base.regions))]
    measured = measure_weights(torch, K, base, args.file_dir)
    res.append(variant("full: striped, O_DIRECT files, measured weights",
                       [dataclasses.replace(r, weight=int(w)) for r, w in zip(base.regions, measured)]))
    print(json.dumps({"metric": "retrieval ms of one request by pool organisation, storage tier (ablation)",
                      "workload": base.name + "-file", "retrieved_bytes": base.retrieved_bytes,
                      "file_device": "the machine's virtio block device (a VM disk, not an NVMe drive)",
                      "steps": args.steps, "warmup": args.warmup, "variants": res}), flush=True)


def host_staged(args):
    """The paper's host path on this machine (Sec. 4.3: the KV is read into host memory, then
    transferred to the GPU), for the host-region part of the request, against the zero-copy kernel on
    the same blocks.  CPU threads (all the process may use) gather the blocks -- each a contiguous
    block-sized range of its region -- into a pinned buffer, one slice at a time; each slice goes to
    HBM by an asynchronous copy as soon as it is gathered, so the next slice's gather overlaps it;
    then a scatter (torch index_copy_, one per layer and K/V) puts every chunk in its slot of the paged
    cache.  The HBM staging regions are left out: a CPU cannot read them.  The destination is then
    compared with the source slots on the GPU."""
    import ctypes

    import numpy as np
    import torch

    from kvgen import workloads
    from paper_2606_14779_amd import kvpool as K
    from paper_2606_14779_amd.runner import WorkloadRun

    torch.cuda.set_device(0)
    wl = workloads.make(args.config, context_tokens=args.context)
    if wl.layout != 0 or len(wl.requests) != 1:
        raise SystemExit("--host-staged takes a one-request head-major workload")
    sh = wl.shape
    bb, C, L2 = sh.block_bytes, sh.chunk_bytes, 2 * sh.layers
    run = WorkloadRun(wl, device=0)
    try:
        run.setup()
        q = wl.requests[0]
        m = run.retrieve_maps[q.request_id]
        host_idx = [i for i, r in enumerate(wl.regions) if r.kind == "host"]
        hb = np.nonzero(np.isin(m["region"], host_idx))[0]
        n = len(hb)
        base = {r: run.pool.region_info(r)["host_ptr"] for r in host_idx}
        src_ptr = [base[int(m["region"][b])] + int(m["offset"][b]) for b in hb]
        pinned = torch.empty(n * bb, dtype=torch.uint8, pin_memory=True)
        dev = torch.empty(n * bb, dtype=torch.uint8, device="cuda")
        pin0 = pinned.data_ptr()
        threads = len(os.sched_getaffinity(0))
        slices = 8
        import concurrent.futures as cf
        pool = cf.ThreadPoolExecutor(max_workers=threads)

        def gather(lo, hi):                        # blocks [lo, hi) into the pinned buffer
            step = max(1, (hi - lo + threads - 1) // threads)

            def part(a):
                for i in range(a, min(hi, a + step)):
                    ctypes.memmove(pin0 + i * bb, src_ptr[i], bb)
            list(pool.map(part, range(lo, hi, step)))

        bounds = [n * k // slices for k in range(slices + 1)]
        stream = torch.cuda.Stream()
        slot_idx = torch.as_tensor(q.dst_slots[hb].astype(np.int64), device="cuda")
        dst8 = run.dst.view(torch.uint8).view(L2, wl.dst_num_slots, C)
        buf3 = dev.view(n, L2, C)

        def scatter():
            with torch.cuda.stream(stream):
                for c in range(L2):
                    dst8[c].index_copy_(0, slot_idx, buf3[:, c, :])

        def pipelined():
            with torch.cuda.stream(stream):
                for k in range(slices):
                    lo, hi = bounds[k], bounds[k + 1]
                    gather(lo, hi)
                    dev[lo * bb:hi * bb].copy_(pinned[lo * bb:hi * bb], non_blocking=True)
            scatter()
            stream.synchronize()

        def wall(fn):
            torch.cuda.synchronize()
            t = time.perf_counter()
            fn()
            torch.cuda.synchronize()
            return (time.perf_counter() - t) * 1e3

        def h2d():
            with torch.cuda.stream(stream):
                dev.copy_(pinned, non_blocking=True)
            stream.synchronize()

        def scatter_sync():
            scatter()
            stream.synchronize()

        res = {"gather": [], "h2d": [], "scatter": [], "pipelined": []}
        for i in range(args.warmup + args.steps):
            run.fill_dst()
            g = wall(lambda: gather(0, n))
            t = wall(h2d)
            sc = wall(scatter_sync)
            run.fill_dst()
            pl = wall(pipelined)
            if i >= args.warmup:
                for k, v in (("gather", g), ("h2d", t), ("scatter", sc), ("pipelined", pl)):
                    res[k].append(v)
        # the destination after the last pipelined run: every host block's slot equals its source slot
        src8 = run.src.view(torch.uint8).view(L2, wl.src_num_slots, C)
        sidx = torch.as_tensor(q.src_slots[hb].astype(np.int64), device="cuda")
        ok = all(torch.equal(dst8[c].index_select(0, slot_idx), src8[c].index_select(0, sidx)) for c in range(L2))
        # the zero-copy kernel on the same blocks
        mh = m.copy()
        mh["region"][~np.isin(mh["region"], host_idx)] = K.ABSENT
        kp, vp = run.layer_ptrs(run.dst)
        cur = torch.cuda.current_stream()
        zc = []
        for i in range(args.warmup + args.steps):
            t = wall(lambda: run.pool.retrieve(mh, q.dst_slots, wl.dst_num_slots, kp, vp, cur.cuda_stream))
            if i >= args.warmup:
                zc.append(t)
        pool.shutdown()
        med = {k: round(statistics.median(v), 2) for k, v in res.items()}
        out = {"metric": "host-region part of one request: the paper's host path (CPU gather into pinned memory, "
                         "copy to HBM, scatter) against the zero-copy kernel",
               "workload": wl.name, "blocks": int(n), "bytes": int(n * bb), "cpu_threads": threads,
               "slices": slices, "cpu_gather_ms": med["gather"], "h2d_ms": med["h2d"],
               "scatter_ms": med["scatter"], "serial_ms": round(med["gather"] + med["h2d"] + med["scatter"], 2),
               "pipelined_ms": med["pipelined"], "zero_copy_kernel_ms": round(statistics.median(zc), 2),
               "verified": bool(ok), "steps": args.steps, "warmup": args.warmup}
        print(json.dumps(out), flush=True)
    finally:
        run.close()


def pipeline(args):
    """Layerwise pipelining (the paper's Sec. 2.2.1 and its blocked I/O time):
    layer l of the request is retrieved on one stream while a compute stream,
    waiting on layer l's completion event, runs a stand-in for that layer's
    work (a bf16 GEMM sized to take `c` ms).  Blocked I/O = total time minus
    the compute-only time: the part of the run during which only I/O proceeds."""
    import torch

    from kvgen import workloads
    from paper_2606_14779_amd import kvpool as K
    from paper_2606_14779_amd.runner import WorkloadRun

    wl = workloads.make(args.config)
    sh = wl.shape
    run = WorkloadRun(wl, device=0)
    if args.sdma:
        if args.copy_ring_mib:
            run.pool.set_copy_ring(args.copy_ring_mib << 20)
        run.pool.set_launch(K.CLASS_HOST, K.OP_RETRIEVE, 0, K.LAUNCH_SDMA)
    if args.staging_grid or args.staging_flags:   # also the ring kernel's shape with --sdma
        run.pool.set_launch(K.CLASS_STAGING, K.OP_RETRIEVE, args.staging_grid, args.staging_flags)
    if (args.host_grid or args.host_flags) and not args.sdma:
        run.pool.set_launch(K.CLASS_HOST, K.OP_RETRIEVE, args.host_grid, args.host_flags)
    run.setup()
    q = wl.requests[0]
    kp, vp = run.layer_ptrs(run.dst)
    m = run.retrieve_maps[q.request_id]
    io = torch.cuda.Stream()
    comp = torch.cuda.Stream()
    if args.stand_in == "gemm":          # compute-bound layer stand-in: bf16 8192^3 GEMM
        a = torch.randn(8192, 8192, dtype=torch.bfloat16, device="cuda")
        b = torch.randn(8192, 8192, dtype=torch.bfloat16, device="cuda").contiguous()

        def work():
            torch.mm(a, b)
    else:                                # HBM-bound stand-in (a decode step reading its KV): 1 GiB copy
        a = torch.empty(1 << 29, dtype=torch.int16, device="cuda")
        b = torch.empty_like(a)
        a.fill_(1)

        def work():
            b.copy_(a)

    def gemm_ms(reps):
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        s.record()
        for _ in range(reps):
            work()
        e.record()
        e.synchronize()
        return s.elapsed_time(e)
    gemm_ms(3)
    one = gemm_ms(20) / 20

    def run_once(reps, with_io=True, with_compute=True):
        evs = [torch.cuda.Event() for _ in range(sh.layers)]
        torch.cuda.synchronize()
        t = time.perf_counter()
        if with_io:
            with torch.cuda.stream(io):
                for l in range(sh.layers):
                    run.pool.retrieve_layers(m, q.dst_slots, wl.dst_num_slots, l, l + 1, kp, vp, io.cuda_stream)
                    evs[l].record(io)
        if with_compute:
            with torch.cuda.stream(comp):
                for l in range(sh.layers):
                    if with_io:
                        comp.wait_event(evs[l])
                    for _ in range(reps):
                        work()
        torch.cuda.synchronize()
        return (time.perf_counter() - t) * 1e3

    retrieve_only = statistics.median([run_once(0, True, False) for _ in range(3)])
    rows = []
    for target in (1.0, 4.0, 6.5, 10.0):
        reps = max(1, int(round(target / one)))
        compute_only = statistics.median([run_once(reps, False, True) for _ in range(2)])
        total = statistics.median([run_once(reps, True, True) for _ in range(3)])
        rows.append({"compute_ms_per_layer": round(compute_only / sh.layers, 3),
                     "compute_only_ms": round(compute_only, 2), "pipelined_total_ms": round(total, 2),
                     "blocked_io_ms": round(max(0.0, total - compute_only), 2),
                     "serial_sum_ms": round(compute_only + retrieve_only, 2)})
        log(json.dumps(rows[-1]))
    print(json.dumps({"metric": "blocked I/O time with layerwise pipelining (stand-in compute)",
                      "workload": wl.name, "layers": sh.layers, "retrieve_only_ms": round(retrieve_only, 2),
                      "host_transport": "copy engines" if args.sdma else "zero-copy kernel",
                      "staging_launch": {"grid": args.staging_grid or None, "flags": args.staging_flags},
                      "host_launch": {"grid": args.host_grid or None, "flags": args.host_flags},
                      "stand_in": "bf16 GEMM 8192^3" if args.stand_in == "gemm" else "1 GiB HBM copy",
                      "stand_in_ms": round(one, 3), "rows": rows}), flush=True)
    run.close()


def latency(args):
    """Call-to-complete time of small retrieves: the first n blocks of the request (striped over all
    regions) for n = 1 ... 1024, one call at a time with a host synchronisation after each.  This is
    the fixed cost per call that a fetch of a few blocks sees.  Calls with a small work list run as one
    launch with the list in the kernel arguments; --upload times them the way larger calls run (work
    list uploaded, one launch per region class)."""
    import torch

    from kvgen import workloads
    from paper_2606_14779_amd import kvpool as K
    from paper_2606_14779_amd.runner import WorkloadRun

    wl = workloads.make(args.config)
    run = WorkloadRun(wl, device=0)
    if args.sdma:
        run.pool.set_launch(K.CLASS_HOST, K.OP_RETRIEVE, 0, K.LAUNCH_SDMA)
    if args.upload:
        run.pool.set_launch(K.CLASS_HOST, K.OP_RETRIEVE, 0, (K.LAUNCH_SDMA if args.sdma else 0) | K.LAUNCH_UPLOAD)
    run.setup()
    q = wl.requests[0]
    kp, vp = run.layer_ptrs(run.dst)
    m = run.retrieve_maps[q.request_id]
    cur = torch.cuda.current_stream()
    bb = wl.shape.block_bytes
    rows = []
    for n in (1, 4, 16, 32, 64, 256, 1024):
        sub, table = m[:n].copy(), q.dst_slots[:n].copy()
        for _ in range(3):
            run.pool.retrieve(sub, table, wl.dst_num_slots, kp, vp, cur.cuda_stream)
        torch.cuda.synchronize()
        wall, span, enq = [], [], []
        for _ in range(20):
            s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            t = time.perf_counter()
            s.record(cur)
            run.pool.retrieve(sub, table, wl.dst_num_slots, kp, vp, cur.cuda_stream)
            te = time.perf_counter()
            e.record(cur)
            e.synchronize()
            wall.append((time.perf_counter() - t) * 1e6)
            enq.append((te - t) * 1e6)
            span.append(s.elapsed_time(e) * 1e3)
        w = statistics.median(wall)
        rows.append({"blocks": n, "bytes": n * bb, "call_to_complete_us": round(w, 1),
                     "enqueue_us": round(statistics.median(enq), 1),
                     "span_us": round(statistics.median(span), 1), "gbps": round(n * bb / w / 1e3, 2)})
        log(json.dumps(rows[-1]))
    print(json.dumps({"metric": "retrieve latency by request size (first n blocks, call to complete)",
                      "workload": wl.name, "host_transport": "copy engines" if args.sdma else "zero-copy kernel",
                      "small_call_launch": not args.upload, "rows": rows}), flush=True)
    run.close()


def decode(args):
    """Offload during decoding (Sec. 4.1.3: the KV caches of each decoding step form an offload set):
    the 128K request is placed and stored, then grows one block at a time -- kv_pool_extend by one
    block and kv_pool_store of that block, synchronised after each -- as an engine offloading every
    16 generated tokens would.  Reports host and call-to-complete time per step and where the new
    blocks land (Eq. 2 sends every one-block set to the region with the largest weight)."""
    import dataclasses

    import numpy as np
    import torch

    from kvgen import workloads
    from paper_2606_14779_amd import kvpool as K
    from paper_2606_14779_amd.runner import WorkloadRun

    base = workloads.make(3)
    n_steps = 256
    regions = [dataclasses.replace(r) for r in base.regions]
    workloads._size_regions(regions, [base.requests[0].n_present, 3 * n_steps], base.shape.block_bytes)
    wl = dataclasses.replace(base, regions=regions)
    run = WorkloadRun(wl, device=0)
    run.setup()
    q = wl.requests[0]
    kp, vp = run.layer_ptrs(run.src)
    cur = torch.cuda.current_stream()
    host_us, total_us, landed = [], [], []
    for i in range(n_steps):
        slot = np.array([q.src_slots[i % q.n_present]], np.int32)    # the new block's values: any source slot
        t = time.perf_counter()
        m = run.pool.extend(q.request_id, 1)
        run.pool.store(m, slot, wl.src_num_slots, kp, vp, cur.cuda_stream)
        th = time.perf_counter()
        torch.cuda.synchronize()
        host_us.append((th - t) * 1e6)
        total_us.append((time.perf_counter() - t) * 1e6)
        landed.append(int(m["region"][0]))
    counts = np.bincount(landed, minlength=len(regions))
    out = {"metric": "per-step offload while decoding: extend by one block + store it (call to complete)",
           "workload": wl.name, "steps": n_steps, "block_bytes": wl.shape.block_bytes,
           "host_us_median": round(statistics.median(host_us[8:]), 1),
           "call_to_complete_us_median": round(statistics.median(total_us[8:]), 1),
           "call_to_complete_us_p99": round(float(np.percentile(total_us[8:], 99)), 1),
           "blocks_per_region": counts.tolist(),
           "request_blocks_after": q.n_present + n_steps}
    print(json.dumps(out), flush=True)
    run.close()


def duplex(args):
    """The host link is full duplex: store (offload) one 128K LLaMA-shaped request while another is
    retrieved, on two streams, against each alone.  Two requests are placed in one pool with the
    128K workload's regions and weights (4:4:1:1:1:1), each with its own source and destination slots."""
    import dataclasses

    import numpy as np
    import torch

    from kvgen import workloads
    from paper_2606_14779_amd import kvpool as K
    from paper_2606_14779_amd.runner import WorkloadRun

    base = workloads.make(3)
    sh = base.shape
    n = base.requests[0].n_present
    regions = [dataclasses.replace(r) for r in base.regions]
    workloads._size_regions(regions, [n, n], sh.block_bytes)
    reqs = [workloads.RequestSpec(i + 1, n, n, np.arange(i * n, (i + 1) * n, dtype=np.int32),
                                  np.arange(i * n, (i + 1) * n, dtype=np.int32)) for i in range(2)]
    wl = workloads.Workload(3, base.name + "-x2", base.seed, sh, 0, regions, reqs, 2 * n, 2 * n)
    run = WorkloadRun(wl, device=0)
    if args.host_grid or args.host_flags:
        run.pool.set_launch(K.CLASS_HOST, K.OP_RETRIEVE, args.host_grid, args.host_flags)
    if args.store_grid or args.store_flags >= 0:
        run.pool.set_launch(K.CLASS_HOST, K.OP_STORE, args.store_grid,
                            args.store_flags if args.store_flags >= 0 else K.LAUNCH_NT_STORE)
    if args.sdma:
        run.pool.set_launch(K.CLASS_HOST, K.OP_RETRIEVE, 0, K.LAUNCH_SDMA)
    run.setup()
    kp_s, vp_s = run.layer_ptrs(run.src)
    kp_d, vp_d = run.layer_ptrs(run.dst)
    q1, q2 = wl.requests
    a, b = torch.cuda.Stream(), torch.cuda.Stream()

    def store(st):
        run.pool.store(run.maps[q1.request_id], q1.src_slots, wl.src_num_slots, kp_s, vp_s, st.cuda_stream)

    def retrieve(st):
        run.pool.retrieve_request(q2.request_id, q2.dst_slots, wl.dst_num_slots, kp_d, vp_d, st.cuda_stream)

    def timed(fn, reps):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        t = time.perf_counter()
        for _ in range(reps):
            fn()
        torch.cuda.synchronize()
        return (time.perf_counter() - t) / reps * 1e3

    reps = max(3, args.steps // 2)
    st_ms = timed(lambda: store(a), reps)
    rt_ms = timed(lambda: retrieve(b), reps)
    both_ms = timed(lambda: (store(a), retrieve(b)), reps)
    host_bytes = sum(int(np.isin(run.maps[q.request_id]["region"],
                                 [i for i, r in enumerate(wl.regions) if r.kind == "host"]).sum())
                     for q in (q1,)) * sh.block_bytes
    out = {"metric": "store and retrieve of two 128K-token requests at once (host link full duplex)",
           "workload": wl.name, "request_bytes": wl.requests[0].n_present * sh.block_bytes,
           "host_link_bytes_each_way": host_bytes,
           "store_alone_ms": round(st_ms, 2), "retrieve_alone_ms": round(rt_ms, 2),
           "both_ms": round(both_ms, 2), "serial_ms": round(st_ms + rt_ms, 2),
           "link_gbps_both_directions": round(2 * host_bytes / both_ms / 1e6, 2),
           "launch": {"retrieve": "copy engines" if args.sdma else
                      {"grid": args.host_grid or "library default: 12, 48 while a store is in flight"},
                      "store": "copy engines" if args.store_flags >= 0 and args.store_flags & K.LAUNCH_SDMA else
                      {"grid": args.store_grid or 12}}}
    print(json.dumps(out), flush=True)
    run.close()


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=3, help="workload 1..5 (3: the 128K LLaMA-shaped request)")
    ap.add_argument("--probe-gib", type=float, default=4.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-probes", action="store_true")
    ap.add_argument("--host-grid", type=int, default=0)
    ap.add_argument("--staging-grid", type=int, default=0)
    ap.add_argument("--host-flags", type=int, default=0)
    ap.add_argument("--store-grid", type=int, default=0, help="host-class store workgroups (0: library default)")
    ap.add_argument("--store-flags", type=int, default=-1, help="host-class store flags (-1: library default)")
    ap.add_argument("--staging-flags", type=int, default=0)
    ap.add_argument("--store-staging-grid", type=int, default=0,
                    help="staging-class store workgroups (0: library default)")
    ap.add_argument("--store-staging-flags", type=int, default=-1, help="staging-class store flags (-1: library default)")
    ap.add_argument("--coherence", type=int, default=0, help="0 default, 1 coherent, 2 non-coherent host memory")
    ap.add_argument("--layout", type=int, default=0, help="pool chunk layout: 0 head-major, 1 token-major (LDS)")
    ap.add_argument("--sdma", action="store_true",
                    help="retrieve the host class through the copy engines and an HBM ring instead of the zero-copy kernel")
    ap.add_argument("--copy-ring-mib", type=int, default=0, help="with --sdma: MiB per ring slot (0: library default)")
    ap.add_argument("--no-copy-engine", action="store_true", help="skip the copy-engine retrieve figure")
    ap.add_argument("--context", type=int, default=None,
                    help="workload 3 with this many tokens instead of 128K (e.g. 524288)")
    ap.add_argument("--batch", action="store_true",
                    help="retrieve all requests of the workload in one call (concatenated maps) per step")
    ap.add_argument("--decode", action="store_true",
                    help="instead of the bench line, time per-step offload (extend by one block + store)")
    ap.add_argument("--duplex", action="store_true",
                    help="instead of the bench line, store one request while retrieving another")
    ap.add_argument("--latency", action="store_true",
                    help="instead of the bench line, time single retrieves of the first 1 ... 1024 blocks")
    ap.add_argument("--upload", action="store_true",
                    help="with --latency: no small-call launch (upload the work list, one launch per class)")
    ap.add_argument("--flush", action="store_true",
                    help="overwrite 1 GiB before each timed step; ms_per_step is then the median event span")
    ap.add_argument("--stand-in", choices=["gemm", "copy"], default="gemm",
                    help="with --pipeline: the per-layer compute stand-in (compute-bound GEMM or HBM-bound copy)")
    ap.add_argument("--pipeline", action="store_true",
                    help="instead of the bench line, overlap per-layer retrieval with stand-in compute")
    ap.add_argument("--host-staged", action="store_true",
                    help="instead of the bench line, the paper's host path (CPU gather into pinned memory, copy "
                         "to HBM, scatter) against the zero-copy kernel on the request's host-region blocks")
    ap.add_argument("--ablation", action="store_true",
                    help="instead of the bench line, compare pool organisations on the same request "
                         "(with --file-regions: striping and direct I/O on the storage tier)")
    ap.add_argument("--measured-weights", action="store_true",
                    help="place with Eq. 1 weights measured by the pool (kv_pool_measure_bandwidth, host regions "
                         "sharing one link) instead of the workload's configured weights")
    ap.add_argument("--weights", default=None,
                    help="with --measured-weights: comma-separated weights measured by an earlier run (MB/s), used "
                         "instead of measuring again, so that repeated runs (profiler passes) place identically")
    ap.add_argument("--file-regions", action="store_true",
                    help="the workload's staging regions as file regions (O_DIRECT files, one worker per region)")
    ap.add_argument("--file-dir", default=None, help="with --file-regions: directory of the region files")
    ap.add_argument("--layerwise", action="store_true",
                    help="also time the request retrieved one layer per call (kv_pool_retrieve_layers)")
    ap.add_argument("--summarize-pmc", metavar="DIR", default=None,
                    help="write profiles/retrieve_<tag>_pmc.txt from the rocprofv3 counter passes under DIR")
    ap.add_argument("--summarize-trace", metavar="DIR", default=None,
                    help="write profiles/retrieve_<tag>_kernel_trace.md from a rocprofv3 kernel trace under DIR")
    ap.add_argument("--tag", default=None, help="with --summarize-*: the workload name in the summary's file name")
    ap.add_argument("--bench-args", default="", help="with --summarize-*: the bench arguments the runs used")
    ap.add_argument("--bench-json", default=None, help="with --summarize-trace: file holding that run's bench line")
    args = ap.parse_args()
    if args.summarize_pmc:
        summarize_pmc(args.summarize_pmc, args.tag, args.bench_args)
        return
    if args.summarize_trace:
        summarize_trace(args.summarize_trace, args.tag, args.bench_args, args.bench_json)
        return
    if args.gpus == 1 and args.ablation:
        file_ablation(args) if args.file_regions else ablation(args)
        return
    if args.gpus == 1 and args.host_staged:
        host_staged(args)
        return
    if args.gpus == 1 and args.pipeline:
        pipeline(args)
        return
    if args.gpus == 1 and args.latency:
        latency(args)
        return
    if args.gpus == 1 and args.duplex:
        duplex(args)
        return
    if args.gpus == 1 and args.decode:
        decode(args)
        return
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the retrieval path has no cross-GPU step; "
              "--gpus %d is not supported" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from kvgen import workloads
    from paper_2606_14779_amd import kvpool as K
    from paper_2606_14779_amd.runner import WorkloadRun

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    wl = workloads.make(args.config, layout=args.layout, context_tokens=args.context)
    sh = wl.shape
    if args.file_regions:     # the staging regions become file regions: the storage tier
        import dataclasses
        wl.regions = [dataclasses.replace(r, kind="file") if r.kind == "staging" else r for r in wl.regions]
        wl.name += "-file"
    measured = None
    if args.weights and not args.measured_weights:
        raise SystemExit("--weights gives measured weights: use it with --measured-weights")
    if args.measured_weights:
        if args.weights:
            measured = [int(x) for x in args.weights.split(",")]
            if len(measured) != len(wl.regions) or min(measured) <= 0:
                raise SystemExit("--weights needs one positive integer per region (%d)" % len(wl.regions))
        else:
            measured = measure_weights(torch, K, wl, args.file_dir)
        import dataclasses
        wl.regions = [dataclasses.replace(r, weight=int(w)) for r, w in zip(wl.regions, measured)]
        workloads._size_regions(wl.regions, [q.n_present for q in wl.requests], sh.block_bytes)
        wl.name += "-measured-weights"
        log("measured weights (MB/s, host regions sharing one link):", measured)
    log("workload", wl.name, "retrieved bytes", wl.retrieved_bytes)
    t = time.perf_counter()
    run = WorkloadRun(wl, device=0, coherence=args.coherence, file_dir=args.file_dir)
    t_create = time.perf_counter() - t
    if args.host_grid or args.host_flags:
        run.pool.set_launch(K.CLASS_HOST, K.OP_RETRIEVE, args.host_grid, args.host_flags)
    if args.sdma:        # retrieve only: the runtime copies device-to-host with a kernel of its own
        if args.copy_ring_mib:
            run.pool.set_copy_ring(args.copy_ring_mib << 20)
        run.pool.set_launch(K.CLASS_HOST, K.OP_RETRIEVE, 0, K.LAUNCH_SDMA)
    if args.staging_grid or args.staging_flags:
        run.pool.set_launch(K.CLASS_STAGING, K.OP_RETRIEVE, args.staging_grid, args.staging_flags)
    if args.store_staging_grid or args.store_staging_flags >= 0:
        run.pool.set_launch(K.CLASS_STAGING, K.OP_STORE, args.store_staging_grid, max(0, args.store_staging_flags))
    if args.store_grid or args.store_flags >= 0:     # the host-class store the line also times
        run.pool.set_launch(K.CLASS_HOST, K.OP_STORE, args.store_grid,
                            K.LAUNCH_NT_STORE if args.store_flags < 0 else args.store_flags)
    log("pool created in %.1f s" % t_create)
    t = time.perf_counter()
    run.fill_source()
    run.fill_dst()
    log("source filled in %.1f s" % (time.perf_counter() - t))
    t = time.perf_counter()
    run.place_all()
    t_place = time.perf_counter() - t
    run.pool.set_timing(True)
    t = time.perf_counter()
    run.store_all()
    torch.cuda.synchronize()
    store_wall = time.perf_counter() - t
    store_t = run.pool.last_timing() if len(wl.requests) == 1 else None
    log("placed in %.3f ms, stored in %.1f ms" % (t_place * 1e3, store_wall * 1e3))

    def kind_idx(kind):
        return [i for i, r in enumerate(wl.regions) if r.kind == kind]

    def blocks_of(kind):
        return sum(int(np.isin(run.maps[q.request_id]["region"], kind_idx(kind)).sum()) for q in wl.requests)

    host_blocks, stage_blocks, file_blocks = blocks_of("host"), blocks_of("staging"), blocks_of("file")
    host_bytes, stage_bytes = host_blocks * sh.block_bytes, stage_blocks * sh.block_bytes
    file_bytes = file_blocks * sh.block_bytes

    def only(q, kind):
        """The request's map with every block outside regions of this kind marked absent."""
        m = run.retrieve_maps[q.request_id].copy()
        m["region"][~np.isin(m["region"], kind_idx(kind))] = K.ABSENT
        return m

    cur = torch.cuda.current_stream()
    run.pool.set_timing(False)
    step = run.retrieve_batch if args.batch else run.retrieve_all
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: K retrieves back to back; the library records HIP events
    # around each kernel on the stream it runs on, summarised afterwards
    log("warm-up done; timing %d steps" % args.steps)
    # --flush: before each step, overwrite 1 GiB (more than the 256 MiB Infinity Cache plus the L2s)
    # on the same stream, so every step starts cold; the per-step event span then excludes the flush
    flush = torch.empty(1 << 29, dtype=torch.int16, device="cuda") if args.flush else None
    run.pool.set_timing(True)
    spans, enqueue_ms = [], []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        if flush is not None:
            flush.fill_(i)
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record(cur)
        tq = time.perf_counter()
        step()
        enqueue_ms.append((time.perf_counter() - tq) * 1e3)
        e.record(cur)
        spans.append((s, e))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    summ = run.pool.timing_summary()
    run.pool.set_timing(False)
    span_ms = [s.elapsed_time(e) for s, e in spans]
    ms_per_step = wall / args.steps * 1e3
    if flush is not None:        # the wall clock includes the flushes: rate per retrieve from the spans
        ms_per_step = statistics.median(span_ms)
        del flush
    gbps = wl.retrieved_bytes / (ms_per_step / 1e3) / 1e9
    host_avg = summ["host_ms_sum"] / summ["host_calls"] if summ["host_calls"] else None
    stage_avg = summ["staging_ms_sum"] / summ["staging_calls"] if summ["staging_calls"] else None

    # staging-side gather alone (HBM->HBM), from a map without the host blocks
    stage_only = None
    if stage_blocks and len(wl.requests) == 1:
        q = wl.requests[0]
        m = only(q, "staging")
        kp, vp = run.layer_ptrs(run.dst)
        for _ in range(args.warmup):
            run.pool.retrieve(m, q.dst_slots, wl.dst_num_slots, kp, vp, cur.cuda_stream)
        torch.cuda.synchronize()
        run.pool.set_timing(True)
        for _ in range(args.steps):
            run.pool.retrieve(m, q.dst_slots, wl.dst_num_slots, kp, vp, cur.cuda_stream)
        ss = run.pool.timing_summary()
        run.pool.set_timing(False)
        avg = ss["staging_ms_sum"] / ss["staging_calls"]
        stage_only = {"ms_avg": round(avg, 3), "ms_min": round(ss["staging_ms_min"], 3),
                      "copied_gbps": round(stage_bytes / (avg / 1e3) / 1e9, 1)}

    # zero-copy gather alone, from a map without the staging blocks (the link with nothing beside it)
    host_only = None
    if host_blocks and (stage_blocks or file_blocks) and len(wl.requests) == 1 and not args.sdma:
        q = wl.requests[0]
        m = only(q, "host")
        kp, vp = run.layer_ptrs(run.dst)
        for _ in range(args.warmup):
            run.pool.retrieve(m, q.dst_slots, wl.dst_num_slots, kp, vp, cur.cuda_stream)
        torch.cuda.synchronize()
        run.pool.set_timing(True)
        for _ in range(args.steps):
            run.pool.retrieve(m, q.dst_slots, wl.dst_num_slots, kp, vp, cur.cuda_stream)
        sh_ = run.pool.timing_summary()
        run.pool.set_timing(False)
        avg = sh_["host_ms_sum"] / sh_["host_calls"]
        host_only = {"ms_avg": round(avg, 3), "ms_min": round(sh_["host_ms_min"], 3),
                     "gbps": round(host_bytes / (avg / 1e3) / 1e9, 2)}

    log("timed region done: %.3f ms per retrieve" % ms_per_step)
    # the storage tier alone: the file regions' blocks retrieved and stored by themselves, call to
    # completion (the file reads and writes run inside the calls)
    file_tier = None
    if file_blocks and len(wl.requests) == 1:
        q = wl.requests[0]
        m = only(q, "file")
        kp, vp = run.layer_ptrs(run.dst)
        ks, vs = run.layer_ptrs(run.src)

        def wall(fn, reps):
            fn()
            torch.cuda.synchronize()
            t = time.perf_counter()
            for _ in range(reps):
                fn()
            torch.cuda.synchronize()
            return (time.perf_counter() - t) / reps * 1e3
        def together():   # the file regions read all at once by their workers, MB/s summed
            w = run.pool.measure_bandwidth(256 << 20, K.MEASURE_FILES_TOGETHER)
            return int(sum(int(x) for i, x in enumerate(w) if wl.regions[i].kind == "file"))
        # the disk's rate drifts within a run: probe it on both sides of the timed retrieves
        before = together()
        rt = wall(lambda: run.pool.retrieve(m, q.dst_slots, wl.dst_num_slots, kp, vp, cur.cuda_stream), args.steps)
        after = together()
        st = wall(lambda: run.pool.store(m[:q.n_present], q.src_slots, wl.src_num_slots, ks, vs, cur.cuda_stream),
                  max(1, args.steps // 2))
        probe = [int(x) for i, x in enumerate(run.pool.measure_bandwidth(256 << 20)) if wl.regions[i].kind == "file"]
        file_tier = {"bytes": file_bytes, "blocks": file_blocks,
                     "retrieve_alone_ms": round(rt, 2), "retrieve_alone_gbps": round(file_bytes / rt / 1e6, 3),
                     "store_alone_ms": round(st, 2), "store_alone_gbps": round(file_bytes / st / 1e6, 3),
                     "read_probe_mbps_per_region": probe,
                     "read_probe_together_mbps": [before, after],
                     "retrieve_vs_probe_together": round(file_bytes / rt / 1e3 / ((before + after) / 2), 3),
                     "files": "O_DIRECT files, one worker thread per region",
                     "device": "the machine's virtio block device (a VM disk, not an NVMe drive)"}
        log("file tier: retrieve %.1f ms, store %.1f ms" % (rt, st))
    # the timed steps' result: every present block of every request equals its source slot (round
    # trip, compared on the GPU layer by layer), every other slot still holds the fill value
    verified = round_trip_ok(torch, run, wl)
    log("round trip verified" if verified else "ROUND TRIP MISMATCH")
    # store (offload) direction: the same request written back into its placed ranges
    store = None
    if len(wl.requests) == 1:
        for _ in range(args.warmup):
            run.store_all()
        torch.cuda.synchronize()
        run.pool.set_timing(True)
        t = time.perf_counter()
        for _ in range(args.steps):
            run.store_all()
        torch.cuda.synchronize()
        st_ms = (time.perf_counter() - t) / args.steps * 1e3
        sm = run.pool.timing_summary()
        run.pool.set_timing(False)
        store = {"ms_per_store": round(st_ms, 3),
                 "gbps": round(wl.retrieved_bytes / st_ms / 1e6, 2),
                 "host_kernel_ms_avg": round(sm["host_ms_sum"] / sm["host_calls"], 3) if sm["host_calls"] else None,
                 "staging_kernel_ms_avg":
                     round(sm["staging_ms_sum"] / sm["staging_calls"], 3) if sm["staging_calls"] else None}
        log("store timed: %.3f ms" % st_ms)
        # the staging-class store alone (HBM -> HBM), from a map with only the staging blocks
        if stage_blocks:
            q = wl.requests[0]
            m = only(q, "staging")[:q.n_present]
            kp, vp = run.layer_ptrs(run.src)
            for _ in range(args.warmup):
                run.pool.store(m, q.src_slots, wl.src_num_slots, kp, vp, cur.cuda_stream)
            torch.cuda.synchronize()
            run.pool.set_timing(True)
            for _ in range(args.steps):
                run.pool.store(m, q.src_slots, wl.src_num_slots, kp, vp, cur.cuda_stream)
            ss = run.pool.timing_summary()
            run.pool.set_timing(False)
            avg = ss["staging_ms_sum"] / ss["staging_calls"]
            store["staging_alone"] = {"ms_avg": round(avg, 3), "ms_min": round(ss["staging_ms_min"], 3),
                                      "copied_gbps": round(stage_bytes / (avg / 1e3) / 1e9, 1)}
            log("staging store alone: %.3f ms" % avg)

    # layerwise retrieval (one call per layer, as an engine overlapping attention on layer l with the
    # fetch of layer l+1 would issue it): total time and per-layer completion spacing
    layerwise = None
    if args.layerwise and len(wl.requests) == 1:
        q = wl.requests[0]
        kp, vp = run.layer_ptrs(run.dst)
        m = run.retrieve_maps[q.request_id]
        tot = []
        per_layer = []
        for it in range(3):
            evs = [torch.cuda.Event(enable_timing=True) for _ in range(sh.layers + 1)]
            torch.cuda.synchronize()
            t = time.perf_counter()
            evs[0].record(cur)
            for l in range(sh.layers):
                run.pool.retrieve_layers(m, q.dst_slots, wl.dst_num_slots, l, l + 1, kp, vp, cur.cuda_stream)
                evs[l + 1].record(cur)
            torch.cuda.synchronize()
            tot.append((time.perf_counter() - t) * 1e3)
            per_layer += [evs[l].elapsed_time(evs[l + 1]) for l in range(sh.layers)]
        layerwise = {"calls_per_request": sh.layers, "ms_total_median": round(statistics.median(tot), 3),
                     "ms_per_layer_median": round(statistics.median(per_layer), 3),
                     "ms_per_layer_max": round(max(per_layer), 3)}
        log("layerwise done: %.3f ms" % statistics.median(tot))

    # the same request through the copy-engine transport (hipMemcpy into an HBM ring, ring kernel on the
    # caller's stream): the option that leaves every CU to compute running beside a retrieve.  Last
    # use of the pool's launch settings, so they need no restoring.
    copy_engine = None
    if host_blocks and not args.sdma and not args.no_copy_engine:
        run.pool.set_launch(K.CLASS_HOST, K.OP_RETRIEVE, 0, K.LAUNCH_SDMA)
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        t = time.perf_counter()
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        ce_ms = (time.perf_counter() - t) / args.steps * 1e3
        copy_engine = {"ms_per_step": round(ce_ms, 3), "gbps": round(wl.retrieved_bytes / ce_ms / 1e6, 2),
                       "ring": "2 x 1 GiB HBM"}
        log("copy-engine retrieve timed: %.3f ms" % ce_ms)

    pr = None if args.no_probes else probes(torch, K, run, int(args.probe_gib * 2**30) // 4096 * 4096,
                                            stage_bytes // max(1, len(wl.requests)))
    log("probes done")
    cpu = None if args.no_cpu_baseline else cpu_baseline(run, wl)
    if cpu:
        log("cpu baseline done")

    # copy form in the kernels' names (template argument 2): 0 plain chunks; 2 token-major chunks
    # through LDS, the library's default for every token-major kernel these figures cover
    kform = 0 if wl.layout == 0 else 2
    # the dominant kernel: the class whose kernel takes longer per step
    dominant_host = bool(host_blocks) and (not stage_blocks or (host_avg or 0.0) >= (stage_avg or 0.0))
    dominant_ms = host_avg if dominant_host else stage_avg
    # per launch: a step of a multi-request workload launches one kernel of each class per request,
    # so the algorithmic bytes of an average launch are the step's bytes over its launches
    host_per_launch = host_bytes * args.steps / summ["host_calls"] if summ["host_calls"] else host_bytes
    stage_per_launch = stage_bytes * args.steps / summ["staging_calls"] if summ["staging_calls"] else stage_bytes
    if dominant_host:
        achieved = host_per_launch / (dominant_ms / 1e3) / 1e9
        tr = pmc_traffic(wl.name, "host_region_copy<true, %d," % kform)
        roof = {"bound": "pcie", "kernel": "host_region_copy (zero-copy gather from pinned host regions)"
                if not args.sdma else "host class by copy engines (hipMemcpy into an HBM ring) + HBM ring scatter",
                "achieved": round(achieved, 2), "peak": PCIE5_X16_GBPS, "unit": "GB/s",
                "frac": round(achieved / PCIE5_X16_GBPS, 4),
                "traffic": round(tr["fetch_bytes"] + tr["write_bytes"]) if tr else None,
                "traffic_detail": traffic_detail(tr, host_per_launch, host_per_launch),
                "bytes_per_launch": round(host_per_launch),
                "launches_per_step": round(summ["host_calls"] / args.steps, 3),
                "measured_peak": pr["host_link_peak_gbps"] if pr else None,
                "frac_measured": round(achieved / pr["host_link_peak_gbps"], 4) if pr else None}
    else:
        achieved = 2 * stage_per_launch / (dominant_ms / 1e3) / 1e9
        trs = pmc_traffic(wl.name, "staging_region_copy<true, %d," % kform)
        copied = stage_per_launch / (dominant_ms / 1e3) / 1e9
        roof = {"bound": "hbm", "kernel": "staging_region_copy (HBM gather, beside the host-class kernel)",
                "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBPS, 4),
                "traffic": round(trs["fetch_bytes"] + trs["write_bytes"]) if trs else None,
                "traffic_detail": traffic_detail(trs, stage_per_launch, stage_per_launch),
                "bytes_per_launch": round(2 * stage_per_launch),
                "launches_per_step": round(summ["staging_calls"] / args.steps, 3),
                "copied_gbps": round(copied, 1),
                "measured_copy_peak": pr["hbm_copy_peak_gbps"] if pr else None,
                "frac_measured": round(copied / pr["hbm_copy_peak_gbps"], 4) if pr else None}
        roof.update(same_bytes_frac(pr, copied))
    hbm_roof = None
    if stage_only:
        a = 2 * stage_bytes / (stage_only["ms_avg"] / 1e3) / 1e9         # bytes read + written in HBM
        trs = pmc_traffic(wl.name, "staging_region_copy<true, %d," % kform)
        hbm_roof = {"bound": "hbm", "kernel": "staging_region_copy (HBM gather, alone)", "achieved": round(a, 1),
                    "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(a / HBM_PEAK_GBPS, 4),
                    "traffic": round(trs["fetch_bytes"] + trs["write_bytes"]) if trs else None,
                    "traffic_detail": traffic_detail(trs, stage_bytes, stage_bytes),
                    "algorithmic_bytes": 2 * stage_bytes,
                    "copied_gbps": stage_only["copied_gbps"],
                    "measured_copy_peak": pr["hbm_copy_peak_gbps"] if pr else None,
                    "frac_measured": round(stage_only["copied_gbps"] / pr["hbm_copy_peak_gbps"], 4) if pr else None}
        hbm_roof.update(same_bytes_frac(pr, stage_only["copied_gbps"]))

    store_staging_roof = None
    if store and store.get("staging_alone"):
        sa = store["staging_alone"]
        a = 2 * stage_bytes / (sa["ms_avg"] / 1e3) / 1e9
        trs = pmc_traffic(wl.name, "staging_region_copy<false, %d," % kform)
        store_staging_roof = {"bound": "hbm", "kernel": "staging_region_copy<false,...> (HBM store, alone)",
                              "achieved": round(a, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                              "frac": round(a / HBM_PEAK_GBPS, 4),
                              "traffic": round(trs["fetch_bytes"] + trs["write_bytes"]) if trs else None,
                              "traffic_detail": traffic_detail(trs, stage_bytes, stage_bytes),
                              "algorithmic_bytes": 2 * stage_bytes, "copied_gbps": sa["copied_gbps"],
                              "measured_copy_peak": pr["hbm_copy_peak_gbps"] if pr else None,
                              "frac_measured": round(sa["copied_gbps"] / pr["hbm_copy_peak_gbps"], 4) if pr else None}
        store_staging_roof.update(same_bytes_frac(pr, sa["copied_gbps"]))

    store_roof = None
    if store and host_blocks:
        a = host_bytes / (store["host_kernel_ms_avg"] / 1e3) / 1e9
        trw = pmc_traffic(wl.name, "host_region_copy<false, %d," % kform)
        store_roof = {"bound": "pcie", "kernel": "host_region_copy<false,...> (zero-copy store to pinned host regions)",
                      "achieved": round(a, 2), "peak": PCIE5_X16_GBPS, "unit": "GB/s",
                      "frac": round(a / PCIE5_X16_GBPS, 4),
                      "traffic": round(trw["fetch_bytes"] + trw["write_bytes"]) if trw else None,
                      "traffic_detail": traffic_detail(trw, host_bytes, host_bytes),
                      "measured_peak": pr["d2h_peak_gbps"] if pr else None,
                      "frac_measured": round(a / pr["d2h_peak_gbps"], 4) if pr else None}

    ideal_ms = None
    if pr:
        ideal_ms = max(host_bytes / (pr["host_link_peak_gbps"] * 1e9) if host_bytes else 0.0,
                       stage_bytes / (pr["hbm_copy_peak_gbps"] * 1e9) if stage_bytes else 0.0) * 1e3
    out = {
        "metric": "retrieved KV GB/s into HBM + retrieval ms per 128K-token request, LLaMA-8B shape",
        "value": round(gbps, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wl.name, "context_tokens": sum(q.n_blocks for q in wl.requests) * sh.block_size,
                   "blocks": wl.present_blocks, "block_bytes": sh.block_bytes,
                   "retrieved_bytes": wl.retrieved_bytes, "host_link_bytes": host_bytes,
                   "staging_bytes": stage_bytes,
                   "regions": [(r.kind, r.weight) for r in wl.regions],
                   "weights": ("measured by the pool: kv_pool_measure_bandwidth, 256 MiB per region (HBM: 1 GiB), "
                               "host regions sharing one link (MB/s)" + ("; from an earlier run (--weights)" if args.weights
                                                                    else "")) if measured else "configured",
                   "layout": "head-major chunks" if wl.layout == 0 else "token-major chunks",
                   "dst_slots": wl.dst_num_slots, "seed": wl.seed},
        "retrieval_ms": {"call_to_complete": round(ms_per_step, 3),
                         "span_median": round(statistics.median(span_ms), 3), "span_min": round(min(span_ms), 3),
                         "host_kernel_avg": round(host_avg, 3) if host_avg else None,
                         "staging_kernel_avg": round(stage_avg, 3) if stage_avg else None,
                         "ideal_at_measured_peaks": round(ideal_ms, 3) if ideal_ms else None,
                         "host_enqueue_median": round(statistics.median(enqueue_ms), 3)},
        "roofline": roof,
        "roofline_staging": hbm_roof,
        "host_alone": dict(host_only, frac_measured=round(host_only["gbps"] / pr["host_link_peak_gbps"], 4)
                           if pr else None) if host_only else None,
        "probes": pr,
        "store": store,
        "roofline_store": store_roof,
        "roofline_store_staging": store_staging_roof,
        "file_tier": file_tier,
        "layerwise": layerwise,
        "copy_engine_retrieve": copy_engine,
        "place_ms": round(t_place * 1e3, 3),
        "store_ms": round(store_wall * 1e3, 1),
        "store_kernels_ms": store_t,
        "cpu_baseline": cpu,
        "caches_flushed_per_step": bool(args.flush),
        "verified_round_trip": verified,
        "requests_per_call": len(wl.requests) if args.batch else 1,
        "launch": {"host_transport": "copy engines" if args.sdma else "zero-copy kernel",
                   "host_grid": args.host_grid or None, "staging_grid": args.staging_grid or None,
                   "host_flags": args.host_flags, "staging_flags": args.staging_flags,
                   "store_grid": args.store_grid or None,
                   "store_flags": None if args.store_flags < 0 else args.store_flags,
                   "store_staging_grid": args.store_staging_grid or None,
                   "store_staging_flags": None if args.store_staging_flags < 0 else args.store_staging_flags,
                   "coherence": args.coherence},
    }
    print(json.dumps(out), flush=True)
    run.close()


if __name__ == "__main__":
    main()
