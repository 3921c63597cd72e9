"""GPU parity of the KV-pool store / retrieve path against the CPU oracle.

All GPU work goes through the C ABI (``paper_2606_14779_amd.kvpool``).  The
bar is bit-exact: the path copies bf16 words and does no arithmetic.
"""
import numpy as np
import pytest

from kvgen import workloads
from paper_2606_14779_amd import kvpool as K
from paper_2606_14779_amd.runner import SENTINEL

from gpu_util import check_full, check_sampled, check_tags, make_run, oracle_pool, say, tag_cache

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def _run_and_check(wl, label, **kw):
    say("case", label, wl.describe()["workload"], "layout", wl.layout,
        "blocks", [q.n_present for q in wl.requests])
    run = make_run(wl, **kw)
    try:
        host = run.setup(keep_host=True)
        run.retrieve_all()
        torch.cuda.synchronize()
        check_full(wl, run, host)
    finally:
        run.close()


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("layout", [0, 1])
def test_parity_scaled_workloads(cfg, layout):
    wl = workloads.make(cfg, max_blocks=61, layout=layout)
    _run_and_check(wl, "scaled")


@pytest.mark.parametrize("grid,flags", [(1, 0), (7, K.LAUNCH_NT_LOAD | K.LAUNCH_NT_STORE),
                                        (4096, K.LAUNCH_NT_LOAD), (300, K.LAUNCH_NT_STORE),
                                        (64, K.LAUNCH_XCD), (96, K.LAUNCH_XCD | K.LAUNCH_SPLIT2),
                                        (12, K.LAUNCH_XCD), (65536, K.LAUNCH_SPLIT2 | K.LAUNCH_NT_LOAD),
                                        (7, K.LAUNCH_CHUNK_MAJOR), (65536, K.LAUNCH_CHUNK_MAJOR | K.LAUNCH_SPLIT2),
                                        (96, K.LAUNCH_CHUNK_MAJOR | K.LAUNCH_XCD | K.LAUNCH_SPLIT2),
                                        # per-class launches (the 45-block call would otherwise take the
                                        # small-call launch, which has no unit order of its own)
                                        (96, K.LAUNCH_XCD | K.LAUNCH_SPLIT2 | K.LAUNCH_UPLOAD),
                                        (7, K.LAUNCH_CHUNK_MAJOR | K.LAUNCH_UPLOAD),
                                        (5, K.LAUNCH_TILE | K.LAUNCH_UPLOAD),
                                        (65536, K.LAUNCH_TILE | K.LAUNCH_SPLIT2 | K.LAUNCH_UPLOAD),
                                        (96, K.LAUNCH_TILE | K.LAUNCH_XCD | K.LAUNCH_SPLIT2 | K.LAUNCH_UPLOAD),
                                        (1, K.LAUNCH_TILE | K.LAUNCH_NT_LOAD | K.LAUNCH_UPLOAD),
                                        # one unit per workgroup (the grid capped at the unit count)
                                        (1 << 20, K.LAUNCH_SPLIT2 | K.LAUNCH_NT_LOAD | K.LAUNCH_NT_STORE |
                                         K.LAUNCH_CHUNK_MAJOR | K.LAUNCH_UPLOAD),
                                        (1 << 20, K.LAUNCH_NT_LOAD | K.LAUNCH_NT_STORE | K.LAUNCH_UPLOAD)])
def test_parity_launch_shapes(grid, flags):
    wl = workloads.make(2, max_blocks=45)
    say("case launch", grid, flags)
    run = make_run(wl)
    try:
        for cls in (K.CLASS_HOST, K.CLASS_STAGING):
            for op in (K.OP_RETRIEVE, K.OP_STORE):
                run.pool.set_launch(cls, op, grid, flags)
        host = run.setup(keep_host=True)
        run.retrieve_all()
        torch.cuda.synchronize()
        check_full(wl, run, host)
    finally:
        run.close()


@pytest.mark.parametrize("flags", [0, K.LAUNCH_LDS, K.LAUNCH_LDS | K.LAUNCH_NT_LOAD,
                                   K.LAUNCH_LDS | K.LAUNCH_CHUNK_MAJOR, K.LAUNCH_CHUNK_MAJOR,
                                   K.LAUNCH_LDS | K.LAUNCH_TILE | K.LAUNCH_UPLOAD, K.LAUNCH_TILE | K.LAUNCH_UPLOAD])
def test_parity_token_major_lds(flags):
    wl = workloads.make(4, max_blocks=33, layout=1)
    say("case token-major", flags)
    run = make_run(wl)
    try:
        for cls in (K.CLASS_HOST, K.CLASS_STAGING):
            for op in (K.OP_RETRIEVE, K.OP_STORE):
                run.pool.set_launch(cls, op, 0, flags)
        host = run.setup(keep_host=True)
        run.retrieve_all()
        torch.cuda.synchronize()
        check_full(wl, run, host)
    finally:
        run.close()


def _custom(shape, regions, n, layout=0, dst_slots=None, src_slots=None, extra_slots=3, absent=()):
    """A one-request workload with an arbitrary shape (ragged chunk sizes)."""
    rng = np.random.default_rng(n * 31 + len(regions))
    src = rng.permutation(n + extra_slots)[:n].astype(np.int32) if src_slots is None else src_slots
    dslots = n + extra_slots
    dst = rng.permutation(dslots)[:n].astype(np.int32) if dst_slots is None else dst_slots
    req = workloads.RequestSpec(1, n, n, src, dst)
    wl = workloads.Workload(0, "custom", 77, shape, layout, regions, [req], n + extra_slots, dslots)
    workloads._size_regions(wl.regions, [n], shape.block_bytes)
    return wl


RAGGED = workloads.KVShape("ragged", 3, 3, 24)          # chunk 2304 B = 144 vectors: tail path


@pytest.mark.parametrize("layout", [0, 1])
@pytest.mark.parametrize("flags", [0, K.LAUNCH_LDS])
def test_parity_ragged_chunk(layout, flags):
    regions = [workloads.RegionSpec("host", 2, 0), workloads.RegionSpec("staging", 3),
               workloads.RegionSpec("host", 1, 1)]
    wl = _custom(RAGGED, regions, 29, layout)
    say("case ragged", layout, flags)
    run = make_run(wl)
    try:
        for cls in (0, 1):
            for op in (0, 1):
                run.pool.set_launch(cls, op, 5, flags)
        host = run.setup(keep_host=True)
        run.retrieve_all()
        torch.cuda.synchronize()
        check_full(wl, run, host)
    finally:
        run.close()


@pytest.mark.parametrize("kind", ["host", "staging"])
def test_single_block_single_region(kind):
    wl = _custom(workloads.LLAMA_8B, [workloads.RegionSpec(kind, 1, 0 if kind == "host" else -1)], 1)
    _run_and_check(wl, "n=1 N=1 " + kind)


def test_last_slot_and_full_region():
    """Destination slot num_slots-1 and a region filled to its last byte."""
    shape = workloads.KVShape("tiny", 2, 2, 64)
    bb = shape.block_bytes                                  # 16 KiB, sector multiple
    n = 6
    dst = np.array([5, 0, 3, 1, 4, 2], np.int32) + 2        # includes slot 7 = num_slots - 1
    wl = _custom(shape, [workloads.RegionSpec("staging", 1), workloads.RegionSpec("host", 1, 0)], n,
                 dst_slots=dst, extra_slots=2)
    for r in wl.regions:
        r.capacity_bytes = (n // 2) * bb                    # exactly full
    _run_and_check(wl, "last slot / full region")


def test_absent_entries_and_all_absent():
    wl = workloads.make(2, max_blocks=40)
    say("case absent")
    run = make_run(wl)
    try:
        host = run.setup(keep_host=True)
        q = wl.requests[0]
        m = run.retrieve_maps[q.request_id].copy()
        skip = np.arange(0, q.n_blocks, 3)
        m["region"][skip] = K.ABSENT
        kp, vp = run.layer_ptrs(run.dst)
        table = q.dst_slots.copy()
        table[skip] = -1                                     # never read for absent entries
        run.pool.retrieve(m, table, wl.dst_num_slots, kp, vp, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        got = run.dst.cpu().numpy().view(np.uint16)
        src = host
        for b in range(q.n_blocks):
            s = q.dst_slots[b]
            if b in set(skip.tolist()):
                assert np.all(got[:, :, s] == SENTINEL)
            else:
                assert np.array_equal(got[:, :, s], src[:, :, q.src_slots[b]])
        m["region"][:] = K.ABSENT                            # nothing to do, nothing launched
        run.pool.retrieve(m, table, wl.dst_num_slots, kp, vp, 0)
        torch.cuda.synchronize()
        # empty calls: zero-length arrays, and NULL map and table with n_blocks = 0
        import ctypes
        before = run.dst.cpu().numpy().copy()
        empty, no_slots = np.zeros(0, dtype=K.LOC_DTYPE), np.zeros(0, np.int32)
        run.pool.retrieve(empty, no_slots, wl.dst_num_slots, kp, vp, 0)
        run.pool.store(empty, no_slots, wl.src_num_slots, *run.layer_ptrs(run.src), 0)
        run.pool.retrieve_layers(empty, no_slots, wl.dst_num_slots, 2, 5, kp, vp, 0)
        assert K._lib.kv_pool_retrieve(run.pool._h, None, 0, None, wl.dst_num_slots, K._ptrs(kp), K._ptrs(vp),
                                       ctypes.c_void_p(0)) == 0
        torch.cuda.synchronize()
        assert np.array_equal(run.dst.cpu().numpy(), before)
    finally:
        run.close()


def test_errors_leave_destination_untouched():
    wl = workloads.make(2, max_blocks=20)
    say("case errors")
    run = make_run(wl)
    try:
        run.setup()
        q = wl.requests[0]
        kp, vp = run.layer_ptrs(run.dst)
        m = run.retrieve_maps[q.request_id]

        def code(fn, *a):
            with pytest.raises(K.KVPoolError) as ei:
                fn(*a)
            return ei.value.name

        bad = q.dst_slots.copy()
        bad[3] = wl.dst_num_slots
        assert code(run.pool.retrieve, m, bad, wl.dst_num_slots, kp, vp, 0) == "INVALID"
        dup = q.dst_slots.copy()
        dup[4] = dup[5]
        assert code(run.pool.retrieve, m, dup, wl.dst_num_slots, kp, vp, 0) == "INVALID"
        assert code(run.pool.retrieve, m, dup, 1 << 24, kp, vp, 0) == "INVALID"   # far more slots than blocks
        dup = q.dst_slots.copy()
        dup[-1] = dup[0]
        assert code(run.pool.retrieve, m, dup, wl.dst_num_slots, kp, vp, 0) == "INVALID"
        mm = m.copy()
        mm["region"][2] = 17
        assert code(run.pool.retrieve, mm, q.dst_slots, wl.dst_num_slots, kp, vp, 0) == "INVALID"
        mm = m.copy()
        mm["offset"][2] += 16                                 # not a block boundary
        assert code(run.pool.retrieve, mm, q.dst_slots, wl.dst_num_slots, kp, vp, 0) == "STALE"
        mm = m.copy()
        mm["gen"][1] += 1
        assert code(run.pool.retrieve, mm, q.dst_slots, wl.dst_num_slots, kp, vp, 0) == "STALE"
        kp2 = list(kp)
        kp2[1] += 8
        assert code(run.pool.retrieve, m, q.dst_slots, wl.dst_num_slots, kp2, vp, 0) == "INVALID"
        same = m.copy()
        same[1] = same[0]
        assert code(run.pool.store, same, q.src_slots, wl.src_num_slots, *run.layer_ptrs(run.src), 0) == "INVALID"
        same = m.copy()
        same[9] = same[0]                                     # other regions' entries in between
        assert code(run.pool.store, same, q.src_slots, wl.src_num_slots, *run.layer_ptrs(run.src), 0) == "INVALID"
        # the smallest call whose unit count would not fit 32 bits: refused before its map is read
        import ctypes
        L = wl.shape.layers
        too_many = (1 << 32) // (4 * L)
        rc = K._lib.kv_pool_retrieve(run.pool._h, m.ctypes.data, too_many, q.dst_slots.ctypes.data,
                                     wl.dst_num_slots, K._ptrs(kp), K._ptrs(vp), ctypes.c_void_p(0))
        assert K.ERRORS[rc] == "INVALID" and b"too large" in K._lib.kv_pool_last_error()
        torch.cuda.synchronize()
        got = run.dst.cpu().numpy().view(np.uint16)
        assert np.all(got == SENTINEL)                        # no failed call touched it
        run.pool.release(q.request_id)
        assert code(run.pool.retrieve, m, q.dst_slots, wl.dst_num_slots, kp, vp, 0) == "STALE"
    finally:
        run.close()


def test_release_and_reuse():
    """A released range is reused by the next placement; old maps turn stale."""
    wl = workloads.make(1, max_blocks=16)
    say("case reuse")
    run = make_run(wl)
    try:
        host = run.setup(keep_host=True)
        q = wl.requests[0]
        old = run.maps[q.request_id].copy()
        run.pool.release(q.request_id)
        new = run.pool.place(q.request_id, q.n_present)
        assert np.array_equal(new["offset"], old["offset"]) and int(new["gen"][0]) == int(old["gen"][0]) + 1
        run.maps[q.request_id] = new
        run.retrieve_maps[q.request_id] = new
        run.store_all()
        run.fill_dst()
        run.retrieve_all()
        torch.cuda.synchronize()
        ora = oracle_pool(wl)                                # same history: place, release
        ora.place(q.request_id, q.n_present)
        assert ora.release(q.request_id) == 0
        check_full(wl, run, host, ora)
    finally:
        run.close()


def test_release_waits_for_a_retrieve_in_flight():
    """Release a request while its retrieve runs on another stream, then place a new request over the
    same ranges and store other values there at once: release waits for the retrieve, so the
    destination holds the original values."""
    from gpu_util import oracle_expectation
    wl = workloads.make(2, max_blocks=300)
    say("case release in flight")
    run = make_run(wl)
    try:
        host = run.setup(keep_host=True)
        q = wl.requests[0]
        kp, vp = run.layer_ptrs(run.dst)
        a = torch.cuda.Stream()
        a.wait_stream(torch.cuda.current_stream())
        run.pool.retrieve_request(q.request_id, q.dst_slots, wl.dst_num_slots, kp, vp, a.cuda_stream)
        run.pool.release(q.request_id)                       # returns once the retrieve is done
        new = run.pool.place(q.request_id + 1, q.n_present)
        assert set(zip(new["region"].tolist(), new["offset"].tolist())) == \
            set(zip(run.maps[q.request_id]["region"].tolist(), run.maps[q.request_id]["offset"].tolist()))
        run.src.bitwise_not_()                               # other values, then stored over the same bytes
        run.pool.store(new, q.src_slots, wl.src_num_slots, *run.layer_ptrs(run.src),
                       torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        _, _, expect = oracle_expectation(wl, run, host)
        assert np.array_equal(run.dst.cpu().numpy().view(np.uint16), expect)
    finally:
        run.close()


SMALL = workloads.KVShape("small", 4, 2, 64)           # 16 KiB blocks


@pytest.mark.parametrize("transport", ["staging", "sdma"])
def test_release_waits_for_every_reader_on_other_streams(transport):
    """Two retrieves of one request on two streams, the first held back behind torch's bounded spin
    kernel so that the second finishes first.  Neither takes the host-link kernel's turn (staging
    regions only, or host regions through the copy engines), so only the request's own completion
    event orders them.  Then release, place a new request over the same ranges and store other
    values there: release waits for both retrieves, so both destinations hold the oracle's values."""
    from gpu_util import oracle_expectation
    kind = "staging" if transport == "staging" else "host"
    regions = [workloads.RegionSpec(kind, 1, -1), workloads.RegionSpec(kind, 1, -1)]
    wl = _custom(SMALL, regions, 40)
    say("case release waits for every reader", transport)
    run = make_run(wl)
    try:
        host = run.setup(keep_host=True)
        if transport == "sdma":
            run.pool.set_launch(K.CLASS_HOST, K.OP_RETRIEVE, 0, K.LAUNCH_SDMA)
        q = wl.requests[0]
        cur = torch.cuda.current_stream()
        second = torch.full_like(run.dst, int(np.uint16(SENTINEL).view(np.int16)))
        a, b = torch.cuda.Stream(), torch.cuda.Stream()
        a.wait_stream(cur)
        b.wait_stream(cur)
        with torch.cuda.stream(a):
            torch.cuda._sleep(100_000_000)                   # bounded spin: 0.05-1 s
        run.pool.retrieve_request(q.request_id, q.dst_slots, wl.dst_num_slots, *run.layer_ptrs(run.dst),
                                  a.cuda_stream)
        run.pool.retrieve_request(q.request_id, q.dst_slots, wl.dst_num_slots, *run.layer_ptrs(second),
                                  b.cuda_stream)
        run.pool.release(q.request_id)                       # returns once both retrieves are done
        new = run.pool.place(q.request_id + 1, q.n_present)
        assert set(zip(new["offset"].tolist(), new["region"].tolist())) == \
            set(zip(run.maps[q.request_id]["offset"].tolist(), run.maps[q.request_id]["region"].tolist()))
        run.src.bitwise_not_()
        run.pool.store(new, q.src_slots, wl.src_num_slots, *run.layer_ptrs(run.src), cur.cuda_stream)
        torch.cuda.synchronize()
        _, _, expect = oracle_expectation(wl, run, host)
        assert np.array_equal(run.dst.cpu().numpy().view(np.uint16), expect), "held-back reader got other bytes"
        assert np.array_equal(second.cpu().numpy().view(np.uint16), expect)
    finally:
        run.close()


def test_destroy_waits_for_a_retrieve_in_flight():
    """Destroy the pool while a retrieve runs on another stream: destroy waits for the work on its
    requests before freeing the regions, and the retrieve completes intact."""
    from gpu_util import oracle_expectation
    wl = workloads.make(2, max_blocks=300)
    say("case destroy in flight")
    run = make_run(wl)
    try:
        host = run.setup(keep_host=True)
        q = wl.requests[0]
        kp, vp = run.layer_ptrs(run.dst)
        a = torch.cuda.Stream()
        a.wait_stream(torch.cuda.current_stream())
        run.pool.retrieve_request(q.request_id, q.dst_slots, wl.dst_num_slots, kp, vp, a.cuda_stream)
        run.pool.close()                                     # returns once the retrieve is done
        torch.cuda.synchronize()
        _, _, expect = oracle_expectation(wl, run, host)
        assert np.array_equal(run.dst.cpu().numpy().view(np.uint16), expect)
    finally:
        run.close()


def test_store_then_retrieve_across_streams():
    """A retrieve on another stream, enqueued right after the store, waits for it."""
    wl = workloads.make(3, max_blocks=200)
    say("case cross-stream")
    run = make_run(wl)
    try:
        host = run.fill_source(keep_host=True)
        run.fill_dst()
        run.place_all()
        torch.cuda.synchronize()
        a, b = torch.cuda.Stream(), torch.cuda.Stream()
        run.store_all(stream=a)
        run.retrieve(wl.requests[0], stream=b)               # no host synchronisation in between
        torch.cuda.synchronize()
        check_full(wl, run, host)
    finally:
        run.close()


@pytest.mark.parametrize("sdma", [False, True])
def test_batch_of_requests_in_one_call(sdma):
    """The four requests of workload 5 (absent tails included) retrieved by one call."""
    wl = workloads.make(5, max_blocks=70)
    say("case batch in one call", "copy engines" if sdma else "kernel")
    run = make_run(wl)
    try:
        if sdma:
            run.pool.set_launch(K.CLASS_HOST, K.OP_RETRIEVE, 0, K.LAUNCH_SDMA)
        host = run.setup(keep_host=True)
        run.retrieve_batch()
        torch.cuda.synchronize()
        check_full(wl, run, host)
    finally:
        run.close()


@pytest.mark.parametrize("sdma", [False, True])
def test_store_waits_for_retrieve_on_other_stream(sdma):
    """Write after read across streams: a store of new values into a request's
    blocks, enqueued on another stream right after a retrieve of the old ones,
    must wait for it; a retrieve after that store sees the new values."""
    wl = workloads.make(1, max_blocks=100)                 # 200 MiB over the host link: ~4 ms each way
    say("case store-after-retrieve", "copy engines" if sdma else "kernel")
    run = make_run(wl)
    try:
        if sdma:
            run.pool.set_copy_ring(64 << 20)
            for op in (K.OP_RETRIEVE, K.OP_STORE):
                run.pool.set_launch(K.CLASS_HOST, op, 0, K.LAUNCH_SDMA)
        run.fill_source()
        run.place_all()
        q = wl.requests[0]
        n = q.n_present
        kp_src, vp_src = run.layer_ptrs(run.src)
        kp_dst, vp_dst = run.layer_ptrs(run.dst)
        src_slots = torch.from_numpy(q.src_slots.astype(np.int64)).cuda()
        v1 = run.src[:, :, src_slots].clone()
        v2 = v1 ^ 0x5A5A                                      # different values, same shape
        a, b, c = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
        torch.cuda.synchronize()
        m = run.maps[q.request_id]
        d1 = np.arange(n, dtype=np.int32)                     # two disjoint destination ranges
        d2 = np.arange(n, 2 * n, dtype=np.int32)
        dst = torch.full((wl.shape.layers, 2, 2 * n) + tuple(run.dst.shape[3:]), 0, dtype=torch.int16,
                         device="cuda")
        kp2 = [dst[l, 0].data_ptr() for l in range(wl.shape.layers)]
        vp2 = [dst[l, 1].data_ptr() for l in range(wl.shape.layers)]
        run.pool.store(m, q.src_slots, wl.src_num_slots, kp_src, vp_src, a.cuda_stream)
        run.pool.retrieve(m, d1, 2 * n, kp2, vp2, b.cuda_stream)
        with torch.cuda.stream(c):                            # new source values, then the store on c
            c.wait_stream(a)                                  # (the source buffer itself is the caller's)
            run.src[:, :, src_slots] = v2
        run.pool.store(m, q.src_slots, wl.src_num_slots, kp_src, vp_src, c.cuda_stream)
        run.pool.retrieve(m, d2, 2 * n, kp2, vp2, a.cuda_stream)
        torch.cuda.synchronize()
        assert torch.equal(dst[:, :, :n], v1), "the retrieve saw values stored after it"
        assert torch.equal(dst[:, :, n:], v2), "the later retrieve missed the later store"
    finally:
        run.close()


def test_timing_reports_both_classes():
    wl = workloads.make(2, max_blocks=64)
    run = make_run(wl)
    try:
        run.setup()
        run.pool.set_timing(True)
        run.retrieve_all()
        t = run.pool.last_timing()
        m = run.maps[1]
        n_host = int(np.sum(np.isin(m["region"], [0, 1])))
        assert t["host_blocks"] == n_host and t["staging_blocks"] == len(m) - n_host
        assert t["host_ms"] > 0 and t["staging_ms"] > 0
    finally:
        run.close()


def test_probes_copy_exactly():
    n = 64 << 20
    src = torch.randint(-32768, 32767, (n // 2,), dtype=torch.int16, device="cuda")
    dst = torch.zeros_like(src)
    K.probe_copy_kernel(dst.data_ptr(), src.data_ptr(), n - 48, 0, 0, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert torch.equal(dst[:(n - 48) // 2], src[:(n - 48) // 2]) and bool((dst[(n - 48) // 2:] == 0).all())
    host = torch.empty(n // 2, dtype=torch.int16, pin_memory=True)
    K.probe_memcpy(host.data_ptr(), src.data_ptr(), n, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert torch.equal(host, src.cpu())


# ---- full-size workloads, in the launch configuration the bench times

@pytest.mark.parametrize("cfg,layout", [(1, 0), (2, 0), (3, 0), (4, 0), (5, 0), (3, 1), (4, 1)])
def test_full_size_workloads(cfg, layout):
    """Every workload at full size in its default launch configuration (the one the bench times),
    and the two 128K-token workloads with a token-major pool (the LDS-staged conversion)."""
    wl = workloads.make(cfg, layout=layout)
    say("case full-size", wl.name, "layout", layout, "bytes", wl.retrieved_bytes)
    run = make_run(wl)
    try:
        run.setup()
        run.retrieve_all()
        torch.cuda.synchronize()
        check_sampled(wl, run)
    finally:
        run.close()
        torch.cuda.empty_cache()


@pytest.mark.parametrize("layout", [0, 1])
def test_full_size_128k_every_block_against_the_oracle(layout):
    """The 128K-token LLaMA-shaped request at full size (8192 blocks, 16 GiB): the pool bytes of
    every block against the oracle's store, and every destination slot by round trip."""
    wl = workloads.make(3, layout=layout)
    say("case full-size every block", wl.name, "layout", layout)
    run = make_run(wl)
    try:
        host = run.setup(keep_host=True)
        run.retrieve_all()
        torch.cuda.synchronize()
        from gpu_util import check_every_block
        check_every_block(wl, run, host)
        del host
    finally:
        run.close()
        torch.cuda.empty_cache()


# ---- layer-range retrieve / store (layerwise pipelining)

def test_retrieve_layer_by_layer_and_subrange():
    wl = workloads.make(2, max_blocks=37)
    say("case layers")
    run = make_run(wl)
    try:
        host = run.setup(keep_host=True)
        q = wl.requests[0]
        kp, vp = run.layer_ptrs(run.dst)
        m = run.retrieve_maps[q.request_id]
        L = wl.shape.layers
        s = torch.cuda.current_stream().cuda_stream
        for l in range(L):                                   # one call per layer
            run.pool.retrieve_layers(m, q.dst_slots, wl.dst_num_slots, l, l + 1, kp, vp, s)
        torch.cuda.synchronize()
        check_full(wl, run, host)
        run.fill_dst()
        kp_part = [p if 3 <= l < 7 else 0 for l, p in enumerate(kp)]   # pointers outside the range unused
        vp_part = [p if 3 <= l < 7 else 0 for l, p in enumerate(vp)]
        run.pool.retrieve_layers(m, q.dst_slots, wl.dst_num_slots, 3, 7, kp_part, vp_part, s)
        torch.cuda.synchronize()
        from gpu_util import oracle_expectation
        _, _, expect = oracle_expectation(wl, run, host)
        got = run.dst.cpu().numpy().view(np.uint16)
        assert np.array_equal(got[3:7], expect[3:7])
        assert np.all(got[:3] == SENTINEL) and np.all(got[7:] == SENTINEL)
        for lo, hi in [(0, 0), (5, 4), (0, L + 1)]:
            with pytest.raises(K.KVPoolError) as ei:
                run.pool.retrieve_layers(m, q.dst_slots, wl.dst_num_slots, lo, hi, kp, vp, s)
            assert ei.value.name == "INVALID"
    finally:
        run.close()


@pytest.mark.parametrize("layout", [0, 1])
def test_store_in_layer_groups_then_retrieve(layout):
    wl = workloads.make(4, max_blocks=29, layout=layout)
    say("case store layers", layout)
    run = make_run(wl)
    try:
        host = run.fill_source(keep_host=True)
        run.fill_dst()
        run.place_all()
        q = wl.requests[0]
        kp, vp = run.layer_ptrs(run.src)
        s = torch.cuda.current_stream().cuda_stream
        L = wl.shape.layers
        for lo, hi in [(0, 5), (5, 6), (6, L)]:
            run.pool.store_layers(run.maps[q.request_id], q.src_slots, wl.src_num_slots, lo, hi, kp, vp, s)
        run.retrieve_all()
        torch.cuda.synchronize()
        check_full(wl, run, host)
    finally:
        run.close()


def test_measured_bandwidths_drive_placement():
    """Pool organizer from measurement: rates are positive, HBM staging reads
    beat the host link, the shared-link flag splits the host figure and the
    shared-HBM flag the staging figure (each by the number of such regions),
    and a pool created without bandwidths places exactly as the oracle does
    with the weights it measured."""
    regions = [K.Region("host", 64 << 20, -1), K.Region("host", 64 << 20, -1), K.Region("staging", 64 << 20),
               K.Region("staging", 64 << 20)]
    spec = K.KVSpec(2, 2, 64)
    with K.KVPool(regions, [1, 1, 1, 1], spec, 0) as p:
        alone = p.measure_bandwidth(32 << 20)
        shared = p.measure_bandwidth(32 << 20, K.MEASURE_SHARED_LINK | K.MEASURE_SHARED_HBM)
        say("measured MB/s", alone.tolist(), shared.tolist())
        assert np.all(alone > 1000) and min(alone[2:]) > max(alone[:2])
        for r in range(4):
            assert 0.3 < shared[r] / alone[r] < 0.7
    with K.KVPool(regions, None, spec, 0) as p:
        bw = [p.region_info(i)["bandwidth"] for i in range(4)]
        assert all(b > 1000 for b in bw)
        import oracle
        ora = oracle.Pool(bw, [r.capacity_bytes for r in regions], spec.block_bytes)
        assert np.array_equal(p.place(1, 300), ora.place(1, 300))


@pytest.mark.parametrize("sdma", [False, True])
def test_concurrent_retrieves_from_threads(sdma):
    """store/retrieve may be called from several threads on different streams
    (with the copy-engine option, all of them share the pool's ring)."""
    import threading
    wl = workloads.make(5, max_blocks=80)
    say("case threads", "copy engines" if sdma else "kernel")
    run = make_run(wl)
    try:
        if sdma:
            run.pool.set_copy_ring(32 << 20)          # a few 1.5 MiB blocks a slot: many slot reuses
            for op in (K.OP_RETRIEVE, K.OP_STORE):
                run.pool.set_launch(K.CLASS_HOST, op, 0, K.LAUNCH_SDMA)
        host = run.setup(keep_host=True)
        streams = [torch.cuda.Stream() for _ in wl.requests]
        cur = torch.cuda.current_stream()
        for s in streams:
            s.wait_stream(cur)
        errs = []

        def work(i, q):
            try:
                for _ in range(3):                           # idempotent: same blocks, same slots
                    run.retrieve(q, streams[i])
            except Exception as e:                           # reported below
                errs.append(e)

        ts = [threading.Thread(target=work, args=(i, q)) for i, q in enumerate(wl.requests)]
        for t in ts:
            t.start()
        for t in ts:
            t.join()
        torch.cuda.synchronize()
        assert not errs, errs
        check_full(wl, run, host)
    finally:
        run.close()


def test_retrieve_request_by_id_errors():
    wl = workloads.make(1, max_blocks=8)
    run = make_run(wl)
    try:
        run.setup()
        q = wl.requests[0]
        kp, vp = run.layer_ptrs(run.dst)
        for req, n, name in [(99, q.n_blocks, "NOTFOUND"), (q.request_id, q.n_blocks - 1, "INVALID")]:
            with pytest.raises(K.KVPoolError) as ei:
                run.pool.retrieve_request(req, q.dst_slots[:n], wl.dst_num_slots, kp, vp, 0)
            assert ei.value.name == name
    finally:
        run.close()


def test_allocation_failure_reports_nomem_and_cleans_up():
    """A staging region larger than HBM fails with NOMEM; the regions already
    allocated are released (a following normal pool still fits)."""
    spec = K.KVSpec(2, 2, 64)
    free_before = torch.cuda.mem_get_info()[0]
    with pytest.raises(K.KVPoolError) as ei:
        K.KVPool([K.Region("staging", 1 << 30), K.Region("staging", 1 << 46)], [1, 1], spec, 0)
    assert ei.value.name == "NOMEM"
    # the failed allocation leaves no HIP error behind for the caller's next launch check
    assert int(torch.full((16,), 3, device="cuda").sum()) == 48
    torch.cuda.synchronize()
    assert torch.cuda.mem_get_info()[0] >= free_before - (64 << 20)
    with K.KVPool([K.Region("staging", 1 << 30)], [1], spec, 0) as p:
        assert p.region_info(0)["device_ptr"]


def test_binding_docstring_example_runs():
    """The round trip shown in KVPool's docstring runs as printed and checks itself."""
    import textwrap
    doc = K.KVPool.__doc__
    code = doc.split("::", 1)[1].split("\n\n    Options:", 1)[0]
    exec(compile(textwrap.dedent(code), "KVPool docstring", "exec"), {})
    torch.cuda.empty_cache()


@pytest.mark.parametrize("sdma", [False, True])
def test_many_regions(sdma):
    """40 regions of both types with random weights: per-region bookkeeping, runs and placement at width."""
    rng = np.random.default_rng(40)
    regions = [workloads.RegionSpec("host" if i % 2 == 0 else "staging", int(rng.integers(1, 9)),
                                    0 if i % 2 == 0 else -1) for i in range(40)]
    shape = workloads.KVShape("many", 4, 2, 64)
    wl = _custom(shape, regions, 300)
    say("case many regions", "copy engines" if sdma else "kernel")
    run = make_run(wl)
    try:
        if sdma:
            run.pool.set_copy_ring(1 << 20)                  # 32 blocks of 32 KiB a slot: many batches
            for op in (K.OP_RETRIEVE, K.OP_STORE):
                run.pool.set_launch(K.CLASS_HOST, op, 0, K.LAUNCH_SDMA)
        host = run.setup(keep_host=True)
        run.retrieve_all()
        torch.cuda.synchronize()
        check_full(wl, run, host)
        counts = np.bincount(run.maps[1]["region"].astype(np.int64), minlength=40)
        assert (counts > 0).sum() >= 35                      # the stripe reaches nearly every region
    finally:
        run.close()


def _hip_last_error():
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipPeekAtLastError.restype = ctypes.c_int
    return hip.hipPeekAtLastError()


@pytest.mark.parametrize("n", [24, 160])
@pytest.mark.parametrize("grid", [0, 12])
def test_retrieve_while_store_in_flight(n, grid):
    """A retrieve enqueued while a host-class store is running (the library then widens a default
    read grid; an explicit one is kept), then a retrieve of the request being stored, which must
    wait for that store.  Both against the oracle; no HIP error is left for the caller."""
    import dataclasses
    base = workloads.make(2, max_blocks=n)
    regions = [dataclasses.replace(r) for r in base.regions]
    workloads._size_regions(regions, [n, n], base.shape.block_bytes)
    reqs = [workloads.RequestSpec(i + 1, n, n, np.arange(i * n, (i + 1) * n, dtype=np.int32)[::-1].copy(),
                                  np.random.default_rng(i).permutation(2 * n)[:n].astype(np.int32))
            for i in range(2)]
    reqs[1] = dataclasses.replace(reqs[1], dst_slots=np.setdiff1d(np.arange(2 * n), reqs[0].dst_slots)[:n]
                                  .astype(np.int32))
    wl = workloads.Workload(2, base.name + "-x2", base.seed, base.shape, 0, regions, reqs, 2 * n, 2 * n)
    say("case duplex", n, grid)
    run = make_run(wl)
    try:
        if grid:
            run.pool.set_launch(K.CLASS_HOST, K.OP_RETRIEVE, grid, 0)
        host = run.setup(keep_host=True)
        q1, q2 = wl.requests
        kp_s, vp_s = run.layer_ptrs(run.src)
        kp_d, vp_d = run.layer_ptrs(run.dst)
        cur = torch.cuda.current_stream()
        a, b = torch.cuda.Stream(), torch.cuda.Stream()
        a.wait_stream(cur)
        b.wait_stream(cur)
        run.pool.store(run.maps[q1.request_id], q1.src_slots, wl.src_num_slots, kp_s, vp_s, a.cuda_stream)
        run.pool.retrieve_request(q2.request_id, q2.dst_slots, wl.dst_num_slots, kp_d, vp_d, b.cuda_stream)
        run.pool.retrieve_request(q1.request_id, q1.dst_slots, wl.dst_num_slots, kp_d, vp_d, b.cuda_stream)
        assert _hip_last_error() == 0
        cur.wait_stream(a)
        cur.wait_stream(b)
        torch.cuda.synchronize()
        check_full(wl, run, host)
    finally:
        run.close()


def test_store_batch_and_retrieve_into_very_many_slots():
    """The four requests of workload 5 stored again in ONE call (several allocations per region in
    one map), then retrieved with a destination slot count far above the blocks moved (the
    duplicate check then sorts instead of using a bitmap); against the oracle."""
    wl = workloads.make(5, max_blocks=40)
    say("case store batch")
    run = make_run(wl)
    try:
        host = run.setup(keep_host=True)
        maps = np.concatenate([run.maps[q.request_id] for q in wl.requests])
        src = np.concatenate([q.src_slots for q in wl.requests]).astype(np.int32)
        run.pool.store(maps, src, wl.src_num_slots, *run.layer_ptrs(run.src), torch.cuda.current_stream().cuda_stream)
        kp, vp = run.layer_ptrs(run.dst)
        for q in wl.requests:
            run.pool.retrieve(run.retrieve_maps[q.request_id], q.dst_slots, 1 << 24, kp, vp,
                              torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        check_full(wl, run, host)
    finally:
        run.close()


@pytest.mark.parametrize("transport", ["small", "upload", "sdma"])
@pytest.mark.parametrize("layout", [0, 1])
def test_extended_request_round_trip(layout, transport):
    """A request placed, then extended three times (an offload set per decoding step); each set is
    stored as it arrives and the whole request is retrieved by id.  Maps, pool bytes and destination
    against the oracle carrying the same place / extend history.  With the copy engines, each
    region holds the request in several ranges, so its blocks cross the link in several runs."""
    import dataclasses

    import oracle
    sizes = [23, 1, 5, 11]
    n = sum(sizes)
    base = workloads.make(2, max_blocks=n, layout=layout)
    regions = [dataclasses.replace(r) for r in base.regions]
    workloads._size_regions(regions, [n, n], base.shape.block_bytes)    # room for several sets
    q = base.requests[0]
    wl = workloads.Workload(2, base.name + "-ext", base.seed, base.shape, layout, regions, [q],
                            base.src_num_slots, base.dst_num_slots)
    say("case extend", layout, transport, sizes)
    run = make_run(wl)
    try:
        if transport == "upload":
            run.pool.set_launch(K.CLASS_HOST, K.OP_STORE, 0, K.LAUNCH_NT_STORE | K.LAUNCH_UPLOAD)
            run.pool.set_launch(K.CLASS_HOST, K.OP_RETRIEVE, 0, (K.LAUNCH_LDS if layout else 0) | K.LAUNCH_UPLOAD)
        elif transport == "sdma":
            run.pool.set_copy_ring(64 << 20)
            for op in (K.OP_STORE, K.OP_RETRIEVE):
                run.pool.set_launch(K.CLASS_HOST, op, 0, K.LAUNCH_SDMA)
        host = run.fill_source(keep_host=True)
        run.fill_dst()
        sh = wl.shape
        L = sh.layers
        ora = oracle.Pool([r.weight for r in regions], [r.capacity_bytes for r in regions], sh.block_bytes)
        kp_s, vp_s = run.layer_ptrs(run.src)
        s = torch.cuda.current_stream().cuda_stream
        sets, first = [], 0
        for k, m in enumerate(sizes):
            lm = run.pool.place(q.request_id, m) if k == 0 else run.pool.extend(q.request_id, m)
            om = ora.place(q.request_id, m) if k == 0 else ora.extend(q.request_id, m)
            assert np.array_equal(lm.view(np.uint8), om.view(np.uint8)), "set %d placed differently" % k
            run.pool.store(lm, q.src_slots[first:first + m], wl.src_num_slots, kp_s, vp_s, s)
            sets.append(om)
            first += m
        whole = np.concatenate(sets)
        assert np.array_equal(run.pool.lookup(q.request_id, n), whole)
        kp, vp = run.layer_ptrs(run.dst)
        run.pool.retrieve_request(q.request_id, q.dst_slots, wl.dst_num_slots, kp, vp, s)
        torch.cuda.synchronize()
        shape = (L, sh.kv_heads, sh.block_size, sh.head_dim, sh.elem_bytes)
        oregions = [np.zeros(r.capacity_bytes, np.uint8) for r in regions]
        oracle.store(whole, q.src_slots, oregions, [host[l, 0] for l in range(L)], [host[l, 1] for l in range(L)],
                     shape, layout)
        expect = np.full(tuple(run.dst.shape), SENTINEL, np.uint16)
        oracle.gather(whole, q.dst_slots, oregions, [expect[l, 0] for l in range(L)],
                      [expect[l, 1] for l in range(L)], shape, layout)
        for r in range(len(regions)):
            offs = whole["offset"][whole["region"] == r]
            if len(offs):
                lo, hi = int(offs.min()), int(offs.max()) + sh.block_bytes
                assert np.array_equal(run.pool.region_read(r, lo, hi - lo), oregions[r][lo:hi]), "region %d" % r
        got = run.dst.cpu().numpy().view(np.uint16)
        assert np.array_equal(got, expect)
        run.pool.release(q.request_id)
    finally:
        run.close()


@pytest.mark.parametrize("two_streams", [False, True])
def test_back_to_back_upload_calls(two_streams):
    """One call per layer for 300 blocks -- too many for the kernel arguments, so every call uploads
    its work list -- issued back to back: from the second call on the caller's stream is still
    busy and the upload goes ahead on the pool's stream.  Against the oracle."""
    wl = workloads.make(2, max_blocks=300)
    say("case back-to-back uploads", two_streams)
    run = make_run(wl)
    try:
        host = run.setup(keep_host=True)
        q = wl.requests[0]
        kp, vp = run.layer_ptrs(run.dst)
        m = run.retrieve_maps[q.request_id]
        cur = torch.cuda.current_stream()
        streams = [torch.cuda.Stream(), torch.cuda.Stream()] if two_streams else [cur]
        for s_ in streams:
            s_.wait_stream(cur)
        for l in range(wl.shape.layers):
            run.pool.retrieve_layers(m, q.dst_slots, wl.dst_num_slots, l, l + 1, kp, vp,
                                     streams[l % len(streams)].cuda_stream)
        for s_ in streams:
            cur.wait_stream(s_)
        torch.cuda.synchronize()
        check_full(wl, run, host)
    finally:
        run.close()


@pytest.mark.parametrize("layout", [0, 1])
def test_tagged_pattern_localises_every_vector(layout):
    """Independent of the oracle: with every source vector tagged with its own coordinates, each
    destination vector must carry (source slot of its block, its own layer, K/V, head, token,
    vector index); a wrong one is reported by what it holds instead."""
    wl = workloads.make(2, max_blocks=61, layout=layout)
    say("case tagged", layout)
    run = make_run(wl)
    try:
        sh = wl.shape
        L, H, bs, D = sh.layers, sh.kv_heads, sh.block_size, sh.head_dim
        tags = tag_cache(L, wl.src_num_slots, H, bs, D)
        run.src.copy_(torch.from_numpy(tags))
        run.fill_dst()
        run.place_all()
        run.store_all()
        run.retrieve_all()
        torch.cuda.synchronize()
        q = wl.requests[0]
        check_tags(tags, run.dst.cpu().numpy(), q.src_slots[:q.n_present], q.dst_slots[:q.n_present],
                   np.int16(np.uint16(SENTINEL).view(np.int16)))
    finally:
        run.close()


def test_upload_ring_wraps_under_four_streams():
    """The 32-slot work-list ring wrapped five times by 160 upload-path calls of four requests on four
    streams, with no host synchronisation: a slot is reused only after the call that last read it."""
    wl = workloads.make(5, max_blocks=40)
    say("case ring wrap", [q.n_present for q in wl.requests])
    run = make_run(wl)
    try:
        run.pool.set_launch(K.CLASS_HOST, K.OP_RETRIEVE, 0, K.LAUNCH_UPLOAD)
        host = run.setup(keep_host=True)
        for _ in range(40):
            run.retrieve_all()
        torch.cuda.synchronize()
        check_full(wl, run, host)
    finally:
        run.close()


@pytest.mark.parametrize("elem_bytes", [1, 4])
@pytest.mark.parametrize("layout", [0, 1])
def test_other_element_sizes(elem_bytes, layout):
    """fp8-sized (1 byte) and fp32-sized (4 bytes) KV elements: the path copies bytes, so any element
    size whose chunks and (token-major) rows are 16-byte multiples works.  Random bytes, a mixed pool,
    a random table with absent entries; against the oracle byte for byte."""
    import oracle
    L, H, bs, D, n = 4, 8, 16, 128, 50
    spec = K.KVSpec(L, H, D, bs, elem_bytes, layout)
    bb = spec.block_bytes
    weights = [3, 2, 1]
    caps = [((w * n // sum(weights) + 2) * bb + 4095) // 4096 * 4096 for w in weights]
    regions = [K.Region("host", caps[0], 0), K.Region("staging", caps[1]), K.Region("host", caps[2], 0)]
    say("case element size", elem_bytes, layout)
    rng = np.random.default_rng(77 + elem_bytes * 3 + layout)
    S = n + 7
    row = D * elem_bytes
    src_h = rng.integers(0, 256, size=(L, 2, S, H, bs, row), dtype=np.uint8)
    src_slots = rng.permutation(S)[:n].astype(np.int32)
    dst_slots = rng.permutation(S)[:n].astype(np.int32)
    dev = torch.device("cuda", 0)
    src = torch.from_numpy(src_h).to(dev)
    dst = torch.zeros((L, 2, S, H, bs, row), dtype=torch.uint8, device=dev)
    kp = lambda t: [t[l, 0].data_ptr() for l in range(L)]           # noqa: E731
    vp = lambda t: [t[l, 1].data_ptr() for l in range(L)]           # noqa: E731
    with K.KVPool(regions, weights, spec, 0) as pool:
        m = pool.place(1, n)
        ora = oracle.Pool(weights, caps, bb)
        om = ora.place(1, n)
        assert np.array_equal(m, om)
        s = torch.cuda.current_stream().cuda_stream
        pool.store(m, src_slots, S, kp(src), vp(src), s)
        rm = m.copy()
        absent = rng.random(n) < 0.2
        rm["region"][absent] = K.ABSENT
        pool.retrieve(rm, dst_slots, S, kp(dst), vp(dst), s)
        torch.cuda.synchronize()
        shape = (L, H, bs, D, elem_bytes)
        oregions = [np.zeros(c, np.uint8) for c in caps]
        oracle.store(om, src_slots, oregions, [src_h[l, 0] for l in range(L)], [src_h[l, 1] for l in range(L)],
                     shape, layout)
        for r in range(len(regions)):
            offs = om["offset"][om["region"] == r]
            if len(offs):
                lo, hi = int(offs.min()), int(offs.max()) + bb
                assert np.array_equal(pool.region_read(r, lo, hi - lo), oregions[r][lo:hi]), "region %d" % r
        expect = np.zeros_like(src_h)
        orm = om.copy()
        orm["region"][absent] = oracle.ABSENT
        oracle.gather(orm, dst_slots, oregions, [expect[l, 0] for l in range(L)], [expect[l, 1] for l in range(L)],
                      shape, layout)
        assert np.array_equal(dst.cpu().numpy(), expect)


def test_two_pools_at_once():
    """Two pools on one GPU, their calls interleaved on two streams (each pool stores on one and
    retrieves on the other): the pools share nothing, and both results equal the oracle's."""
    wls = [workloads.make(2, max_blocks=70, seed=11), workloads.make(4, max_blocks=90, seed=12)]
    say("case two pools")
    runs = [make_run(w) for w in wls]
    try:
        hosts = []
        for r in runs:
            hosts.append(r.fill_source(keep_host=True))
            r.fill_dst()
            r.place_all()
        streams = [torch.cuda.Stream(), torch.cuda.Stream()]
        for s_ in streams:
            s_.wait_stream(torch.cuda.current_stream())
        for i, r in enumerate(runs):                          # pool i stores on stream i ...
            r.store_all(streams[i])
        streams[0].wait_stream(streams[1])
        streams[1].wait_stream(streams[0])
        for i, r in enumerate(runs):                          # ... and retrieves on the other one
            for q in r.wl.requests:
                r.retrieve(q, streams[1 - i])
        for s_ in streams:
            torch.cuda.current_stream().wait_stream(s_)
        torch.cuda.synchronize()
        for w, r, h in zip(wls, runs, hosts):
            check_full(w, r, h)
    finally:
        for r in runs:
            r.close()


@pytest.mark.parametrize("sdma", [False, True])
def test_hundreds_of_requests_in_one_call(sdma):
    """300 requests of 1-6 blocks each, placed separately on a mixed pool, then stored in one call and
    retrieved in one call (maps and tables concatenated, a permuted destination), through the kernel
    and through the copy engines: every request is listed once for its ordering events, and every
    destination vector carries its own tags.  Releasing each request then waits on those events."""
    L, H, bs, D = 4, 2, 16, 64
    spec = K.KVSpec(L, H, D, bs)
    rng = np.random.default_rng(300)
    sizes = rng.integers(1, 7, size=300)
    n = int(sizes.sum())
    S = n + 40
    weights = [2, 1, 1]                      # a 3-block set already reaches the staging region
    caps = [((w * n // sum(weights) + 320) * spec.block_bytes + 4095) // 4096 * 4096 for w in weights]
    regions = [K.Region("host", caps[0], 0), K.Region("staging", caps[1]), K.Region("host", caps[2], 0)]
    say("case many requests", n, "sdma", sdma)
    dev = torch.device("cuda", 0)
    tags = tag_cache(L, S, H, bs, D)
    src = torch.from_numpy(tags).to(dev)
    sentinel = np.int16(np.uint16(SENTINEL).view(np.int16))
    dst = torch.full(tuple(tags.shape), int(sentinel), dtype=torch.int16, device=dev)
    kp = lambda t: [t[l, 0].data_ptr() for l in range(L)]           # noqa: E731
    vp = lambda t: [t[l, 1].data_ptr() for l in range(L)]           # noqa: E731
    src_slots = rng.permutation(S)[:n].astype(np.int32)
    dst_slots = rng.permutation(S)[:n].astype(np.int32)
    with K.KVPool(regions, weights, spec, 0) as pool:
        if sdma:
            pool.set_launch(K.CLASS_HOST, K.OP_RETRIEVE, 0, K.LAUNCH_SDMA)
            pool.set_launch(K.CLASS_HOST, K.OP_STORE, 0, K.LAUNCH_SDMA)
        m = np.concatenate([pool.place(1000 + i, int(c)) for i, c in enumerate(sizes)])
        s = torch.cuda.current_stream().cuda_stream
        pool.store(m, src_slots, S, kp(src), vp(src), s)
        pool.retrieve(m, dst_slots, S, kp(dst), vp(dst), s)
        torch.cuda.synchronize()
        check_tags(tags, dst.cpu().numpy(), src_slots, dst_slots, sentinel)
        for i in range(len(sizes)):
            pool.release(1000 + i)


def test_request_size_limit():
    """n_blocks * 4 * L may reach 2^31 and no more: a kernel's units and its workgroup stride are summed
    in 32 bits.  At the limit, a map of absent entries is accepted (and moves nothing); one block more
    is refused with INVALID before anything is read or launched."""
    L = 32
    spec = K.KVSpec(L, 1, 8)                                   # 256-byte chunks
    cache = torch.zeros(L, 2, 4, 16, 8, dtype=torch.int16, device="cuda")
    ks = [cache[l, 0].data_ptr() for l in range(L)]
    vs = [cache[l, 1].data_ptr() for l in range(L)]
    s = torch.cuda.current_stream().cuda_stream
    limit = (1 << 31) // (4 * L)
    with K.KVPool([K.Region("staging", 1 << 20)], [1], spec, 0) as p:
        for n, ok in ((limit, True), (limit + 1, False)):
            m = np.zeros(n, dtype=K.LOC_DTYPE)
            m["region"] = K.ABSENT
            table = np.full(n, -1, np.int32)
            if ok:
                p.retrieve(m, table, 4, ks, vs, s)
            else:
                with pytest.raises(K.KVPoolError) as ei:
                    p.retrieve(m, table, 4, ks, vs, s)
                assert ei.value.name == "INVALID" and "too large" in str(ei.value)
            del m, table
    torch.cuda.synchronize()
    assert int(cache.abs().sum()) == 0
