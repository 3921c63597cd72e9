"""The allocation-free retrieve (kv_pool_retrieve_noalloc) against kv_pool_retrieve.

Both run through the C ABI on the same pool and the same seeded inputs; the
bar is bit-exact (the path copies bf16 words).  The work list of the
allocation-free call lives in a static device array shared by every call on
the GPU, so the checks run calls back to back, the second one smaller, and
on two streams at once.
"""
import numpy as np
import pytest

from kvgen import workloads
from paper_2606_14779_amd import kvpool as K
from paper_2606_14779_amd.runner import SENTINEL

from gpu_util import check_full, make_run, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SCRATCH = 1 << 20


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def _subset(full_map, table, n):
    """The first n present entries of a map, the rest marked absent."""
    m = full_map.copy()
    m["region"][n:] = K.ABSENT
    return m, table


@pytest.mark.parametrize("layout", [0, 1])
def test_noalloc_equals_retrieve_on_two_calls(layout):
    """Call 1: a 300-block LLaMA-shaped request over 2 host + 4 staging regions (both kernels, the
    staging one forked).  Call 2, right after on the same stream: only its first 37 blocks.  Each
    allocation-free result equals kv_pool_retrieve's, and call 1 also equals the oracle's."""
    wl = workloads.make(3, max_blocks=300, layout=layout)
    say("case noalloc two calls, layout", layout)
    run = make_run(wl)
    try:
        host = run.setup(keep_host=True)
        q = wl.requests[0]
        m = run.retrieve_maps[q.request_id]
        kp, vp = run.layer_ptrs(run.dst)
        s = torch.cuda.current_stream().cuda_stream
        for n in (q.n_present, 37):
            sub, table = _subset(m, q.dst_slots, n)
            run.fill_dst()
            run.pool.retrieve(sub, table, wl.dst_num_slots, kp, vp, s)
            torch.cuda.synchronize()
            ref = run.dst.clone()
            run.fill_dst()
            run.pool.retrieve_noalloc(sub, table, wl.dst_num_slots, kp, vp, s)
            torch.cuda.synchronize()
            assert torch.equal(run.dst, ref), "allocation-free retrieve of %d blocks differs" % n
            if n == q.n_present:
                check_full(wl, run, host)
    finally:
        run.close()


def test_noalloc_back_to_back_on_two_streams():
    """Two allocation-free calls enqueued back to back on two streams with no host synchronisation,
    the second smaller, then a third on the first stream: the library orders the users of the shared
    array, so every destination equals kv_pool_retrieve's result for the same call."""
    wl = workloads.make(2, max_blocks=200)
    say("case noalloc two streams")
    run = make_run(wl)
    try:
        run.setup()
        q = wl.requests[0]
        m = run.retrieve_maps[q.request_id]
        kp, vp = run.layer_ptrs(run.dst)
        cur = torch.cuda.current_stream()
        # reference results, one destination cache per call
        cuts = (q.n_present, 50, 9)
        refs = []
        for n in cuts:
            sub, table = _subset(m, q.dst_slots, n)
            run.fill_dst()
            run.pool.retrieve(sub, table, wl.dst_num_slots, kp, vp, cur.cuda_stream)
            torch.cuda.synchronize()
            refs.append(run.dst.clone())
        dsts = [torch.full_like(run.dst, int(np.uint16(SENTINEL).view(np.int16))) for _ in cuts]
        a, b = torch.cuda.Stream(), torch.cuda.Stream()
        a.wait_stream(cur)
        b.wait_stream(cur)
        for n, d, st in zip(cuts, dsts, (a, b, a)):
            sub, table = _subset(m, q.dst_slots, n)
            dk, dv = run.layer_ptrs(d)
            run.pool.retrieve_noalloc(sub, table, wl.dst_num_slots, dk, dv, st.cuda_stream)
        torch.cuda.synchronize()
        for n, d, r in zip(cuts, dsts, refs):
            assert torch.equal(d, r), "allocation-free retrieve of %d blocks differs" % n
    finally:
        run.close()


def test_noalloc_ignores_copy_engine_setting():
    """With the copy-engine transport set for the host class, the allocation-free call still runs
    the zero-copy kernel and returns the same bytes as kv_pool_retrieve."""
    wl = workloads.make(2, max_blocks=64)
    say("case noalloc with sdma set")
    run = make_run(wl)
    try:
        run.setup()
        q = wl.requests[0]
        m = run.retrieve_maps[q.request_id]
        kp, vp = run.layer_ptrs(run.dst)
        s = torch.cuda.current_stream().cuda_stream
        run.pool.set_launch(K.CLASS_HOST, K.OP_RETRIEVE, 0, K.LAUNCH_SDMA)
        run.fill_dst()
        run.pool.retrieve(m, q.dst_slots, wl.dst_num_slots, kp, vp, s)
        torch.cuda.synchronize()
        ref = run.dst.clone()
        run.fill_dst()
        run.pool.retrieve_noalloc(m, q.dst_slots, wl.dst_num_slots, kp, vp, s)
        torch.cuda.synchronize()
        assert torch.equal(run.dst, ref)
    finally:
        run.close()


def test_noalloc_size_limit():
    """One-layer blocks of 32 bytes: a work list of one 16-byte pointer row plus 65,535 items fills
    the 1 MiB array exactly and runs (equal to kv_pool_retrieve); one block more is refused with
    INVALID before any work, leaving the destination untouched."""
    n_max = (SCRATCH - 16) // 16
    spec = K.KVSpec(1, 1, 8, 1, 2, 0)                       # C = 16 B, block = 32 B
    bb = 32
    regions = [K.Region("staging", (n_max + 1) * bb + 4096), K.Region("host", 64 * 4096, -1)]
    say("case noalloc size limit", n_max)
    with K.KVPool(regions, [1000000, 1], spec, 0) as p:
        m = p.place(1, n_max + 1)
        assert int(np.sum(m["region"] == 1)) == 0          # every block on the staging region
        slots = n_max + 1
        src = torch.randint(-32768, 32767, (1, 2, slots, 1, 1, 8), dtype=torch.int16, device="cuda")
        ks, vs = [src[0, 0].data_ptr()], [src[0, 1].data_ptr()]
        s = torch.cuda.current_stream().cuda_stream
        table = np.arange(n_max + 1, dtype=np.int32)
        p.store(m, table, slots, ks, vs, s)
        dst = torch.zeros_like(src)
        ref = torch.zeros_like(src)
        dk, dv = [dst[0, 0].data_ptr()], [dst[0, 1].data_ptr()]
        with pytest.raises(K.KVPoolError) as ei:
            p.retrieve_noalloc(m, table, slots, dk, dv, s)
        assert ei.value.name == "INVALID" and "static scratch" in str(ei.value)
        torch.cuda.synchronize()
        assert bool((dst == 0).all())
        fit = m.copy()
        fit["region"][n_max:] = K.ABSENT                     # exactly n_max present blocks
        p.retrieve_noalloc(fit, table, slots, dk, dv, s)
        p.retrieve(fit, table, slots, [ref[0, 0].data_ptr()], [ref[0, 1].data_ptr()], s)
        torch.cuda.synchronize()
        assert torch.equal(dst, ref)
        assert torch.equal(dst[:, :, :n_max], src[:, :, :n_max]) and bool((dst[:, :, n_max:] == 0).all())
