"""Small calls: a store or retrieve whose work list fits in the kernel
arguments (384 words: one engine pointer per moved chunk, two words per
present block) runs both region classes in one launch, with no upload.

Every case runs the same seeded inputs through that launch and through the
upload path (KVP_LAUNCH_UPLOAD: work list uploaded, one launch per class),
and checks each against the oracle bit for bit.  Sizes sit on both sides of
the inline capacity: 160 blocks for the 32-layer LLaMA shape, 168 for the
24-layer GPT-OSS shape, 191 when one layer of a 32-layer cache moves.
"""
import numpy as np
import pytest

from kvgen import workloads
from paper_2606_14779_amd import kvpool as K
from paper_2606_14779_amd.runner import SENTINEL

from gpu_util import check_full, make_run, oracle_expectation, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

INLINE_WORDS = 384


def _capacity(layers_moved):
    return (INLINE_WORDS - 2 * layers_moved) // 2


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def _upload(run, layout):
    """KVP_LAUNCH_UPLOAD on the host class of both ops, the defaults otherwise."""
    run.pool.set_launch(K.CLASS_HOST, K.OP_RETRIEVE, 0, (K.LAUNCH_LDS if layout == 1 else 0) | K.LAUNCH_UPLOAD)
    run.pool.set_launch(K.CLASS_HOST, K.OP_STORE, 0, K.LAUNCH_NT_STORE | K.LAUNCH_UPLOAD)


def test_capacity_figures():
    assert _capacity(32) == 160 and _capacity(24) == 168 and _capacity(1) == 191


@pytest.mark.parametrize("upload", [False, True])
@pytest.mark.parametrize("layout", [0, 1])
@pytest.mark.parametrize("cfg,n", [(1, 1), (1, 160), (1, 161), (2, 5), (2, 47), (4, 168), (4, 169), (5, 61)])
def test_both_paths_match_oracle(cfg, n, layout, upload):
    wl = workloads.make(cfg, max_blocks=n, layout=layout)
    say("case small-call", wl.name, "n", n, "layout", layout, "upload", upload,
        "blocks", [q.n_present for q in wl.requests])
    run = make_run(wl)
    try:
        if upload:
            _upload(run, layout)
        host = run.setup(keep_host=True)      # the store goes through the same path
        run.retrieve_all()
        torch.cuda.synchronize()
        check_full(wl, run, host)
    finally:
        run.close()


@pytest.mark.parametrize("layout", [0, 1])
@pytest.mark.parametrize("upload", [False, True])
@pytest.mark.parametrize("n,lo,hi", [(191, 7, 8), (192, 7, 8), (23, 0, 1), (23, 30, 32), (23, 29, 32)])
def test_layer_range(n, lo, hi, upload, layout):
    """A layer range shortens the pointer table: the capacity grows to 191 blocks for one layer, and
    the table starts at the range's first layer (first and last layers covered)."""
    wl = workloads.make(2, max_blocks=n, layout=layout)
    say("case small-call layers", n, lo, hi, "upload", upload, "layout", layout)
    run = make_run(wl)
    try:
        if upload:
            _upload(run, layout)
        host = run.setup(keep_host=True)
        q = wl.requests[0]
        kp, vp = run.layer_ptrs(run.dst)
        kp = [p if lo <= l < hi else 0 for l, p in enumerate(kp)]    # pointers outside the range unused
        vp = [p if lo <= l < hi else 0 for l, p in enumerate(vp)]
        run.pool.retrieve_layers(run.retrieve_maps[q.request_id], q.dst_slots, wl.dst_num_slots, lo, hi, kp, vp,
                                 torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        _, _, expect = oracle_expectation(wl, run, host)
        got = run.dst.cpu().numpy().view(np.uint16)
        assert np.array_equal(got[lo:hi], expect[lo:hi])
        assert np.all(got[:lo] == SENTINEL) and np.all(got[hi:] == SENTINEL)
    finally:
        run.close()


@pytest.mark.parametrize("layout", [0, 1])
@pytest.mark.parametrize("grid_host,grid_staging,flags", [
    (1, 1, 0), (1, 65536, K.LAUNCH_SPLIT2), (12, 3, K.LAUNCH_NT_LOAD | K.LAUNCH_NT_STORE),
    (7, 7, K.LAUNCH_XCD | K.LAUNCH_CHUNK_MAJOR), (4096, 1, K.LAUNCH_LDS)])
def test_launch_shapes(grid_host, grid_staging, flags, layout):
    """Per-class grids from one to more workgroups than units, and flags the small-call launch
    takes (copy form) or drops (XCD renumbering, chunk-major order)."""
    wl = workloads.make(2, max_blocks=37, layout=layout)
    say("case small-call launch", grid_host, grid_staging, flags, layout)
    run = make_run(wl)
    try:
        for op in (K.OP_RETRIEVE, K.OP_STORE):
            run.pool.set_launch(K.CLASS_HOST, op, grid_host, flags)
            run.pool.set_launch(K.CLASS_STAGING, op, grid_staging, flags)
        host = run.setup(keep_host=True)
        run.retrieve_all()
        torch.cuda.synchronize()
        check_full(wl, run, host)
    finally:
        run.close()


def test_back_to_back_small_calls_on_two_streams():
    """Many small retrieves of disjoint slices, alternating between two streams with no host
    synchronisation: each launch carries its own work list, so nothing is shared between calls."""
    wl = workloads.make(2, max_blocks=120)
    say("case small-call streams")
    run = make_run(wl)
    try:
        host = run.setup(keep_host=True)
        q = wl.requests[0]
        kp, vp = run.layer_ptrs(run.dst)
        m = run.retrieve_maps[q.request_id]
        streams = [torch.cuda.Stream(), torch.cuda.Stream()]
        for s in streams:
            s.wait_stream(torch.cuda.current_stream())
        for i, b in enumerate(range(0, q.n_present, 3)):
            e = min(b + 3, q.n_present)
            run.pool.retrieve(m[b:e].copy(), q.dst_slots[b:e].copy(), wl.dst_num_slots, kp, vp,
                              streams[i % 2].cuda_stream)
        for s in streams:
            torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        check_full(wl, run, host)
    finally:
        run.close()


def test_thousands_of_queued_small_calls():
    """2000 one-block retrieves enqueued on one stream with no synchronisation: each launch holds
    its own 3 KiB argument block until it runs; the result is the same as one call."""
    wl = workloads.make(2, max_blocks=37)
    say("case small-call queue")
    run = make_run(wl)
    try:
        host = run.setup(keep_host=True)
        q = wl.requests[0]
        kp, vp = run.layer_ptrs(run.dst)
        m = run.retrieve_maps[q.request_id]
        s = torch.cuda.current_stream().cuda_stream
        one = [(m[b:b + 1].copy(), q.dst_slots[b:b + 1].copy()) for b in range(q.n_present)]
        for i in range(2000):
            mb, tb = one[i % q.n_present]
            run.pool.retrieve(mb, tb, wl.dst_num_slots, kp, vp, s)
        torch.cuda.synchronize()
        check_full(wl, run, host)
    finally:
        run.close()
