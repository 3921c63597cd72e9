"""Seeded random GPU parity cases: shapes, region mixes and weights, tables,
absent entries, layouts, launch shapes and flags; every case is compared with
the oracle element by element (pool bytes and destination cache)."""
import os

import numpy as np
import pytest

import kvgen
import oracle
from paper_2606_14779_amd import kvpool as K

from gpu_util import say

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

SENT = 0x7FA5


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def _case(seed):
    rng = np.random.default_rng(seed)
    layout = int(rng.integers(0, 2))
    while True:
        L = int(rng.choice([1, 2, 3, 5]))
        H = int(rng.choice([1, 2, 3, 4, 8]))
        bs = int(rng.choice([1, 2, 4, 16]))
        D = int(rng.choice([8, 16, 24, 40, 64, 128]))
        C = H * bs * D * 2
        if C % 16 == 0 and (layout == 0 or (D * 2) % 16 == 0):
            break
    N = int(rng.integers(1, 7))
    kinds = ["host" if rng.random() < 0.5 else "staging" for _ in range(N)]
    weights = [int(w) for w in rng.integers(1, 6, size=N)]
    n = int(rng.integers(1, 150))
    grid = [int(rng.choice([1, 3, 12, 64, 8192])) for _ in range(4)]
    flags = [int(rng.choice([0, K.LAUNCH_NT_LOAD, K.LAUNCH_NT_STORE, K.LAUNCH_NT_LOAD | K.LAUNCH_NT_STORE]))
             | (K.LAUNCH_LDS if layout == 1 and rng.random() < 0.5 else 0) for _ in range(4)]
    # unit order drawn from a generator of its own, so the draws above stay as they were
    order = np.random.default_rng(seed + 7919)
    flags = [f | (K.LAUNCH_CHUNK_MAJOR if order.random() < 0.4 else 0) for f in flags]
    # every case here fits the small-call launch; about half are sent through the upload path
    # instead (the flag on the host class of both ops), again from a generator of its own
    if np.random.default_rng(seed + 104729).random() < 0.5:
        flags[0] |= K.LAUNCH_UPLOAD
        flags[1] |= K.LAUNCH_UPLOAD
    return rng, layout, (L, H, bs, D), kinds, weights, n, grid, flags


# KVP_FUZZ_SEEDS widens the run (e.g. 540 for a longer soak); 40 by default
@pytest.mark.parametrize("seed", list(range(int(os.environ.get("KVP_FUZZ_SEEDS", "40")))))
def test_random_case(seed):
    rng, layout, (L, H, bs, D), kinds, weights, n, grid, flags = _case(seed)
    say("fuzz", seed, dict(layout=layout, L=L, H=H, bs=bs, D=D, kinds=kinds, w=weights, n=n, grid=grid, flags=flags))
    spec = K.KVSpec(L, H, D, bs, 2, layout)
    bb = spec.block_bytes
    W = sum(weights)
    caps = [((w * n // W + 1) * bb + 4095) // 4096 * 4096 + int(rng.integers(0, 3)) * 4096 for w in weights]
    regions = [K.Region(k, c, 0 if k == "host" else -1) for k, c in zip(kinds, caps)]
    src_slots_n, dst_slots_n = n + int(rng.integers(0, 5)), n + int(rng.integers(0, 9))
    src_slots = rng.permutation(src_slots_n)[:n].astype(np.int32)
    dst_slots = rng.permutation(dst_slots_n)[:n].astype(np.int32)
    host_src = np.zeros((L, 2, src_slots_n, H, bs, D), np.uint16)
    kvgen.fill_cache(seed, 1, np.arange(n, dtype=np.uint64), src_slots, L, H, bs, D,
                     [host_src[l, 0].ctypes.data for l in range(L)], [host_src[l, 1].ctypes.data for l in range(L)])
    src = torch.from_numpy(host_src.view(np.int16)).cuda()
    dst = torch.full((L, 2, dst_slots_n, H, bs, D), int(np.uint16(SENT).view(np.int16)), dtype=torch.int16,
                     device="cuda")
    kp = lambda t: [t[l, 0].data_ptr() for l in range(L)]           # noqa: E731
    vp = lambda t: [t[l, 1].data_ptr() for l in range(L)]           # noqa: E731
    with K.KVPool(regions, weights, spec, 0) as pool:
        for i, (cls, op) in enumerate([(0, 0), (0, 1), (1, 0), (1, 1)]):
            pool.set_launch(cls, op, grid[i], flags[i])
        m = pool.place(1, n)
        ora = oracle.Pool(weights, caps, bb)
        om = ora.place(1, n)
        assert np.array_equal(m, om)
        s = torch.cuda.current_stream().cuda_stream
        pool.store(m, src_slots, src_slots_n, kp(src), vp(src), s)
        rm = m.copy()
        absent = rng.random(n) < 0.2
        rm["region"][absent] = K.ABSENT
        table = dst_slots.copy()
        table[absent] = -1
        pool.retrieve(rm, table, dst_slots_n, kp(dst), vp(dst), s)
        torch.cuda.synchronize()
        shape = (L, H, bs, D, 2)
        oregions = [np.zeros(c, np.uint8) for c in caps]
        oracle.store(om, src_slots, oregions, [host_src[l, 0] for l in range(L)],
                     [host_src[l, 1] for l in range(L)], shape, layout)
        for r in range(len(regions)):
            offs = om["offset"][om["region"] == r]
            if len(offs):
                lo, hi = int(offs.min()), int(offs.max()) + bb
                assert np.array_equal(pool.region_read(r, lo, hi - lo), oregions[r][lo:hi]), "region %d" % r
        expect = np.full((L, 2, dst_slots_n, H, bs, D), SENT, np.uint16)
        orm = om.copy()
        orm["region"][absent] = oracle.ABSENT
        oracle.gather(orm, table, oregions, [expect[l, 0] for l in range(L)], [expect[l, 1] for l in range(L)],
                      shape, layout)
        got = dst.cpu().numpy().view(np.uint16)
        assert np.array_equal(got, expect)


# shapes whose chunks pair up into 4096-byte sectors (file regions need 2 x chunk to be a multiple)
_FILE_SHAPES = [(1, 1, 16, 64), (2, 2, 16, 64), (3, 4, 16, 64), (2, 1, 16, 128), (5, 2, 16, 128),
                (1, 8, 16, 128), (4, 4, 4, 128), (2, 8, 8, 64)]


@pytest.mark.parametrize("seed", list(range(int(os.environ.get("KVP_FUZZ_FILE_SEEDS", "16")))))
def test_random_case_with_file_regions(seed, tmp_path):
    """Random cases with some regions as file regions (the storage tier): shapes, region mixes and
    weights, ring sizes from one block up, launch flags, absent entries; map, pool bytes (read back
    through the library, i.e. from the files) and destination against the oracle."""
    rng = np.random.default_rng(50000 + seed)
    layout = int(rng.integers(0, 2))
    L, H, bs, D = _FILE_SHAPES[int(rng.integers(0, len(_FILE_SHAPES)))]
    spec = K.KVSpec(L, H, D, bs, 2, layout)
    bb = spec.block_bytes
    N = int(rng.integers(1, 6))
    kinds = [str(rng.choice(["host", "staging", "file"])) for _ in range(N)]
    kinds[int(rng.integers(0, N))] = "file"                                  # at least one file region
    weights = [int(w) for w in rng.integers(1, 6, size=N)]
    n = int(rng.integers(1, 120))
    W = sum(weights)
    caps = [((w * n // W + 1) * bb + 4095) // 4096 * 4096 + int(rng.integers(0, 3)) * 4096 for w in weights]
    ring_blocks = int(rng.choice([1, 2, 3, 7, 64]))
    flags = [int(rng.choice([0, K.LAUNCH_NT_LOAD | K.LAUNCH_NT_STORE, K.LAUNCH_UPLOAD])) for _ in range(2)]
    say("fuzz file", seed, dict(layout=layout, shape=(L, H, bs, D), kinds=kinds, w=weights, n=n,
                                ring_blocks=ring_blocks, flags=flags))
    regions = [K.Region(k, c, path=str(tmp_path / ("r%d.bin" % i)) if k == "file" else None)
               for i, (k, c) in enumerate(zip(kinds, caps))]
    src_slots_n, dst_slots_n = n + int(rng.integers(0, 5)), n + int(rng.integers(0, 9))
    src_slots = rng.permutation(src_slots_n)[:n].astype(np.int32)
    dst_slots = rng.permutation(dst_slots_n)[:n].astype(np.int32)
    host_src = np.zeros((L, 2, src_slots_n, H, bs, D), np.uint16)
    kvgen.fill_cache(50000 + seed, 1, np.arange(n, dtype=np.uint64), src_slots, L, H, bs, D,
                     [host_src[l, 0].ctypes.data for l in range(L)], [host_src[l, 1].ctypes.data for l in range(L)])
    src = torch.from_numpy(host_src.view(np.int16)).cuda()
    dst = torch.full((L, 2, dst_slots_n, H, bs, D), int(np.uint16(SENT).view(np.int16)), dtype=torch.int16,
                     device="cuda")
    kp = lambda t: [t[l, 0].data_ptr() for l in range(L)]           # noqa: E731
    vp = lambda t: [t[l, 1].data_ptr() for l in range(L)]           # noqa: E731
    with K.KVPool(regions, weights, spec, 0) as pool:
        pool.set_file_ring(max(64 << 10, (ring_blocks * bb + 4095) // 4096 * 4096))
        for op in (K.OP_RETRIEVE, K.OP_STORE):
            pool.set_launch(K.CLASS_HOST, op, 0, flags[op] | (K.LAUNCH_NT_STORE if op == K.OP_STORE else 0))
        m = pool.place(1, n)
        ora = oracle.Pool(weights, caps, bb)
        om = ora.place(1, n)
        assert np.array_equal(m, om)
        s = torch.cuda.current_stream().cuda_stream
        pool.store(m, src_slots, src_slots_n, kp(src), vp(src), s)
        rm = m.copy()
        absent = rng.random(n) < 0.2
        rm["region"][absent] = K.ABSENT
        table = dst_slots.copy()
        table[absent] = -1
        pool.retrieve(rm, table, dst_slots_n, kp(dst), vp(dst), s)
        torch.cuda.synchronize()
        shape = (L, H, bs, D, 2)
        oregions = [np.zeros(c, np.uint8) for c in caps]
        oracle.store(om, src_slots, oregions, [host_src[l, 0] for l in range(L)],
                     [host_src[l, 1] for l in range(L)], shape, layout)
        for r in range(len(regions)):
            offs = om["offset"][om["region"] == r]
            if len(offs):
                lo, hi = int(offs.min()), int(offs.max()) + bb
                assert np.array_equal(pool.region_read(r, lo, hi - lo), oregions[r][lo:hi]), "region %d" % r
        expect = np.full((L, 2, dst_slots_n, H, bs, D), SENT, np.uint16)
        orm = om.copy()
        orm["region"][absent] = oracle.ABSENT
        oracle.gather(orm, table, oregions, [expect[l, 0] for l in range(L)], [expect[l, 1] for l in range(L)],
                      shape, layout)
        got = dst.cpu().numpy().view(np.uint16)
        assert np.array_equal(got, expect)
        # a random layer range into a fresh destination: file spans narrower than a block
        lo = int(rng.integers(0, L))
        hi = int(rng.integers(lo + 1, L + 1))
        dst.fill_(int(np.uint16(SENT).view(np.int16)))
        pool.retrieve_layers(rm, table, dst_slots_n, lo, hi, kp(dst), vp(dst), s)
        torch.cuda.synchronize()
        got = dst.cpu().numpy().view(np.uint16)
        assert np.array_equal(got[lo:hi], expect[lo:hi]), "layers [%d, %d)" % (lo, hi)
        assert np.all(got[:lo] == SENT) and np.all(got[hi:] == SENT)
