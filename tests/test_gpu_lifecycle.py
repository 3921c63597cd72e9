"""One long-lived pool under a seeded random sequence of operations.

Requests are placed, stored, retrieved and released in random order, on
three streams with no host synchronisation between the operations of a
round; released ranges are placed again; placed requests grow by further
offload sets (kv_pool_extend); the host-class transport is switched between
the zero-copy kernel and the copy engines along the way, and small calls
between their one-launch form and the upload path.
Checked against what placement and the round trip fix:

- every map equals the oracle's, the oracle pool carrying the same place /
  release history;
- after each round, every destination slot holds exactly what the last
  retrieve into it wrote -- the source values of that block, for the layers
  the call covered -- and every other slot still holds the sentinel.

A retrieve writes only slots no other call of the same round writes, so the
expected contents do not depend on how the streams interleave; ordering
between the store and the retrieves of one request, and between a release
and the next placement in the same range, is the library's to enforce.
"""
import os

import numpy as np
import pytest

import kvgen
import oracle
from kvgen import workloads
from paper_2606_14779_amd import kvpool as K
from paper_2606_14779_amd.runner import SENTINEL

from gpu_util import say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

L, H, BS, D = 4, 2, 16, 64            # chunk 4 KiB, block 32 KiB
SEED = 4242
# KVP_LIFECYCLE_SEEDS / KVP_LIFECYCLE_ROUNDS widen the run for a longer soak (1 seed, 12 rounds by default)
SEEDS = [SEED] + [5000 + 7 * k for k in range(int(os.environ.get("KVP_LIFECYCLE_SEEDS", "1")) - 1)]
ROUNDS = int(os.environ.get("KVP_LIFECYCLE_ROUNDS", "12"))
SRC_SLOTS, DST_SLOTS = 4096, 2048


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("tier", ["memory", "file"])
@pytest.mark.parametrize("seed", SEEDS)
@pytest.mark.parametrize("layout", [0, 1])
def test_random_lifecycle(layout, seed, tier, tmp_path):
    """tier "file": the last region is a file region (the storage tier) instead of HBM staging."""
    rng = np.random.default_rng(seed + layout)
    path_rng = np.random.default_rng(seed + 17 + layout)   # upload bit: apart, so rng's sequence is unchanged
    ext_rng = np.random.default_rng(seed + 29 + layout)    # extensions: apart as well
    shape = workloads.KVShape("lifecycle", L, H, D)
    bb = shape.block_bytes
    weights = [3, 1, 2, 2]
    kinds = ["host", "staging", "host", "staging" if tier == "memory" else "file"]
    caps = [150 * bb, 60 * bb, 110 * bb, 110 * bb]   # small enough to fill: NOSPACE and fragmentation
    path = str(tmp_path / "region3.bin")
    pool = K.KVPool([K.Region(k, c, path=path if k == "file" else None) for k, c in zip(kinds, caps)], weights,
                    K.KVSpec(L, H, D, BS, 2, layout), 0)
    if tier == "file":
        pool.set_file_ring(16 * bb)     # several batches per call, the ring wrapping
    ora = oracle.Pool(weights, caps, bb)
    dev = torch.device("cuda", 0)
    src = torch.empty((L, 2, SRC_SLOTS, H, BS, D), dtype=torch.int16, device=dev)
    dst = torch.empty((L, 2, DST_SLOTS, H, BS, D), dtype=torch.int16, device=dev)
    sent = int(np.uint16(SENTINEL).view(np.int16))
    dst.fill_(sent)
    expect = np.full(tuple(dst.shape), SENTINEL, np.uint16)
    kp_src = [src[l, 0].data_ptr() for l in range(L)]
    vp_src = [src[l, 1].data_ptr() for l in range(L)]
    kp_dst = [dst[l, 0].data_ptr() for l in range(L)]
    vp_dst = [dst[l, 1].data_ptr() for l in range(L)]
    streams = [torch.cuda.Stream(device=dev) for _ in range(3)]
    free_src = list(rng.permutation(SRC_SLOTS))
    live = {}                              # request -> dict(n, map, src, vals, stored)
    next_req = 1
    sdma = {K.OP_RETRIEVE: False, K.OP_STORE: False}
    counts = dict(place=0, nospace=0, store=0, retrieve=0, release=0, toggle=0, extend=0)
    try:
        for rnd in range(ROUNDS):
            for s in streams:
                s.wait_stream(torch.cuda.current_stream())
            used_dst = set()
            for _ in range(14):
                op = rng.choice(["place", "store", "retrieve", "retrieve", "release", "toggle"],
                                p=[0.25, 0.2, 0.15, 0.15, 0.15, 0.1])
                st = streams[int(rng.integers(3))]
                if op == "place" or not live:
                    n = int(rng.integers(1, 61))
                    if len(free_src) < n:
                        continue
                    rc, om = ora.try_place(next_req, n)
                    if rc != 0:
                        with pytest.raises(K.KVPoolError):
                            pool.place(next_req, n)
                        counts["nospace"] += 1
                        next_req += 1
                        continue
                    m = pool.place(next_req, n)
                    assert np.array_equal(m.view(np.uint8), om.view(np.uint8)), "placement differs"
                    slots = np.array([free_src.pop() for _ in range(n)], np.int64)
                    vals = np.stack([kvgen.block_values(seed, next_req, b, L, H, BS, D) for b in range(n)], 2)
                    # [L][2][n][H][bs][D] into the source slots, stream-ordered before any store
                    src[:, :, torch.from_numpy(slots).to(dev)] = torch.from_numpy(vals.view(np.int16)).to(dev)
                    for s in streams:
                        s.wait_stream(torch.cuda.current_stream())
                    live[next_req] = dict(n=n, map=m, src=slots.astype(np.int32), vals=vals, stored=False)
                    next_req += 1
                    counts["place"] += 1
                elif op == "store":
                    r = int(rng.choice(list(live)))
                    q = live[r]
                    if rng.random() < 0.3:       # in two layer groups
                        cut = int(rng.integers(1, L))
                        pool.store_layers(q["map"], q["src"], SRC_SLOTS, 0, cut, kp_src, vp_src, st.cuda_stream)
                        pool.store_layers(q["map"], q["src"], SRC_SLOTS, cut, L, kp_src, vp_src, st.cuda_stream)
                    else:
                        pool.store(q["map"], q["src"], SRC_SLOTS, kp_src, vp_src, st.cuda_stream)
                    q["stored"] = True
                    counts["store"] += 1
                elif op == "retrieve":
                    stored = [r for r, q in live.items() if q["stored"]]
                    if not stored:
                        continue
                    r = int(rng.choice(stored))
                    q = live[r]
                    avail = np.setdiff1d(np.arange(DST_SLOTS), np.fromiter(used_dst, np.int64, len(used_dst)))
                    if len(avail) < q["n"]:
                        continue
                    slots = rng.choice(avail, size=q["n"], replace=False).astype(np.int32)
                    m = q["map"].copy()
                    absent = rng.random(q["n"]) < 0.2
                    m["region"][absent] = K.ABSENT
                    order = rng.permutation(q["n"])
                    lo, hi = (0, L) if rng.random() < 0.6 else sorted(rng.choice(L + 1, 2, replace=False))
                    if rng.random() < 0.3 and lo == 0 and hi == L and not absent.any():
                        pool.retrieve_request(r, slots, DST_SLOTS, kp_dst, vp_dst, st.cuda_stream)
                    else:
                        pool.retrieve_layers(m[order], slots[order], DST_SLOTS, int(lo), int(hi),
                                             kp_dst, vp_dst, st.cuda_stream)
                    for b in range(q["n"]):
                        if not absent[b]:
                            expect[lo:hi, :, slots[b]] = q["vals"][lo:hi, :, b]
                    used_dst.update(int(x) for x in slots)
                    counts["retrieve"] += 1
                elif op == "release":
                    r = int(rng.choice(list(live)))
                    pool.release(r)
                    assert ora.release(r) == 0
                    free_src.extend(int(x) for x in live[r]["src"])
                    del live[r]
                    counts["release"] += 1
                elif op == "toggle":
                    o = int(rng.integers(2))
                    sdma[o] = not sdma[o]
                    # back to the library's defaults for the zero-copy kernel
                    default = K.LAUNCH_NT_STORE if o == K.OP_STORE else (K.LAUNCH_LDS if layout == 1 else 0)
                    upload = K.LAUNCH_UPLOAD if path_rng.random() < 0.5 else 0
                    pool.set_launch(K.CLASS_HOST, o, 0, (K.LAUNCH_SDMA if sdma[o] else default) | upload)
                    counts["toggle"] += 1
                if live and ext_rng.random() < 0.2:
                    # the next offload set of a live request: new blocks, their own ranges
                    r = int(ext_rng.choice(sorted(live)))
                    q = live[r]
                    m = int(ext_rng.integers(1, 13))
                    if len(free_src) >= m:
                        rc, om = ora.try_extend(r, m)
                        if rc != 0:
                            with pytest.raises(K.KVPoolError):
                                pool.extend(r, m)
                        else:
                            em = pool.extend(r, m)
                            assert np.array_equal(em.view(np.uint8), om.view(np.uint8)), "extension differs"
                            slots = np.array([free_src.pop() for _ in range(m)], np.int64)
                            vals = np.stack([kvgen.block_values(seed, r, b, L, H, BS, D)
                                             for b in range(q["n"], q["n"] + m)], 2)
                            src[:, :, torch.from_numpy(slots).to(dev)] = torch.from_numpy(vals.view(np.int16)).to(dev)
                            for s_ in streams:
                                s_.wait_stream(torch.cuda.current_stream())
                            q["map"] = np.concatenate([q["map"], em])
                            q["src"] = np.concatenate([q["src"], slots.astype(np.int32)])
                            q["vals"] = np.concatenate([q["vals"], vals], 2)
                            q["n"] += m
                            q["stored"] = False          # the new blocks hold nothing until stored
                            counts["extend"] += 1
            torch.cuda.synchronize()
            got = dst.cpu().numpy().view(np.uint16)
            if not np.array_equal(got, expect):
                bad = np.argwhere(got != expect)
                raise AssertionError("round %d: %d elements differ, first %s" % (rnd, len(bad), bad[:4].tolist()))
        say("lifecycle", layout, seed, counts)
        if seed == SEED and ROUNDS == 12:     # the default run exercises every kind of operation
            assert counts["retrieve"] >= 10 and counts["release"] >= 5 and counts["toggle"] >= 3
            assert counts["nospace"] >= 1 and counts["extend"] >= 5
    finally:
        torch.cuda.synchronize()
        pool.close()
        ora.close()
