"""Helpers of the GPU tests: run a workload through the library and compare
with the oracle.  Only the tests import this module."""
import sys

import numpy as np

import kvgen
import oracle
from paper_2606_14779_amd.runner import SENTINEL, WorkloadRun


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def oracle_pool(wl):
    return oracle.Pool([r.weight for r in wl.regions], [r.capacity_bytes for r in wl.regions],
                       wl.shape.block_bytes)


def oracle_expectation(wl, run, host_src, ora=None):
    """Oracle placement, pool contents and destination cache for a whole workload."""
    sh = wl.shape
    L = sh.layers
    shape = (L, sh.kv_heads, sh.block_size, sh.head_dim, sh.elem_bytes)
    ora = ora or oracle_pool(wl)
    regions = [np.zeros(r.capacity_bytes, np.uint8) for r in wl.regions]
    expect = np.full(tuple(run.dst.shape), SENTINEL, np.uint16)
    maps = {}
    for q in wl.requests:
        m = ora.place(q.request_id, q.n_present)
        maps[q.request_id] = m
        oracle.store(m, q.src_slots, regions, [host_src[l, 0] for l in range(L)],
                     [host_src[l, 1] for l in range(L)], shape, wl.layout)
    for q in wl.requests:
        full = np.zeros(q.n_blocks, dtype=oracle.LOC_DTYPE)
        full[:q.n_present] = maps[q.request_id]
        full["region"][q.n_present:] = oracle.ABSENT
        oracle.gather(full, q.dst_slots, regions, [expect[l, 0] for l in range(L)],
                      [expect[l, 1] for l in range(L)], shape, wl.layout)
    return maps, regions, expect


def check_full(wl, run, host_src, ora=None):
    """Element-by-element comparison of maps, pool bytes and destination.

    ``ora``: an oracle pool carrying the same place/release history as the
    library's pool before the workload's placements (default: a fresh one)."""
    maps, regions, expect = oracle_expectation(wl, run, host_src, ora)
    bb = wl.shape.block_bytes
    for q in wl.requests:
        assert np.array_equal(run.maps[q.request_id], maps[q.request_id]), "placement differs"
        m = maps[q.request_id]
        for r in range(len(wl.regions)):
            offs = m["offset"][m["region"] == r]
            if len(offs) == 0:
                continue
            lo, hi = int(offs.min()), int(offs.max()) + bb
            got = run.pool.region_read(r, lo, hi - lo)
            assert np.array_equal(got, regions[r][lo:hi]), "pool region %d bytes differ" % r
    got = run.dst.cpu().numpy().view(np.uint16)
    if not np.array_equal(got, expect):
        bad = np.argwhere(got != expect)
        raise AssertionError("destination differs at %d elements, first %s" % (len(bad), bad[:4].tolist()))


def check_sampled(wl, run, n_sample=48, seed=0):
    """Full-size check: sampled blocks through the oracle, every block by round trip,
    every untouched slot by sentinel."""
    sh = wl.shape
    L, bb = sh.layers, sh.block_bytes
    shape = (L, sh.kv_heads, sh.block_size, sh.head_dim, sh.elem_bytes)
    rng = np.random.default_rng(seed)
    ora = oracle.Pool([r.weight for r in wl.regions], [r.capacity_bytes for r in wl.regions], bb)
    for q in wl.requests:
        om = ora.place(q.request_id, q.n_present)
        assert np.array_equal(om, run.maps[q.request_id]), "placement differs"
        picks = {0, q.n_present - 1} | set(rng.integers(0, q.n_present, n_sample).tolist())
        for b in sorted(picks):
            vals = kvgen.block_values(wl.seed, q.request_id, b, L, sh.kv_heads, sh.block_size, sh.head_dim)
            src1 = np.ascontiguousarray(vals[:, :, None])           # [L][2][1 slot][H][bs][D]
            loc = np.zeros(1, dtype=oracle.LOC_DTYPE)               # same block in a 1-block pool
            reg = np.zeros(bb, np.uint8)
            oracle.store(loc, [0], [reg], [src1[l, 0] for l in range(L)], [src1[l, 1] for l in range(L)],
                         shape, wl.layout)
            got_pool = run.pool.region_read(int(om["region"][b]), int(om["offset"][b]), bb)
            assert np.array_equal(got_pool, reg), "pool block %d of request %d differs" % (b, q.request_id)
            dst1 = np.full_like(src1, SENTINEL)
            oracle.gather(loc, [0], [reg], [dst1[l, 0] for l in range(L)], [dst1[l, 1] for l in range(L)],
                          shape, wl.layout)
            slot = int(q.dst_slots[b])
            got = run.dst[:, :, slot].cpu().numpy().view(np.uint16)
            assert np.array_equal(got, dst1[:, :, 0]), "dst slot %d (block %d) differs" % (slot, b)
    check_round_trip(wl, run)


def check_every_block(wl, run, host_src):
    """Full-size check of every block: the pool bytes of every present block equal the oracle's
    store of the same source (regions compared span by span), and every destination slot equals its
    source slot (round trip, on the GPU).  Since the oracle's gather of its own store returns the
    source (pinned on the CPU), the destination then equals the oracle's gather for every block."""
    sh = wl.shape
    L, bb = sh.layers, sh.block_bytes
    shape = (L, sh.kv_heads, sh.block_size, sh.head_dim, sh.elem_bytes)
    ora = oracle_pool(wl)
    regions = [np.zeros(r.capacity_bytes, np.uint8) for r in wl.regions]
    for q in wl.requests:
        m = ora.place(q.request_id, q.n_present)
        assert np.array_equal(m, run.maps[q.request_id]), "placement differs"
        oracle.store(m, q.src_slots, regions, [host_src[l, 0] for l in range(L)],
                     [host_src[l, 1] for l in range(L)], shape, wl.layout)
        for r in range(len(wl.regions)):
            offs = m["offset"][m["region"] == r]
            if len(offs) == 0:
                continue
            lo, hi = int(offs.min()), int(offs.max()) + bb
            got = run.pool.region_read(r, lo, hi - lo)
            if not np.array_equal(got, regions[r][lo:hi]):
                bad = np.flatnonzero(got != regions[r][lo:hi])
                raise AssertionError("region %d: %d bytes differ from the oracle's store, first at offset %d"
                                     % (r, len(bad), lo + int(bad[0])))
            del got
    del regions
    check_round_trip(wl, run)


def check_round_trip(wl, run):
    """Every present block: retrieve(store(x)) == x, layer by layer on the GPU; every other slot
    still holds the sentinel."""
    import torch
    L = wl.shape.layers
    dev = run.dst.device
    touched = np.zeros(wl.dst_num_slots, bool)
    for q in wl.requests:
        ds = torch.from_numpy(q.dst_slots[:q.n_present].astype(np.int64)).to(dev)
        ss = torch.from_numpy(q.src_slots.astype(np.int64)).to(dev)
        touched[q.dst_slots[:q.n_present]] = True
        for l in range(L):
            assert torch.equal(run.dst[l].index_select(1, ds), run.src[l].index_select(1, ss)), \
                "round trip differs in layer %d of request %d" % (l, q.request_id)
    rest = torch.from_numpy(np.flatnonzero(~touched).astype(np.int64)).to(dev)
    sent = int(np.uint16(SENTINEL).view(np.int16))
    for l in range(L):
        assert bool((run.dst[l].index_select(1, rest) == sent).all()), "untouched slot changed (layer %d)" % l


def make_run(wl, **kw):
    run = WorkloadRun(wl, device=0, **kw)
    return run


def tag_cache(L, S, H, bs, D):
    """Source cache whose every 16-byte vector names itself: (slot, layer, K/V, head, token, vector,
    0x5A5A, 0x0F0F) as eight 16-bit words, [L][2][S][H][bs][D]."""
    nv = D // 8
    t = np.zeros((L, 2, S, H, bs, nv, 8), np.int16)
    t[..., 0] = np.arange(S, dtype=np.int16)[None, None, :, None, None, None]
    t[..., 1] = np.arange(L, dtype=np.int16)[:, None, None, None, None, None]
    t[..., 2] = np.arange(2, dtype=np.int16)[None, :, None, None, None, None]
    t[..., 3] = np.arange(H, dtype=np.int16)[None, None, None, :, None, None]
    t[..., 4] = np.arange(bs, dtype=np.int16)[None, None, None, None, :, None]
    t[..., 5] = np.arange(nv, dtype=np.int16)[None, None, None, None, None, :]
    t[..., 6] = 0x5A5A
    t[..., 7] = 0x0F0F
    return t.reshape(L, 2, S, H, bs, D)


def check_tags(tags, dst, src_slots, dst_slots, sentinel):
    """Every destination slot dst_slots[b] must hold, vector for vector, the tags of source slot
    src_slots[b] (same layer, K/V, head, token, vector); every other slot the sentinel.  A wrong
    vector is reported by the coordinates it sits at and the tag it holds."""
    L, _, S, H, bs, D = tags.shape
    t = tags.reshape(L, 2, S, H, bs, D // 8, 8)
    got = dst.reshape(L, 2, dst.shape[2], H, bs, D // 8, 8)
    for b in range(len(src_slots)):
        want, have = t[:, :, src_slots[b]], got[:, :, dst_slots[b]]
        if not np.array_equal(have, want):
            bad = np.argwhere(np.any(have != want, axis=-1))[0]
            raise AssertionError("block %d, slot %d, (layer, kv, head, token, vector) %s holds tag %s, expected %s"
                                 % (b, dst_slots[b], bad.tolist(), have[tuple(bad)].tolist(),
                                    want[tuple(bad)].tolist()))
    untouched = np.setdiff1d(np.arange(dst.shape[2]), np.asarray(dst_slots))
    assert np.all(got[:, :, untouched] == sentinel), "a slot no block names was written"
