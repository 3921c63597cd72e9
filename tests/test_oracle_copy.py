"""Pins of the oracle's store (offload) and gather (retrieval) copies.

References independent of the oracle's memcpy loops: a pure-Python element
loop on tiny shapes, numpy advanced indexing / axis swaps on a single-device
pool, the identity block table, and the store->retrieve round trip.
"""
import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

import oracle

SENT = 0xBEEF


def _cache(L, slots, H, bs, D, fill=None, rng=None):
    if rng is not None:
        return rng.integers(0, 1 << 16, size=(L, 2, slots, H, bs, D), dtype=np.uint16)
    return np.full((L, 2, slots, H, bs, D), SENT if fill is None else fill, dtype=np.uint16)


def _layers(c):
    return [c[l, 0] for l in range(c.shape[0])], [c[l, 1] for l in range(c.shape[0])]


def _place(weights, n, bb):
    p = oracle.Pool(weights, [(n + 2) * bb * 2 + 8192] * len(weights), bb)
    return p, p.place(1, n)


def _regions(p, weights, n, bb):
    return [np.zeros((n + 2) * bb * 2 + 8192, dtype=np.uint8) for _ in weights]


def test_element_loop_tiny_both_layouts():
    L, H, bs, D = 2, 2, 2, 4
    C = H * bs * D * 2
    bb = 2 * L * C
    rng = np.random.default_rng(5)
    for layout in (0, 1):
        w, n = [2, 1], 5
        p, m = _place(w, n, bb)
        regs = _regions(p, w, n, bb)
        src = _cache(L, 7, H, bs, D, rng=rng)
        src_slots = np.array([6, 0, 3, 2, 5], np.int32)
        oracle.store(m, src_slots, regs, *_layers(src), (L, H, bs, D, 2), layout)
        # expected pool bytes by an element loop written from the layout definition
        for b in range(n):
            r, off = int(m["region"][b]), int(m["offset"][b])
            pool16 = regs[r][off:off + bb].view(np.uint16)
            for l in range(L):
                for kv in range(2):
                    for h in range(H):
                        for t in range(bs):
                            for d in range(D):
                                if layout == 0:
                                    e = (((2 * l + kv) * H + h) * bs + t) * D + d
                                else:
                                    e = (((2 * l + kv) * bs + t) * H + h) * D + d
                                assert pool16[e] == src[l, kv, src_slots[b], h, t, d]
        dst = _cache(L, 9, H, bs, D)
        dst_slots = np.array([8, 1, 4, 0, 7], np.int32)
        oracle.gather(m, dst_slots, regs, *_layers(dst), (L, H, bs, D, 2), layout)
        for b in range(n):
            for l in range(L):
                for kv in range(2):
                    for h in range(H):
                        for t in range(bs):
                            for d in range(D):
                                assert dst[l, kv, dst_slots[b], h, t, d] == src[l, kv, src_slots[b], h, t, d]
        untouched = sorted(set(range(9)) - set(dst_slots.tolist()))
        assert np.all(dst[:, :, untouched] == SENT)


@pytest.mark.parametrize("layout", [0, 1])
def test_single_device_gather_equals_numpy_indexing(layout):
    """N = 1: the region holds blocks in index order, so the gather is an
    advanced-indexing assignment on a view of the region."""
    L, H, bs, D = 3, 4, 16, 8
    C = H * bs * D * 2
    bb = 2 * L * C
    n = 11
    rng = np.random.default_rng(7)
    p = oracle.Pool([1], [(n * bb + 4095) // 4096 * 4096], bb)
    m = p.place(1, n)
    assert list(m["offset"]) == [b * bb for b in range(n)]
    region = rng.integers(0, 256, size=n * bb, dtype=np.uint8)
    dst = _cache(L, 20, H, bs, D)
    dst_slots = rng.permutation(20)[:n].astype(np.int32)
    oracle.gather(m, dst_slots, [region], *_layers(dst), (L, H, bs, D, 2), layout)
    if layout == 0:
        pool = region.view(np.uint16).reshape(n, L, 2, H, bs, D)
        expect = pool.transpose(1, 2, 0, 3, 4, 5)                  # [L][2][n][H][bs][D]
    else:
        pool = region.view(np.uint16).reshape(n, L, 2, bs, H, D)
        expect = pool.transpose(1, 2, 0, 4, 3, 5)                  # token-major -> head-major
    assert np.array_equal(dst[:, :, dst_slots], expect)


def test_identity_table_is_layer_slice():
    L, H, bs, D = 2, 2, 16, 16
    C = H * bs * D * 2
    bb = 2 * L * C
    n = 6
    p = oracle.Pool([1], [n * bb], bb)
    m = p.place(1, n)
    region = np.arange(n * bb // 2, dtype=np.uint16).view(np.uint8)
    dst = _cache(L, n, H, bs, D)
    oracle.gather(m, np.arange(n, dtype=np.int32), [region], *_layers(dst), (L, H, bs, D, 2), 0)
    pool = region.view(np.uint16).reshape(n, L, 2, C // 2)
    for l in range(L):
        for kv in range(2):
            assert np.array_equal(dst[l, kv].reshape(n, -1), pool[:, l, kv])


@settings(max_examples=40, deadline=None)
@given(st.lists(st.integers(1, 5), min_size=1, max_size=5), st.integers(1, 30),
       st.integers(1, 3), st.sampled_from([1, 2, 4]), st.sampled_from([1, 2, 16]),
       st.sampled_from([4, 8, 64]), st.integers(0, 1), st.integers(0, 2**31))
def test_round_trip_identity(weights, n, L, H, bs, D, layout, seed):
    C = H * bs * D * 2
    bb = 2 * L * C
    rng = np.random.default_rng(seed)
    p, m = _place(weights, n, bb)
    regs = _regions(p, weights, n, bb)
    src = _cache(L, n + 3, H, bs, D, rng=rng)
    src_slots = rng.permutation(n + 3)[:n].astype(np.int32)
    oracle.store(m, src_slots, regs, *_layers(src), (L, H, bs, D, 2), layout)
    dst = _cache(L, n + 5, H, bs, D)
    dst_slots = rng.permutation(n + 5)[:n].astype(np.int32)
    oracle.gather(m, dst_slots, regs, *_layers(dst), (L, H, bs, D, 2), layout)
    assert np.array_equal(dst[:, :, dst_slots], src[:, :, src_slots])
    rest = sorted(set(range(n + 5)) - set(dst_slots.tolist()))
    assert np.all(dst[:, :, rest] == SENT)


def test_absent_entries_are_skipped():
    L, H, bs, D = 2, 2, 4, 8
    C = H * bs * D * 2
    bb = 2 * L * C
    n = 8
    rng = np.random.default_rng(3)
    p, m = _place([1, 1], n, bb)
    regs = _regions(p, [1, 1], n, bb)
    src = _cache(L, n, H, bs, D, rng=rng)
    oracle.store(m, np.arange(n, dtype=np.int32), regs, *_layers(src), (L, H, bs, D, 2), 0)
    mm = m.copy()
    mm["region"][[1, 5, 6]] = oracle.ABSENT
    dst = _cache(L, n, H, bs, D)
    oracle.gather(mm, np.arange(n, dtype=np.int32), regs, *_layers(dst), (L, H, bs, D, 2), 0)
    for b in range(n):
        if b in (1, 5, 6):
            assert np.all(dst[:, :, b] == SENT)
        else:
            assert np.array_equal(dst[:, :, b], src[:, :, b])
