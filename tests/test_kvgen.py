"""Checks of the seeded input generator (not part of the method)."""
import numpy as np

import kvgen
from kvgen import workloads


def _as_f32(u16):
    return (u16.astype(np.uint32) << 16).view(np.float32)


def test_block_values_deterministic_and_independent():
    a = kvgen.block_values(11, 2, 5, 2, 2, 16, 8)
    b = kvgen.block_values(11, 2, 5, 2, 2, 16, 8)
    c = kvgen.block_values(11, 2, 6, 2, 2, 16, 8)
    d = kvgen.block_values(11, 3, 5, 2, 2, 16, 8)
    assert np.array_equal(a, b)
    assert not np.array_equal(a, c) and not np.array_equal(a, d)


def test_elems_offsets_consistent():
    full = kvgen.elems(1, 1, 1, 0, 1001)
    for e0, cnt in [(1, 10), (7, 1), (500, 501), (0, 1), (999, 2)]:
        assert np.array_equal(kvgen.elems(1, 1, 1, e0, cnt), full[e0:e0 + cnt])


def test_fill_cache_matches_block_values():
    L, H, bs, D = 3, 2, 16, 8
    slots = 9
    cache = np.zeros((L, 2, slots, H, bs, D), dtype=np.uint16)
    ids = np.array([4, 0, 7, 2], dtype=np.uint64)
    sl = np.array([8, 1, 3, 5], dtype=np.int32)
    kp = [cache[l, 0].ctypes.data for l in range(L)]
    vp = [cache[l, 1].ctypes.data for l in range(L)]
    kvgen.fill_cache(77, 5, ids, sl, L, H, bs, D, kp, vp, threads=3)
    for blk, s in zip(ids, sl):
        v = kvgen.block_values(77, 5, int(blk), L, H, bs, D)
        assert np.array_equal(cache[:, :, s], v)
    assert np.all(cache[:, :, [0, 2, 4, 6, 7]] == 0)


def test_values_are_standard_normal_bf16():
    v = _as_f32(kvgen.elems(1003, 1, 0, 0, 1 << 21)).astype(np.float64)
    assert np.all(np.isfinite(v))
    assert abs(v.mean()) < 0.005 and abs(v.std() - 1.0) < 0.005
    assert abs(np.mean(np.abs(v) < 1.0) - 0.6827) < 0.003
    assert abs(np.mean(np.abs(v) < 2.0) - 0.9545) < 0.002


def _bf16_rne(x):
    """Round float64 values to bf16 bits (ties to even) with exact comparisons."""
    f = x.astype(np.float32)
    u = f.view(np.uint32)
    lo = (u & 0xFFFF0000).astype(np.uint32)
    hi = lo + 0x10000
    dlo = np.abs(x - lo.view(np.float32).astype(np.float64))
    dhi = np.abs(hi.view(np.float32).astype(np.float64) - x)
    pick_hi = (dhi < dlo) | ((dhi == dlo) & ((lo >> 16) & 1 == 1))
    return np.where(pick_hi, hi >> 16, lo >> 16).astype(np.uint16)


def test_normal_table_matches_scipy_quantiles():
    from scipy.special import ndtri
    q = kvgen.normal_table()
    expect = _bf16_rne(ndtri((np.arange(65536) + 0.5) / 65536.0))
    assert np.array_equal(q, expect)
    assert abs(kvgen.ppnd16(0.975) - 1.959963984540054) < 1e-14
    assert kvgen.ppnd16(0.5) == 0.0


def test_workloads_structure_full_size():
    bytes_expect = {1: 2 * 2**30, 2: 8 * 2**30, 3: 16 * 2**30, 4: 6 * 2**30}
    for cfg in (1, 2, 3, 4):
        wl = workloads.make(cfg)
        assert wl.retrieved_bytes == bytes_expect[cfg]
        r = wl.requests[0]
        assert len(np.unique(r.dst_slots)) == r.n_blocks
        assert r.dst_slots.min() >= 0 and r.dst_slots.max() < wl.dst_num_slots
        assert len(np.intersect1d(r.dst_slots, wl.occupied_dst_slots)) == 0
    wl3 = workloads.make(3)
    assert wl3.dst_num_slots == 10240 and len(wl3.occupied_dst_slots) == 2048
    assert np.all(np.diff(wl3.requests[0].dst_slots) > 0)           # free slots ascending
    wl5 = workloads.make(5)
    assert len(wl5.requests) == 4 and wl5.n_streams == 4
    all_dst = np.concatenate([q.dst_slots[:q.n_present] for q in wl5.requests])
    assert len(np.unique(all_dst)) == len(all_dst) and all_dst.max() < wl5.dst_num_slots
    for q in wl5.requests:
        assert 16384 // 16 <= q.n_blocks <= 131072 // 16
        assert q.n_blocks // 2 - 1 <= q.n_present <= q.n_blocks
        assert np.all(q.dst_slots[q.n_present:] == -1)


def test_workloads_scaled_keep_structure():
    for cfg in (1, 2, 3, 4, 5):
        wl = workloads.make(cfg, max_blocks=37)
        assert all(q.n_blocks <= 37 for q in wl.requests)
        assert [r.weight for r in wl.regions] == [r.weight for r in workloads.make(cfg).regions]
