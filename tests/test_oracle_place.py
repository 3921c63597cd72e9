"""Pins of the oracle's placement: Algorithm 1's partition, the contiguous
range per (request, device) of Sec. 4.2, and the GLT record.

Independent references used here: a hand-worked block sequence, the smooth
weighted round-robin scheduler (nginx, M. Dounin 2012) which the deficit rule
must equal when n is a multiple of the total weight, plain round robin for
equal weights, a first-fit allocator's textbook behaviour, and invariants that
every valid placement must satisfy.
"""
import os

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
SECTOR = 4096


def _read_interleave():
    d = {}
    with open(os.path.join(GOLDEN, "interleave.txt")) as f:
        for line in f:
            if line.startswith("#") or ":" not in line:
                continue
            k, v = line.split(":", 1)
            d[k.strip()] = [int(x) for x in v.split(",")]
    return d["weights"], d["n"][0], d["sequence"]


def test_interleave_golden():
    w, n, seq = _read_interleave()
    p = oracle.Pool(w, [1 << 30] * len(w), 8192)
    m = p.place(1, n)
    assert list(m["region"]) == seq


def _smooth_wrr(weights, n):
    """nginx smooth weighted round robin: add w_i to every current weight, pick
    the largest (first on ties), subtract the total from the pick."""
    cur = [0] * len(weights)
    total = sum(weights)
    out = []
    for _ in range(n):
        for i, w in enumerate(weights):
            cur[i] += w
        best = max(range(len(weights)), key=lambda i: (cur[i], -i))
        cur[best] -= total
        out.append(best)
    return out


@settings(max_examples=200, deadline=None)
@given(st.lists(st.integers(1, 9), min_size=1, max_size=7), st.integers(1, 6))
def test_interleave_equals_smooth_wrr_when_exact(weights, periods):
    n = periods * sum(weights)
    p = oracle.Pool(weights, [1 << 32] * len(weights), SECTOR)
    assert list(p.place(3, n)["region"]) == _smooth_wrr(weights, n)


@pytest.mark.parametrize("N", [1, 2, 3, 6])
def test_equal_weights_round_robin(N):
    n = 5 * N
    p = oracle.Pool([3] * N, [1 << 30] * N, SECTOR)
    assert list(p.place(1, n)["region"]) == [j % N for j in range(n)]


def _check_invariants(p, weights, caps, block_bytes, live):
    """live: {request: map}.  Checks what any valid placement must satisfy."""
    used = [[] for _ in weights]
    for req, m in live.items():
        n = len(m)
        c = oracle.counts(weights, n)
        reg = m["region"].astype(np.int64)
        assert np.all(reg < len(weights))
        assert list(np.bincount(reg, minlength=len(weights))) == [int(x) for x in c]
        assert len(set(m["gen"])) == 1
        for i in range(len(weights)):
            offs = np.sort(m["offset"][reg == i].astype(np.int64))
            if len(offs) == 0:
                continue
            base = int(offs[0])
            # one contiguous run of c_i blocks (Sec. 4.2), sector aligned, in capacity
            assert base % SECTOR == 0
            assert np.all(offs == base + block_bytes * np.arange(len(offs)))
            length = (len(offs) * block_bytes + SECTOR - 1) // SECTOR * SECTOR
            assert base + length <= caps[i] // SECTOR * SECTOR
            used[i].append((base, base + length))
    for i, spans in enumerate(used):       # ranges of live requests are disjoint
        spans.sort()
        for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
            assert a1 <= b0, (i, spans)


@settings(max_examples=60, deadline=None)
@given(st.lists(st.integers(1, 8), min_size=1, max_size=6),
       st.sampled_from([4096, 8192, 12288, 1000, 3 * 4096 + 16]),
       st.lists(st.tuples(st.booleans(), st.integers(1, 70)), min_size=1, max_size=25))
def test_place_release_invariants(weights, block_bytes, ops):
    caps = [(w * 40 + 3) * block_bytes + 5000 for w in weights]
    p = oracle.Pool(weights, caps, block_bytes)
    live, next_req, last_gen = {}, 1, 0
    for is_release, n in ops:
        if is_release and live:
            req = sorted(live)[n % len(live)]
            assert p.release(req) == 0
            del live[req]
            continue
        rc, m = p.try_place(next_req, n)
        if rc == 0:
            assert int(m["gen"][0]) == last_gen + 1
            last_gen += 1
            live[next_req] = m.copy()
            assert np.array_equal(p.lookup(next_req, n), m)
        else:
            assert rc == -3
        next_req += 1
        _check_invariants(p, weights, caps, block_bytes, live)


def test_prefix_balance_on_workload_pools():
    """Quality of the striping: every prefix of the request stays within one block
    of its proportional share on every device (not an invariant of Algorithm 1)."""
    for w, n in [([1, 1], 1024), ([4, 4, 1, 1], 4096), ([4, 4, 1, 1, 1, 1], 8192),
                 ([3, 3, 1, 1], 8192)]:
        p = oracle.Pool(w, [1 << 40] * len(w), SECTOR)
        reg = p.place(1, n)["region"].astype(np.int64)
        c = oracle.counts(w, n).astype(np.float64)
        onehot = np.zeros((n, len(w)))
        onehot[np.arange(n), reg] = 1
        a = np.cumsum(onehot, axis=0)
        m = np.arange(1, n + 1)[:, None]
        assert np.max(np.abs(a - m * c[None, :] / n)) < 1.0


def test_first_fit_reuses_lowest_hole_and_coalesces():
    bb = 2 * SECTOR
    p = oracle.Pool([1], [100 * bb], bb)
    a = p.place(1, 10)
    b = p.place(2, 20)
    c = p.place(3, 10)
    assert int(a["offset"][0]) == 0 and int(b["offset"][0]) == 10 * bb and int(c["offset"][0]) == 30 * bb
    assert p.release(2) == 0
    d = p.place(4, 5)                       # first fit: lowest-addressed hole that fits
    assert int(d["offset"][0]) == 10 * bb
    e = p.place(5, 30)                      # too big for the hole -> after request 3
    assert int(e["offset"][0]) == 40 * bb
    for r in (1, 3, 4, 5):
        assert p.release(r) == 0
    assert p.largest_free(0) == 100 * bb     # everything coalesced back
    f = p.place(6, 100)
    assert int(f["offset"][0]) == 0


def test_no_space_changes_nothing():
    bb = SECTOR
    p = oracle.Pool([1, 1], [10 * bb, 4 * bb], bb)
    rc, _ = p.try_place(1, 12)               # device 1 would need 6 blocks, has 4
    assert rc == -3
    assert p.largest_free(0) == 10 * bb and p.largest_free(1) == 4 * bb
    m = p.place(2, 8)                        # gen is not consumed by the failure
    assert int(m["gen"][0]) == 1
    assert int(m["offset"][m["region"] == 0][0]) == 0


def test_lookup_and_release_errors():
    p = oracle.Pool([1, 2], [1 << 20, 1 << 20], SECTOR)
    m = p.place(9, 7)
    assert np.array_equal(p.lookup(9, 7), m)
    with pytest.raises(oracle.PlacementError):
        p.lookup(9, 6)
    with pytest.raises(oracle.PlacementError):
        p.place(9, 3)                        # already placed
    assert p.release(9) == 0
    assert p.release(9) == -4
    with pytest.raises(oracle.PlacementError):
        p.lookup(9, 7)


def test_sector_rounding_of_range_length():
    """Range length is ceil(c * KV_size / sector) sectors (Sec. 4.2)."""
    bb = 1000                                  # not a sector multiple
    p = oracle.Pool([1], [1 << 20], bb)
    a = p.place(1, 5)                          # 5000 B -> 2 sectors
    b = p.place(2, 1)
    assert int(a["offset"][0]) == 0 and list(a["offset"]) == [0, 1000, 2000, 3000, 4000]
    assert int(b["offset"][0]) == 2 * SECTOR
