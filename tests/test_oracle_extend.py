"""Pins of the oracle's extension of a placed request (Sec. 4.1.3: each
decoding step's KV caches form an offload set of their own, Algorithm 1 run on
that set; Sec. 4.2: each set's share of a device is one contiguous range).

Independent references: a hand-worked sequence of one place and four
extensions (tests/golden/extend.txt), Eq. 2's closed form per set checked in
exact rationals, invariants every valid placement must satisfy, and the
defining property of reading R6 -- an extension lands exactly where a fresh
request of the same size would on the same pool state.
"""
import os
from fractions import Fraction

import numpy as np
from hypothesis import given, settings
from hypothesis import strategies as st

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
SECTOR = 4096


def _read_golden():
    head, steps = {}, []
    with open(os.path.join(GOLDEN, "extend.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith(("place ", "extend ")):
                op, n = line.split()
                steps.append({"op": op, "n": int(n)})
            else:
                k, v = line.split(":", 1)
                vals = [int(x) for x in v.split(",")]
                if steps:
                    steps[-1][k.strip()] = vals
                else:
                    head[k.strip()] = vals
    return head, steps


def test_extend_golden():
    head, steps = _read_golden()
    w, bb, cap = head["weights"], head["block_bytes"][0], head["capacity"][0]
    p = oracle.Pool(w, [cap] * len(w), bb)
    total = []
    for s in steps:
        m = p.place(1, s["n"]) if s["op"] == "place" else p.extend(1, s["n"])
        assert list(m["region"]) == s["regions"], s
        assert list(m["offset"]) == s["offsets"], s
        assert set(m["gen"].tolist()) == {1}
        total.append(m)
    whole = np.concatenate(total)
    assert np.array_equal(p.lookup(1, len(whole)), whole)
    assert p.release(1) == 0
    assert all(p.largest_free(i) == cap for i in range(len(w)))


def _closed_form(weights, n, m):
    """Eq. 2 per set: every device's count is floor(w_i n / W) or one more, summing to n."""
    W = sum(weights)
    counts = np.bincount(m["region"].astype(np.int64), minlength=len(weights))
    assert counts.sum() == n
    for i, w in enumerate(weights):
        share = Fraction(w * n, W)
        floor = share.numerator // share.denominator
        assert floor <= int(counts[i]) <= floor + 1


@settings(max_examples=150, deadline=None)
@given(st.lists(st.integers(1, 9), min_size=1, max_size=6),
       st.lists(st.integers(1, 40), min_size=1, max_size=8), st.integers(1, 3))
def test_extensions_keep_earlier_blocks_and_stay_valid(weights, sizes, block_sectors):
    bb = block_sectors * SECTOR
    cap = (sum(sizes) + 8) * bb
    p = oracle.Pool(weights, [cap] * len(weights), bb)
    maps = []
    for k, n in enumerate(sizes):
        m = p.place(7, n) if k == 0 else p.extend(7, n)
        _closed_form(weights, n, m)
        maps.append(m)
        whole = np.concatenate(maps)
        assert np.array_equal(p.lookup(7, len(whole)), whole)       # earlier entries never move
    whole = np.concatenate(maps)
    assert set(whole["gen"].tolist()) == {int(maps[0]["gen"][0])}
    keys = set(zip(whole["region"].tolist(), whole["offset"].tolist()))
    assert len(keys) == len(whole)                                    # every block its own place
    assert np.all(whole["offset"] % bb % SECTOR == 0)
    assert np.all(whole["offset"] + bb <= cap)
    # each set's share of a device is one contiguous run of blocks
    for m in maps:
        for r in np.unique(m["region"]):
            offs = np.sort(m["offset"][m["region"] == r])
            assert np.all(np.diff(offs) == bb)
    assert p.release(7) == 0
    assert all(p.largest_free(i) == cap // SECTOR * SECTOR for i in range(len(weights)))


@settings(max_examples=100, deadline=None)
@given(st.lists(st.integers(1, 9), min_size=1, max_size=6), st.integers(1, 30), st.integers(1, 30),
       st.integers(1, 30))
def test_extension_lands_where_a_new_request_would(weights, n0, n_other, n_new):
    """R6: an extension is an offload set of its own.  Two pools with the same history; in one the
    request is extended, in the other a new request of the same size is placed: same places."""
    bb = SECTOR
    cap = (n0 + n_other + n_new + 8) * bb
    a = oracle.Pool(weights, [cap] * len(weights), bb)
    b = oracle.Pool(weights, [cap] * len(weights), bb)
    for p in (a, b):
        p.place(1, n0)
        p.place(2, n_other)
        p.release(2)                      # leave a hole before the extension
    ext = a.extend(1, n_new)
    new = b.place(3, n_new)
    assert np.array_equal(ext["region"], new["region"])
    assert np.array_equal(ext["offset"], new["offset"])


def test_extension_failure_changes_nothing():
    w = [2, 1]
    bb = SECTOR
    p = oracle.Pool(w, [8 * bb, 4 * bb], bb)
    first = p.place(1, 6)                                   # 4 + 2 blocks
    before = [p.largest_free(i) for i in range(2)]
    rc, _ = p.try_extend(1, 9)                              # 6 + 3: device 0 has room for 4 only
    assert rc == -3
    assert np.array_equal(p.lookup(1, 6), first)
    assert [p.largest_free(i) for i in range(2)] == before
    m = p.extend(1, 3)                                      # 2 + 1 fits
    assert list(m["region"]) == [0, 1, 0]
    assert np.array_equal(p.lookup(1, 9), np.concatenate([first, m]))


def test_extension_error_codes():
    p = oracle.Pool([1, 1], [1 << 20, 1 << 20], SECTOR)
    assert p.try_extend(5, 3)[0] == -4                      # not placed
    p.place(5, 2)
    assert p.try_extend(5, 0)[0] == -1                      # empty set
    assert p.release(5) == 0
    assert p.try_extend(5, 1)[0] == -4                      # released
