"""Pins of the oracle's target counts (Eq. 1, Eq. 2 and Algorithm 1's counting part).

Each check comes from something other than the oracle's own code: hand-worked
values of the closed form, exact rational arithmetic, and a brute-force search
over every count vector that Eq. (2) allows.
"""
import itertools
import os
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_counts():
    rows = []
    with open(os.path.join(GOLDEN, "counts.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            w, n, c = [x.strip() for x in line.split("|")]
            rows.append(([int(x) for x in w.split(",")], int(n), [int(x) for x in c.split(",")]))
    return rows


@pytest.mark.parametrize("weights,n,expect", _golden_counts())
def test_counts_golden(weights, n, expect):
    assert list(oracle.counts(weights, n)) == expect


def _floor_share(weights, n):
    """floor(p_i * n) with p_i = b_i / sum_j b_j in exact rational arithmetic (Eq. 1)."""
    W = sum(weights)
    return [int(Fraction(w, W) * n) for w in weights]


@settings(max_examples=300, deadline=None)
@given(st.lists(st.integers(1, 10**6), min_size=1, max_size=12), st.integers(0, 10**7))
def test_counts_closed_form(weights, n):
    c = [int(x) for x in oracle.counts(weights, n)]
    fl = _floor_share(weights, n)
    assert sum(c) == n                                       # sum constraint of Eq. (2)
    assert all(ci - fi in (0, 1) for ci, fi in zip(c, fl))   # r_i in {0, 1}
    W = sum(weights)
    # within one block: the deviation reaches exactly 1 only when a device
    # whose share p_i*n is an integer receives one of the leftovers
    assert all(abs(Fraction(ci) - Fraction(w * n, W)) <= 1 for ci, w in zip(c, weights))
    for ci, w in zip(c, weights):
        if abs(Fraction(ci) - Fraction(w * n, W)) == 1:
            assert (w * n) % W == 0 and ci == w * n // W + 1


def test_leftover_to_device_with_integral_share():
    """2:1:1 at n = 2: shares 1, 1/2, 1/2; the one leftover goes to the largest p_i
    (device 0), whose share was already whole -- one block above its share."""
    assert list(oracle.counts([2, 1, 1], 2)) == [2, 0, 0]


@settings(max_examples=100, deadline=None)
@given(st.lists(st.integers(1, 2**40), min_size=1, max_size=6), st.integers(0, 2**40))
def test_counts_large_values_exact(weights, n):
    """Products above 2**64 must not lose precision (b_i * n is formed exactly)."""
    c = [int(x) for x in oracle.counts(weights, n)]
    fl = _floor_share(weights, n)
    assert sum(c) == n and all(ci - fi in (0, 1) for ci, fi in zip(c, fl))


def _brute_force(weights, n):
    """Every vector Eq. (2) allows, filtered by the remainder rule, by enumeration.

    Allowed: c_i = floor(p_i n) + r_i, r_i >= 0, sum c_i = n.  Rule: leftovers go
    to devices with larger p_i, one each; equal p_i -> lower index first.  A
    vector obeys it when r_i <= 1 and no device with r = 0 outranks one with r = 1.
    """
    fl = _floor_share(weights, n)
    rank = sorted(range(len(weights)), key=lambda i: (-Fraction(weights[i], sum(weights)), i))
    pos = {i: k for k, i in enumerate(rank)}
    winners = []
    R = n - sum(fl)              # sum r_i = R and r_i >= 0, so each r_i lies in [0, R]
    for c in itertools.product(*[range(f, f + R + 1) for f in fl]):
        if sum(c) != n:
            continue
        r = [ci - fi for ci, fi in zip(c, fl)]
        if any(x > 1 for x in r):
            continue
        ok = all(not (r[i] == 0 and r[j] == 1 and pos[i] < pos[j])
                 for i in range(len(c)) for j in range(len(c)))
        if ok:
            winners.append(list(c))
    return winners


@pytest.mark.parametrize("n_dev", [1, 2, 3, 4])
def test_counts_brute_force_tiny(n_dev):
    top = 6 if n_dev < 4 else 5
    for weights in itertools.product(range(1, top), repeat=n_dev):
        for n in range(0, 13):
            winners = _brute_force(list(weights), n)
            assert len(winners) == 1, (weights, n, winners)
            assert [int(x) for x in oracle.counts(list(weights), n)] == winners[0], (weights, n)


def test_counts_single_device_takes_all():
    for n in (0, 1, 17, 8192):
        assert list(oracle.counts([5], n)) == [n]


def test_literal_single_device_remainder_breaks_one_block_bound():
    """Why the remainder goes to several devices (reading of Sec. 4.1.3 vs Algorithm 1).

    Giving all r leftovers to the one largest-p_i device would put device 0 of
    a 4:4:1:1:1:1 pool more than one block above its share p_0 * n at n = 8192;
    the plural reading keeps every device within one block.
    """
    w, n = [4, 4, 1, 1, 1, 1], 8192
    fl = _floor_share(w, n)
    literal = list(fl)
    literal[0] += n - sum(fl)
    assert abs(Fraction(literal[0]) - Fraction(w[0] * n, sum(w))) > 1
    c = oracle.counts(w, n)
    assert all(abs(Fraction(int(ci)) - Fraction(wi * n, sum(w))) < 1 for ci, wi in zip(c, w))


def test_counts_rejects_zero_bandwidth():
    with pytest.raises(ValueError):
        oracle.counts([1, 0], 4)
    with pytest.raises(ValueError):
        oracle.counts([], 4)


def test_counts_are_uint64_array():
    c = oracle.counts([1, 1], 3)
    assert c.dtype == np.uint64 and list(c) == [2, 1]
