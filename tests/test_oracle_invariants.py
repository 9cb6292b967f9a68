"""Pins of the oracle by invariants, closed forms and special cases.

* Exchange invariant: swapping two adjacent requests of the same class
  changes the total wait by exactly (later length - earlier length) >= 0, so
  no such swap improves the schedule; swapping across classes breaks the
  rank order that Eq. 2 requires.
* Closed forms: total = sum_k (n-1-k) * l[order[k]]; the class totals add up
  to the total; the last wait plus the last length is the sum of lengths.
* Special cases that reduce to textbook policies: one class gives
  shortest-job-first (a stable argsort by length); constant length L gives a
  stable counting sort by rank with wait[k] = k*L and total = L*n(n-1)/2;
  all keys equal gives the identity order.
* The hand-worked example in tests/golden/hand_example.json.
* Input validation.
"""

import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import OracleRangeError, schedule_batched, schedule_queue

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def total_of(order, length):
    """Total exclusive wait of an arbitrary order, by direct simulation."""
    t, s = 0, 0
    for i in order:
        s += t
        t += length[i]
    return s


queues = st.integers(0, 40).flatmap(
    lambda n: st.tuples(
        st.lists(st.integers(0, 4), min_size=n, max_size=n),
        st.lists(st.integers(0, 12), min_size=n, max_size=n)))


@settings(max_examples=200, deadline=None)
@given(queues)
def test_exchange_invariant(q):
    rank, length = q
    order, wait, totals = schedule_queue(rank, length, 5)
    base = total_of(order, length)
    assert base == totals[0]
    for k in range(len(order) - 1):
        a, b = order[k], order[k + 1]
        swapped = order[:k] + [b, a] + order[k + 2:]
        if rank[a] == rank[b]:
            delta = total_of(swapped, length) - base
            assert delta == length[b] - length[a]
            assert delta >= 0
        else:
            # a cross-class swap would serve a less urgent request first
            assert rank[a] < rank[b]


@settings(max_examples=200, deadline=None)
@given(queues)
def test_closed_forms(q):
    rank, length = q
    n = len(rank)
    order, wait, totals = schedule_queue(rank, length, 5)
    assert sorted(order) == list(range(n))
    assert totals[0] == sum((n - 1 - k) * length[order[k]] for k in range(n))
    assert totals[0] == sum(totals[1:])
    if n:
        assert wait[0] == 0
        assert wait[-1] + length[order[-1]] == sum(length)
    for k in range(1, n):
        assert wait[k] - wait[k - 1] == length[order[k - 1]]
    for c in range(5):
        assert totals[1 + c] == sum(wait[k] for k in range(n) if rank[order[k]] == c)


@pytest.mark.parametrize("seed", range(5))
def test_single_class_is_sjf(seed):
    rng = np.random.default_rng(seed)
    n = 300
    length = rng.integers(0, 50, n)
    order, _, _ = schedule_queue([0] * n, length.tolist(), 1)
    assert order == np.argsort(length, kind="stable").tolist()


def counting_sort_by_rank(rank, classes):
    count = [0] * classes
    for r in rank:
        count[r] += 1
    start = [0] * classes
    for c in range(1, classes):
        start[c] = start[c - 1] + count[c - 1]
    out = [None] * len(rank)
    for i, r in enumerate(rank):
        out[start[r]] = i
        start[r] += 1
    return out


@pytest.mark.parametrize("seed", range(5))
def test_constant_length_is_counting_sort(seed):
    rng = np.random.default_rng(100 + seed)
    n, L, classes = 257, int(rng.integers(0, 1000)), 7
    rank = rng.integers(0, classes, n).tolist()
    order, wait, totals = schedule_queue(rank, [L] * n, classes)
    assert order == counting_sort_by_rank(rank, classes)
    assert wait == [k * L for k in range(n)]
    assert totals[0] == L * n * (n - 1) // 2


def test_all_keys_equal_is_identity():
    order, wait, totals = schedule_queue([3] * 50, [7] * 50, 4)
    assert order == list(range(50))
    assert totals[4] == totals[0] == 7 * 50 * 49 // 2
    assert totals[1] == totals[2] == totals[3] == 0


def test_empty_and_single():
    assert schedule_queue([], [], 4) == ([], [], [0] * 5)
    assert schedule_queue([2], [9], 4) == ([0], [0], [0] * 5)


def test_hand_worked_example():
    with open(os.path.join(GOLDEN, "hand_example.json")) as f:
        g = json.load(f)
    order, wait, totals = schedule_queue(g["priority"], g["length"], g["num_classes"])
    assert order == g["order"]
    assert wait == g["wait"]
    assert totals == g["totals"]


def test_batched_is_per_queue():
    p = [1, 0, 1, 0, 0, 2, 2]
    l = [4, 4, 1, 9, 3, 5, 5]
    off = [0, 3, 3, 7]
    order, wait, totals = schedule_batched(p, l, off, 3)
    assert order == [1, 2, 0, 1, 0, 2, 3]
    assert wait == [0, 4, 5, 0, 3, 12, 17]
    assert totals == [9, 0, 9, 0, 0, 0, 0, 0, 32, 3, 0, 29]


def test_range_errors():
    with pytest.raises(OracleRangeError):
        schedule_queue([0, 1], [3, -1], 4)
    with pytest.raises(OracleRangeError):
        schedule_queue([0, 4], [3, 1], 4)
    with pytest.raises(ValueError):
        schedule_queue([0], [1], 0)
    with pytest.raises(ValueError):
        schedule_batched([0, 0], [1, 1], [0, 3, 2], 2)
    with pytest.raises(ValueError):
        schedule_batched([0, 0], [1, 1], [1, 2], 2)
