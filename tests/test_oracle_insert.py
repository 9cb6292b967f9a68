"""Pins of the incremental oracle (insert_queue): Algorithm 1's HeapInsert.

The incremental schedule is pinned to a literal binary min-heap (the
library's ``heapq``) keyed by the priority tuple (rank, predicted length)
with the arrival index as the last key: earlier requests are pushed first,
the arrivals are pushed one by one, and draining the heap gives the order;
the waits are the running sum of lengths along it. No code is shared with
the oracle's sort.
"""

import heapq
import random

import pytest

from oracle import c_oracle_insert, insert_queue, schedule_queue
from workloads import fuzz_queue


def heap_drain(p, l):
    h = []
    for i in range(len(p)):
        heapq.heappush(h, (int(p[i]), int(l[i]), i))
    order, wait, acc = [], [], 0
    while h:
        _, li, i = heapq.heappop(h)
        order.append(i)
        wait.append(acc)
        acc += li
    return order, wait


@pytest.mark.parametrize("seed", range(12))
def test_insert_equals_heap_insertion(seed):
    rnd = random.Random(seed)
    n = rnd.randint(0, 60)
    n_old = rnd.randint(0, n)
    p = [rnd.randint(0, 3) for _ in range(n)]
    l = [rnd.randint(0, 6) for _ in range(n)]  # small ranges: many exact ties
    o_old, w_old, _ = schedule_queue(p[:n_old], l[:n_old])
    order, wait, totals = insert_queue(p, l, n_old, o_old, w_old)
    ho, hw = heap_drain(p, l)
    assert order == ho and wait == hw
    assert totals[0] == sum(hw)
    for c in range(4):
        assert totals[1 + c] == sum(w for o, w in zip(ho, hw) if p[o] == c)


def test_ties_go_to_the_earlier_request():
    # every arrival has the key of an earlier request
    p = [1, 0, 1, 0, 1, 0]
    l = [5, 5, 5, 5, 5, 5]
    o_old, w_old, _ = schedule_queue(p[:3], l[:3])
    order, _, _ = insert_queue(p, l, 3, o_old, w_old)
    assert order == [1, 3, 5, 0, 2, 4]


def test_chained_inserts_equal_one_schedule():
    p, l = fuzz_queue(500, seed=9, classes=5, max_len=40, tie_frac=0.3)
    cuts = [0, 1, 120, 121, 400, 500]
    o, w, _ = schedule_queue(p[:0], l[:0])
    for a, b in zip(cuts, cuts[1:]):
        o, w, t = insert_queue(p[:b], l[:b], a, o, w)
    assert (o, w, t) == schedule_queue(p, l)


def test_wrong_earlier_schedule_is_rejected():
    p, l = [0, 1, 2], [3, 2, 1]
    with pytest.raises(ValueError):
        insert_queue(p, l, 2, [1, 0], [0, 2])


def test_c_oracle_insert_matches_python():
    import numpy as np
    p, l = fuzz_queue(3000, seed=4, classes=6, max_len=200, tie_frac=0.3)
    o_old, w_old, _ = schedule_queue(p[:1700], l[:1700])
    co, cw, ct = c_oracle_insert(p, l, 1700, np.array(o_old, np.int32),
                                 np.array(w_old, np.int64))
    po, pw, pt = insert_queue(p, l, 1700, o_old, w_old)
    assert co.tolist() == po and cw.tolist() == pw and list(ct) == pt
