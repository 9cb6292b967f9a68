"""The definition check used for the largest GPU queue (tests/_lib.py,
check_queue_by_definition) accepts the oracle's schedules and rejects each
kind of plausible mistake: two requests out of key order, a tie broken the
wrong way, a repeated id, a wait off by one, a wrong grand or class total."""

import numpy as np
import pytest

from oracle import c_oracle_queue
from tests._lib import check_queue_by_definition
from workloads import fuzz_queue


def schedule(seed, n=3000):
    p, l = fuzz_queue(n, seed=seed, classes=5, max_len=200, tie_frac=0.3)
    order, wait, totals = c_oracle_queue(p, l)
    return p, l, order.copy(), wait.copy(), list(totals)


@pytest.mark.parametrize("seed", range(5))
def test_accepts_the_oracle(seed):
    check_queue_by_definition(*schedule(seed))


def test_accepts_empty_and_single():
    for n in (0, 1):
        p = np.zeros(n, np.uint8)
        l = np.full(n, 7, np.int32)
        order, wait, totals = c_oracle_queue(p, l)
        check_queue_by_definition(p, l, order, wait, list(totals))


def rejects(p, l, order, wait, totals):
    with pytest.raises(AssertionError):
        check_queue_by_definition(p, l, order, wait, totals)


def test_rejects_a_key_inversion():
    p, l, order, wait, totals = schedule(1)
    k = next(i for i in range(len(order) - 1)
             if (p[order[i]], l[order[i]]) != (p[order[i + 1]], l[order[i + 1]]))
    order[k], order[k + 1] = order[k + 1], order[k]
    rejects(p, l, order, wait, totals)


def test_rejects_a_tie_broken_by_the_larger_id():
    p, l, order, wait, totals = schedule(2)
    k = next(i for i in range(len(order) - 1)
             if (p[order[i]], l[order[i]]) == (p[order[i + 1]], l[order[i + 1]]))
    order[k], order[k + 1] = order[k + 1], order[k]
    rejects(p, l, order, wait, totals)


def test_rejects_a_repeated_id():
    p, l, order, wait, totals = schedule(3)
    order[5] = order[4]
    rejects(p, l, order, wait, totals)


def test_rejects_a_wait_off_by_one():
    p, l, order, wait, totals = schedule(4)
    wait[100] += 1
    rejects(p, l, order, wait, totals)


@pytest.mark.parametrize("slot", [0, 1, 3])
def test_rejects_a_wrong_total(slot):
    p, l, order, wait, totals = schedule(5)
    totals[slot] += 1
    rejects(p, l, order, wait, totals)
