"""Pins of the comparison policies (FCFS, SJF, HPJF) of the oracle.

The experiments of Section 4 (request spikes) compare semantic scheduling
with first-come-first-served, shortest job first and highest-priority job
first. ``schedule_policy`` orders a queue by each of them; these tests fix
that order and the waits by routes that share nothing with it:

* FCFS is the arrival order itself: the waits are numpy's cumulative sum
  of the lengths in id order.
* SJF minimises the total wait over every permutation (the textbook
  shortest-processing-time rule, checked by exhaustion for n <= 7), and
  among the minimisers the oracle returns the one whose ties are in id
  order; at any size it is ``numpy.lexsort((id, length))``.
* HPJF is a stable sort by rank: ``numpy.argsort(rank, kind="stable")``.
* Relations between the policies: SJF's total is never above the semantic
  total (the semantic order is one of the permutations SJF minimises over),
  and under the rank constraint of Eq. 2 every class total of the semantic
  schedule is at most the HPJF class total (both serve the classes in the
  same contiguous blocks; inside a class the semantic order is SJF).
* Totals are split by each request's own rank under every policy: the class
  totals add up to the total and each one is the sum of its members' waits.
"""

import itertools
import random

import numpy as np
import pytest

from oracle import (POLICIES, POLICY_FCFS, POLICY_HPJF, POLICY_SEMANTIC, POLICY_SJF,
                    OracleRangeError, c_oracle_policy, schedule_policy, schedule_queue)
from workloads import fuzz_queue, generate


def excl_cumsum(values):
    out = np.zeros(len(values), np.int64)
    if len(values) > 1:
        np.cumsum(np.asarray(values, np.int64)[:-1], out=out[1:])
    return out


def class_totals(p, order, wait, num_classes=256):
    tot = [0] * (1 + num_classes)
    for k, i in enumerate(order):
        tot[0] += int(wait[k])
        tot[1 + int(p[i])] += int(wait[k])
    return tot


def test_fcfs_is_arrival_order():
    p, l = fuzz_queue(500, seed=11, classes=6, max_len=300)
    order, wait, totals = schedule_policy(p, l, POLICY_FCFS)
    assert order == list(range(500))
    assert wait == excl_cumsum(l).tolist()
    assert totals == class_totals(p, order, wait)


@pytest.mark.parametrize("seed", range(25))
def test_sjf_minimises_total_wait_by_exhaustion(seed):
    rng = random.Random(seed)
    n = rng.randint(1, 7)
    p = [rng.randrange(4) for _ in range(n)]
    l = [rng.randrange(5) for _ in range(n)]  # small range: many ties
    order, wait, totals = schedule_policy(p, l, POLICY_SJF)
    best, argmins = None, []
    for perm in itertools.permutations(range(n)):
        t, tot = 0, 0
        for i in perm:
            tot += t
            t += l[i]
        if best is None or tot < best:
            best, argmins = tot, [perm]
        elif tot == best:
            argmins.append(perm)
    assert totals[0] == best
    assert tuple(order) in argmins
    # the id-ordered member of the argmin set
    assert tuple(order) == min(argmins, key=lambda perm: [l[i] for i in perm] + list(perm))


def test_sjf_and_hpjf_match_stable_library_sorts():
    p, l = fuzz_queue(3000, seed=5, classes=7, max_len=100)
    ids = np.arange(len(p))
    o, w, _ = schedule_policy(p, l, POLICY_SJF)
    want = np.lexsort((ids, l.astype(np.int64)))
    assert o == want.tolist()
    assert w == excl_cumsum(l[want]).tolist()
    o, w, _ = schedule_policy(p, l, POLICY_HPJF)
    want = np.argsort(p, kind="stable")
    assert o == want.tolist()
    assert w == excl_cumsum(l[want]).tolist()


@pytest.mark.parametrize("seed", range(10))
def test_relations_between_policies(seed):
    p, l = fuzz_queue(400, seed=seed, classes=5, max_len=1000)
    sem = schedule_policy(p, l, POLICY_SEMANTIC)[2]
    assert sem == schedule_queue(p, l)[2]
    sjf = schedule_policy(p, l, POLICY_SJF)[2]
    hp = schedule_policy(p, l, POLICY_HPJF)[2]
    fc = schedule_policy(p, l, POLICY_FCFS)[2]
    assert sjf[0] <= sem[0] <= hp[0]
    for c in range(256):
        assert sem[1 + c] <= hp[1 + c]
    for t in (sem, sjf, hp, fc):
        assert sum(t[1:]) == t[0]


def test_policies_reduce_to_each_other():
    # one class: the semantic order is SJF; constant length: it is HPJF;
    # one class and constant length: every policy is FCFS
    rng = np.random.default_rng(3)
    l = rng.integers(0, 50, 700).astype(np.int32)
    p1 = np.zeros(700, np.uint8)
    assert schedule_policy(p1, l, POLICY_SEMANTIC) == schedule_policy(p1, l, POLICY_SJF)
    p = rng.integers(0, 4, 700).astype(np.uint8)
    lc = np.full(700, 9, np.int32)
    assert schedule_policy(p, lc, POLICY_SEMANTIC) == schedule_policy(p, lc, POLICY_HPJF)
    for pol in POLICIES:
        assert schedule_policy(p1, lc, pol) == schedule_policy(p1, lc, POLICY_FCFS)


@pytest.mark.parametrize("policy", POLICIES)
def test_c_oracle_matches_python(policy):
    for seed in range(4):
        p, l = fuzz_queue(2000 + 37 * seed, seed=seed, classes=9, max_len=4000)
        a = c_oracle_policy(p, l, policy)
        b = schedule_policy(p, l, policy)
        assert a[0].tolist() == b[0] and a[1].tolist() == b[1] and a[2] == b[2]
    w = generate("c2", scale=1 / 64)
    a = c_oracle_policy(w.priority, w.length, policy)
    b = schedule_policy(w.priority, w.length, policy)
    assert a[0].tolist() == b[0] and a[1].tolist() == b[1] and a[2] == b[2]


@pytest.mark.parametrize("policy", POLICIES)
def test_range_errors_and_empty(policy):
    with pytest.raises(OracleRangeError):
        schedule_policy([0, 1], [3, -1], policy)
    with pytest.raises(OracleRangeError):
        c_oracle_policy(np.array([0, 1], np.uint8), np.array([3, -1], np.int32), policy)
    assert schedule_policy([], [], policy) == ([], [], [0] * 257)
    o, w, t = c_oracle_policy(np.zeros(0, np.uint8), np.zeros(0, np.int32), policy)
    assert len(o) == 0 and t == [0] * 257


def test_unknown_policy():
    with pytest.raises(ValueError):
        schedule_policy([0], [1], 7)
    with pytest.raises(ValueError):
        c_oracle_policy(np.zeros(1, np.uint8), np.ones(1, np.int32), 7)
