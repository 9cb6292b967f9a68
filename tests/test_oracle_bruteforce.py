"""Pin the oracle to the optimisation problem itself (Eq. 1 under Eq. 2).

For tiny queues every permutation of the requests is enumerated. Each one is
run through a one-server simulation that assigns finishing times; the
permutations that satisfy the relative constraint of Eq. 2 (with all
arrivals at time 0) are kept, and the average-waiting-time objective of
Eq. 1 is evaluated on them. None of this uses the oracle's code: it is the
problem statement, solved by exhaustion.

Checked against the oracle:
* its total wait equals the exhaustive minimum (Eq. 1 counts finish minus
  arrival, which is the oracle's exclusive wait plus each request's own
  length, a constant);
* each class total is individually minimal as well;
* the set of minimisers is exactly the set of orders sorted by
  (rank, length), and the oracle returns the one whose ties are in
  ascending id order.
"""

import itertools
import random

import pytest

from oracle import schedule_queue


def simulate(perm, length):
    """One server, arrivals at 0: finishing time of each request."""
    t = 0
    finish = {}
    for i in perm:
        t += length[i]
        finish[i] = t
    return finish


def satisfies_eq2(perm, rank, finish):
    """Eq. 2 with a_i = 0: f_i < f_j implies f_i < a_j or r(p_i) <= r(p_j)."""
    for i in perm:
        for j in perm:
            if finish[i] < finish[j] and not (finish[i] < 0 or rank[i] <= rank[j]):
                return False
    return True


def exhaustive(rank, length, num_classes):
    n = len(rank)
    best = None
    best_class = [None] * num_classes
    argmins = []
    for perm in itertools.permutations(range(n)):
        finish = simulate(perm, length)
        if not satisfies_eq2(perm, rank, finish):
            continue
        obj = sum(finish[i] - 0 for i in perm)  # Eq. 1 numerator
        if best is None or obj < best:
            best, argmins = obj, [perm]
        elif obj == best:
            argmins.append(perm)
        for c in range(num_classes):
            oc = sum(finish[i] for i in perm if rank[i] == c)
            if best_class[c] is None or oc < best_class[c]:
                best_class[c] = oc
    return best, best_class, argmins


def sorted_by_key_orders(rank, length):
    """All orders non-decreasing in (rank, length): permute within equal keys."""
    groups = {}
    for i in range(len(rank)):
        groups.setdefault((rank[i], length[i]), []).append(i)
    keys = sorted(groups)
    out = [()]
    for k in keys:
        out = [o + p for o in out for p in itertools.permutations(groups[k])]
    return set(out)


CASES = []
_rng = random.Random(20250612)
for n in range(0, 8):
    for trial in range(6 if n < 7 else 3):
        classes = _rng.randint(1, 3)
        max_len = _rng.choice([2, 3, 9])  # small ranges force exact ties
        CASES.append((n, classes,
                      [_rng.randrange(classes) for _ in range(n)],
                      [_rng.randint(1, max_len) for _ in range(n)]))
# one n = 8 case (8! = 40,320 permutations)
CASES.append((8, 3, [2, 0, 1, 0, 2, 1, 0, 1], [5, 9, 3, 9, 1, 7, 2, 3]))


@pytest.mark.parametrize("n,classes,rank,length", CASES)
def test_oracle_is_the_constrained_optimum(n, classes, rank, length):
    order, wait, totals = schedule_queue(rank, length, classes)
    best, best_class, argmins = exhaustive(rank, length, classes)
    sum_len = sum(length)
    if n == 0:
        assert order == [] and wait == [] and totals == [0] * (1 + classes)
        return
    # Eq. 1 objective (finish - arrival) = exclusive wait + own length.
    assert totals[0] + sum_len == best
    for c in range(classes):
        own = sum(length[i] for i in range(n) if rank[i] == c)
        assert totals[1 + c] + own == best_class[c]
    # The minimisers are exactly the (rank, length)-sorted orders ...
    assert set(argmins) == sorted_by_key_orders(rank, length)
    # ... and the oracle picks the one with ascending ids inside each tie.
    assert tuple(order) in set(argmins)
    for k in range(n - 1):
        a, b = order[k], order[k + 1]
        if (rank[a], length[a]) == (rank[b], length[b]):
            assert a < b
