"""CPU oracle for the semantic-scheduling hot path (pure Python).

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or
link this module: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it. It shares no code with the HIP
library.

What it computes, for one queue of requests i = 0..n-1 with urgency rank
``p[i]`` (Definition 1, graded poset: rank 0 is the most urgent ESI level)
and predicted service time ``l[i]`` (the estimated remaining computation
time f_t of Section 3.3, here the predicted generation length in tokens):

1. ``order``: request ids sorted ascending by ``(p[i], l[i], i)``. This is the
   sequence obtained by draining the min-heap keyed by the priority tuple
   (f_e, f_t) of Algorithm 1 (MinHeap Construction) and the paragraph on
   scheduling the highest-priority requests. With all arrivals equal, the
   relative constraint (Eq. 2) forces the order to be non-decreasing in rank,
   and within one rank the average waiting time (Eq. 1) is minimised by
   shortest-predicted-length first. Exact (rank, length) ties are broken by
   arrival id, a reading the paper leaves open (it gives no tie rule).
2. ``wait``: the time each request waits before its service starts, in
   schedule order: ``wait[0] = 0``, ``wait[k] = wait[k-1] + l[order[k-1]]``.
   Eq. 1 uses finish minus arrival, which adds each request's own service
   time; that constant does not change the minimiser, and the exclusive form
   is what is returned (completion time = wait + length).
3. ``totals``: ``[sum(wait), sum over class 0, ..., class C-1]``, exact
   integers (they exceed 2^64 at n = 2^26).

Inputs are rejected (``OracleRangeError``) when a length is negative or a
rank is not below the number of classes.

Pins (see tests/test_oracle_*): brute force over every rank-respecting
permutation for n <= 8, the adjacent-exchange invariant, closed forms,
special cases that reduce to textbook policies, ``numpy.lexsort``, a
hand-worked example and a 128-bit width case.

``schedule_policy`` orders the same queue by the comparison policies of the
paper's experiments (Section 4, request spikes: first-come-first-served,
shortest job first, highest-priority job first) as well as by the semantic
tuple; waits and per-class totals are defined as above for every policy.

``insert_queue`` is the incremental form (Section 3.3, asynchronous queue
management; Algorithm 1's HeapInsert): new arrivals are inserted into the
heap that already holds the earlier requests, and draining it gives the
schedule of all of them. It is pinned to a literal binary min-heap
(``heapq``) that receives the arrivals one by one (tests/test_oracle_insert).
"""

from __future__ import annotations

from typing import List, Sequence, Tuple

MAX_CLASSES = 256


class OracleRangeError(ValueError):
    """A length is negative or a rank is >= the number of classes."""


def _check(p: Sequence[int], l: Sequence[int], num_classes: int) -> None:
    if len(p) != len(l):
        raise ValueError("priority and length differ in size")
    if not 1 <= num_classes <= MAX_CLASSES:
        raise ValueError("num_classes must be in [1, 256]")
    for i in range(len(p)):
        if l[i] < 0:
            raise OracleRangeError(f"length[{i}] = {l[i]} < 0")
        if not 0 <= p[i] < num_classes:
            raise OracleRangeError(f"priority[{i}] = {p[i]} >= {num_classes}")


def schedule_queue(p: Sequence[int], l: Sequence[int],
                   num_classes: int = MAX_CLASSES
                   ) -> Tuple[List[int], List[int], List[int]]:
    """Schedule one queue; returns (order, wait, totals) as Python lists.

    ``totals`` has ``1 + num_classes`` entries: the grand total first, then
    one entry per class (zero for an empty class).
    """
    p = [int(x) for x in p]
    l = [int(x) for x in l]
    _check(p, l, num_classes)
    n = len(p)
    # Step 1: the drained min-heap = ids ascending by the priority tuple.
    order = sorted(range(n), key=lambda i: (p[i], l[i], i))
    # Step 2: each request waits for the service of everything ahead of it.
    wait = [0] * n
    for k in range(1, n):
        wait[k] = wait[k - 1] + l[order[k - 1]]
    # Step 3: Eq. 1's numerator, overall and per urgency class.
    totals = [0] * (1 + num_classes)
    for k in range(n):
        totals[0] += wait[k]
        totals[1 + p[order[k]]] += wait[k]
    return order, wait, totals


POLICY_SEMANTIC = 0  # (rank, length, id): the priority tuple of Algorithm 1
POLICY_FCFS = 1      # (id): arrival order
POLICY_SJF = 2       # (length, id): shortest predicted job first, rank ignored
POLICY_HPJF = 3      # (rank, id): most urgent first, length ignored
POLICIES = (POLICY_SEMANTIC, POLICY_FCFS, POLICY_SJF, POLICY_HPJF)


def policy_key(policy: int, p: Sequence[int], l: Sequence[int]):
    """Sort key of request i under ``policy``; the id closes every key, so
    the order is total (ties go to the earlier arrival)."""
    if policy == POLICY_SEMANTIC:
        return lambda i: (p[i], l[i], i)
    if policy == POLICY_FCFS:
        return lambda i: (i,)
    if policy == POLICY_SJF:
        return lambda i: (l[i], i)
    if policy == POLICY_HPJF:
        return lambda i: (p[i], i)
    raise ValueError(f"unknown policy {policy}")


def schedule_policy(p: Sequence[int], l: Sequence[int], policy: int,
                    num_classes: int = MAX_CLASSES
                    ) -> Tuple[List[int], List[int], List[int]]:
    """Schedule one queue under ``policy``; returns (order, wait, totals).

    The comparison policies of Section 4: FCFS serves in arrival order, SJF
    by predicted length alone, HPJF by urgency rank alone (each with the
    arrival id as the last key). Waits are the exclusive prefix of the
    lengths in the chosen order and ``totals[1 + c]`` adds the waits of the
    requests whose rank is c, whatever the policy.
    """
    p = [int(x) for x in p]
    l = [int(x) for x in l]
    _check(p, l, num_classes)
    n = len(p)
    order = sorted(range(n), key=policy_key(policy, p, l))
    wait = [0] * n
    for k in range(1, n):
        wait[k] = wait[k - 1] + l[order[k - 1]]
    totals = [0] * (1 + num_classes)
    for k in range(n):
        totals[0] += wait[k]
        totals[1 + p[order[k]]] += wait[k]
    return order, wait, totals


def insert_queue(p: Sequence[int], l: Sequence[int], n_old: int,
                 order_old: Sequence[int], wait_old: Sequence[int],
                 num_classes: int = MAX_CLASSES
                 ) -> Tuple[List[int], List[int], List[int]]:
    """Insert requests ``n_old .. len(p)-1`` into the schedule of the first
    ``n_old`` requests; returns the schedule (order, wait, totals) of all.

    ``order_old`` / ``wait_old`` must be the schedule of requests
    ``0 .. n_old-1`` (checked: ValueError otherwise). The arrivals carry the
    next arrival indices as ids, so an exact (rank, length) tie between an
    earlier request and a new one goes to the earlier request. Inserting them
    into the heap and draining it yields the ids ascending by the priority
    tuple over all requests: the plain definition of ``schedule_queue``.
    """
    p = [int(x) for x in p]
    l = [int(x) for x in l]
    if not 0 <= n_old <= len(p):
        raise ValueError("n_old must be in [0, n]")
    want_o, want_w, _ = schedule_queue(p[:n_old], l[:n_old], num_classes)
    if [int(x) for x in order_old] != want_o or [int(x) for x in wait_old] != want_w:
        raise ValueError("order_old / wait_old are not the schedule of the first n_old requests")
    return schedule_queue(p, l, num_classes)


def schedule_batched(p: Sequence[int], l: Sequence[int],
                     offsets: Sequence[int], num_classes: int
                     ) -> Tuple[List[int], List[int], List[int]]:
    """Schedule S independent queues laid out back to back.

    Queue s holds requests ``offsets[s] .. offsets[s+1]-1``; its ids are local
    arrival indices (0-based inside the queue). Outputs are concatenated in
    the same layout; ``totals`` is ``S * (1 + num_classes)`` long, queue-major.
    """
    offsets = [int(x) for x in offsets]
    if len(offsets) < 1 or offsets[0] != 0 or offsets[-1] != len(p):
        raise ValueError("offsets must start at 0 and end at n")
    for s in range(len(offsets) - 1):
        if offsets[s + 1] < offsets[s]:
            raise ValueError("offsets must be non-decreasing")
    order: List[int] = []
    wait: List[int] = []
    totals: List[int] = []
    for s in range(len(offsets) - 1):
        a, b = offsets[s], offsets[s + 1]
        o, w, t = schedule_queue(p[a:b], l[a:b], num_classes)
        order += o
        wait += w
        totals += t
    return order, wait, totals
