"""CPU oracle of batch selection and eviction (Section 3.3, Algorithms 2-4).

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it. It shares no code with the HIP
library.

Every request has a key (rank p, predicted remaining time l, id); the most
urgent request is the one with the smallest key (the min-heap of
Algorithm 1). A request is in the prefill stage (0) or the decoding stage (1).

``select_batch`` follows Algorithm 2 (Scheduling with Stage Awareness):

1. C = the b smallest keys among the waiting requests: the heap H (given as
   its drained order) and the not yet inserted buffer U (ExtractTopb looks
   at both, so that no urgent arrival is overlooked);
2. p* = the smallest key in C and the ongoing requests O;
3. if p* is in the prefill stage, M = C and O merged by key; else M = the
   decoding members of C and O merged, and C's prefill members go back to H;
4. the next batch is M's first b; the rest of M goes back to H.

Readings: "Priority" ranks by the scheduling key (smaller key = higher
priority); requests pushed back are returned as one list sorted by key
(PushBack only reinserts them, so their order carries no meaning, and a
sorted list makes the result unique); H's members outside C stay where
they are and are not returned.

``evict`` follows Algorithms 3 and 4 (MaxHeap Construction, Priority-Based
Eviction): the cached requests R form a max-heap keyed by the inverse of the
scheduling key (least urgent rank first, then longest remaining time; the
exact reverse of the schedule order, so among equal (p, l) the later
arrival goes first). For each incoming request j (in the given order) with
KV demand s_j: while s_j + c > capacity and R is not empty, pop the root,
evict it (c -= its KV size); then c += s_j. Reading for a batch: the
incoming requests join the cache after their own eviction step but are not
victims of later incoming requests in the same call (they are running).
The result is the victims in eviction order and, per incoming request, the
number of victims evicted up to and including its step.

Pins (tests/test_oracle_batch.py): Algorithm 2 written a second time with
plain list filtering and sorting against this heapq version, invariants of
the batch, Algorithm 4 against the prefix-sum closed form, and special cases.
"""

from __future__ import annotations

import heapq
from typing import List, Sequence, Tuple

PREFILL = 0
DECODE = 1


def _key(p, l, i):
    return (int(p[i]), int(l[i]), int(i))


def select_batch(p: Sequence[int], l: Sequence[int], stage: Sequence[int],
                 heap_order: Sequence[int], buffer: Sequence[int],
                 ongoing: Sequence[int], b: int) -> Tuple[List[int], List[int]]:
    """Algorithm 2. Returns (next batch in key order, pushed-back requests
    in key order). Ids index ``p``, ``l`` and ``stage``."""
    if b < 0:
        raise ValueError("b must be >= 0")
    key = lambda i: _key(p, l, i)
    # ExtractTopb over the heap (drained in order) and the unsorted buffer:
    # a min-heap fed with both, popped b times
    h = [(key(i), i) for i in list(heap_order) + list(buffer)]
    heapq.heapify(h)
    cand = [heapq.heappop(h)[1] for _ in range(min(b, len(h)))]
    pool = cand + list(ongoing)
    if not pool:
        return [], []
    top = min(pool, key=key)
    pushed = []
    if int(stage[top]) == PREFILL:
        merged = sorted(cand + list(ongoing), key=key)
    else:
        dec = [i for i in cand if int(stage[i]) == DECODE]
        pushed += [i for i in cand if int(stage[i]) != DECODE]
        merged = sorted(dec + list(ongoing), key=key)
    batch = merged[:b]
    pushed += merged[b:]
    return batch, sorted(pushed, key=key)


def eviction_order(p: Sequence[int], l: Sequence[int], cached: Sequence[int]) -> List[int]:
    """Algorithm 3: the cached requests drained from a max-heap keyed by the
    inverse of the scheduling key."""
    h = [tuple(-x for x in _key(p, l, i)) + (i,) for i in cached]
    heapq.heapify(h)
    return [heapq.heappop(h)[-1] for _ in range(len(h))]


def evict(p: Sequence[int], l: Sequence[int], cached: Sequence[int],
          kv: Sequence[int], usage: int, capacity: int,
          demands: Sequence[int]) -> Tuple[List[int], List[int]]:
    """Algorithm 4 for incoming requests with KV demands ``demands``;
    ``kv[j]`` is the KV size of ``cached[j]``. Returns (victims in eviction
    order, victims evicted up to each incoming request)."""
    size = {int(i): int(kv[j]) for j, i in enumerate(cached)}
    h = [tuple(-x for x in _key(p, l, i)) + (int(i),) for i in cached]
    heapq.heapify(h)
    c = int(usage)
    victims: List[int] = []
    upto: List[int] = []
    for s in demands:
        s = int(s)
        if s < 0:
            raise ValueError("negative demand")
        while s + c > capacity and h:
            v = heapq.heappop(h)[-1]
            victims.append(v)
            c -= size[v]
        c += s
        upto.append(len(victims))
    return victims, upto
