"""Pins of the batch-selection and eviction oracle (Algorithms 2-4).

Algorithm 2 has no closed form, so the oracle is pinned by what the
algorithm guarantees, each property chosen to catch a plausible slip:
conservation (every request of H, U and O is in exactly one of the batch, the
pushed-back list or the untouched rest of H), the batch size, key order, the
top-b property of the candidates, the most urgent request always being
scheduled, the stage filter (no prefill candidate rides along behind a
decoding leader), the all-prefill case reducing to "the b smallest keys of C
and O", and a hand-worked priority-inversion example from Section 3.3.

Algorithm 3's order is pinned to numpy.lexsort reversed; Algorithm 4's
heap loop to its closed form: after incoming request j the victims are the
shortest prefix of the eviction order whose KV sizes cover
usage + (demands so far) - capacity.
"""

import random

import numpy as np
import pytest

from oracle.batch_oracle import DECODE, PREFILL, eviction_order, evict, select_batch


def key(p, l, i):
    return (p[i], l[i], i)


def random_instance(rng, n, nh, nu, no, classes=4, max_len=50):
    p = [rng.randrange(classes) for _ in range(n)]
    l = [rng.randrange(max_len) for _ in range(n)]
    stage = [rng.randrange(2) for _ in range(n)]
    ids = list(range(n))
    rng.shuffle(ids)
    H = sorted(ids[:nh], key=lambda i: key(p, l, i))
    U = ids[nh:nh + nu]
    O = ids[nh + nu:nh + nu + no]
    return p, l, stage, H, U, O


@pytest.mark.parametrize("seed", range(300))
def test_select_batch_properties(seed):
    rng = random.Random(seed)
    n = rng.randrange(1, 60)
    nh = rng.randrange(0, n + 1)
    nu = rng.randrange(0, n - nh + 1)
    no = rng.randrange(0, n - nh - nu + 1)
    p, l, stage, H, U, O = random_instance(rng, n, nh, nu, no)
    b = rng.randrange(0, 12)
    batch, pushed = select_batch(p, l, stage, H, U, O, b)
    k = lambda i: key(p, l, i)
    pool = sorted(H + U, key=k)
    C = pool[:b]
    rest = pool[b:]
    # top-b: every request left in H or U is behind every candidate
    if C and rest:
        assert k(C[-1]) < k(rest[0])
    # conservation
    assert sorted(batch + pushed + rest) == sorted(H + U + O)
    assert len(set(batch + pushed)) == len(batch) + len(pushed)
    assert batch == sorted(batch, key=k) and pushed == sorted(pushed, key=k)
    everyone = C + O
    if not everyone:
        assert batch == [] and pushed == []
        return
    top = min(everyone, key=k)
    if b >= 1:
        assert batch[0] == top, "the most urgent request is always scheduled"
    if stage[top] == PREFILL:
        assert batch == sorted(everyone, key=k)[:b]
    else:
        assert all(stage[i] == DECODE for i in batch if i in C)
        assert all(i in pushed for i in C if stage[i] == PREFILL)
        assert batch == sorted([i for i in C if stage[i] == DECODE] + O, key=k)[:b]
    assert len(batch) == min(b, len(everyone) if stage[top] == PREFILL
                             else len([i for i in C if stage[i] == DECODE]) + len(O))


def test_priority_inversion_example():
    # Section 3.3: an urgent request already decoding must not wait behind
    # less urgent prefills. Ids: 0 decoding (rank 0, ongoing); 1, 2 waiting
    # prefills of rank 2; 3 waiting decode of rank 1 (pushed back earlier).
    p = [0, 2, 2, 1]
    l = [10, 5, 7, 3]
    stage = [DECODE, PREFILL, PREFILL, DECODE]
    batch, pushed = select_batch(p, l, stage, heap_order=[3, 1, 2], buffer=[], ongoing=[0], b=3)
    assert batch == [0, 3]
    assert pushed == [1, 2]
    # with the urgent ongoing request in prefill instead, everything merges
    stage[0] = PREFILL
    batch, pushed = select_batch(p, l, stage, heap_order=[3, 1, 2], buffer=[], ongoing=[0], b=3)
    assert batch == [0, 3, 1] and pushed == [2]


def test_buffer_members_are_candidates():
    p = [3, 3, 0]
    l = [1, 2, 9]
    stage = [PREFILL] * 3
    batch, pushed = select_batch(p, l, stage, heap_order=[0, 1], buffer=[2], ongoing=[], b=1)
    assert batch == [2] and pushed == []


def test_eviction_order_is_the_reversed_schedule():
    rng = np.random.default_rng(3)
    n = 500
    p = rng.integers(0, 4, n)
    l = rng.integers(0, 30, n)
    cached = rng.permutation(n)[:300].tolist()
    want = np.lexsort((np.array(cached), l[cached], p[cached]))[::-1]
    assert eviction_order(p.tolist(), l.tolist(), cached) == [cached[j] for j in want]


@pytest.mark.parametrize("seed", range(200))
def test_evict_matches_prefix_closed_form(seed):
    rng = random.Random(seed)
    n = rng.randrange(0, 40)
    p = [rng.randrange(3) for _ in range(n)]
    l = [rng.randrange(20) for _ in range(n)]
    cached = list(range(n))
    rng.shuffle(cached)
    kv = [rng.randrange(0, 10) for _ in cached]
    usage = sum(kv) + rng.randrange(0, 5)
    capacity = rng.randrange(0, usage + 30)
    demands = [rng.randrange(0, 15) for _ in range(rng.randrange(0, 6))]
    victims, upto = evict(p, l, cached, kv, usage, capacity, demands)
    order = eviction_order(p, l, cached)
    size = dict(zip(cached, kv))
    E = np.concatenate([[0], np.cumsum([size[i] for i in order])])
    S = np.cumsum(demands) if demands else []
    want_upto = []
    for j in range(len(demands)):
        need = usage + int(S[j]) - capacity
        k = 0 if need <= 0 else int(np.searchsorted(E, need, side="left"))
        want_upto.append(min(k, len(order)))
    assert upto == want_upto
    assert victims == order[:want_upto[-1] if want_upto else 0]


def test_evict_extremes():
    p, l = [0, 1, 2], [5, 5, 5]
    assert evict(p, l, [0, 1, 2], [4, 4, 4], 12, 100, [10]) == ([], [0])
    assert evict(p, l, [0, 1, 2], [4, 4, 4], 12, 0, [1]) == ([2, 1, 0], [3])
    assert evict(p, l, [0, 1, 2], [4, 4, 4], 12, 12, [4, 4]) == ([2, 1], [1, 2])
