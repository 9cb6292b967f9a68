"""Cross-checks of the two oracle implementations and the 128-bit pins.

* ``numpy.lexsort((id, length, rank))`` (a stable library sort) followed by
  an exclusive cumulative sum is an independent route to order and wait.
* The C oracle (oracle.c) must agree with the pure-Python oracle on fuzz
  queues, on scaled-down workloads and on batched inputs.
* Totals need more than 64 bits: with one class and every length
  2^31 - 1, wait[k] = k * (2^31 - 1) and the total is
  (2^31 - 1) * n (n - 1) / 2, which passes 2^63 at n = 2^17 and 2^64 at
  n = 2^18.
"""

import numpy as np
import pytest

from oracle import (OracleRangeError, c_oracle_batched, c_oracle_queue,
                    schedule_batched, schedule_queue)
from workloads import fuzz_queue, fuzz_segments, generate


def lexsort_route(p, l):
    n = len(p)
    ids = np.arange(n)
    order = np.lexsort((ids, l.astype(np.int64), p.astype(np.int64)))
    svc = l.astype(np.int64)[order]
    wait = np.zeros(n, np.int64)
    if n > 1:
        np.cumsum(svc[:-1], out=wait[1:])
    return order, wait


@pytest.mark.parametrize("n,seed,tie", [(0, 0, 0.0), (1, 1, 0.0), (17, 2, 0.5),
                                        (1000, 3, 0.3), (5000, 4, 0.0)])
def test_python_oracle_vs_lexsort(n, seed, tie):
    p, l = fuzz_queue(n, seed, classes=6, max_len=40, tie_frac=tie)
    order, wait, totals = schedule_queue(p, l)
    lo, lw = lexsort_route(p, l)
    assert order == lo.tolist()
    assert wait == lw.tolist()
    assert totals[0] == sum(int(x) for x in lw)


@pytest.mark.parametrize("n,seed,tie,max_len", [(0, 0, 0.0, 5), (1, 1, 0.0, 5),
                                                (63, 2, 0.5, 3), (4097, 3, 0.2, 100),
                                                (20000, 4, 0.1, 1 << 30)])
def test_c_oracle_vs_python_oracle(n, seed, tie, max_len):
    p, l = fuzz_queue(n, seed, classes=9, max_len=max_len, tie_frac=tie)
    po, pw, pt = schedule_queue(p, l)
    co, cw, ct = c_oracle_queue(p, l)
    assert co.tolist() == po
    assert cw.tolist() == pw
    assert ct == pt


@pytest.mark.parametrize("name,scale", [("c1", 1.0), ("c2", 1 / 64), ("c3", 1 / 4096)])
def test_c_oracle_vs_python_oracle_workloads(name, scale):
    w = generate(name, scale)
    po, pw, pt = schedule_queue(w.priority, w.length)
    co, cw, ct = c_oracle_queue(w.priority, w.length)
    assert co.tolist() == po and cw.tolist() == pw and ct == pt


@pytest.mark.parametrize("name,scale", [("c4", 1 / 512), ("c5", 1 / 256)])
def test_c_oracle_vs_python_oracle_batched(name, scale):
    w = generate(name, scale)
    po, pw, pt = schedule_batched(w.priority, w.length, w.offsets, w.num_classes)
    co, cw, ct = c_oracle_batched(w.priority, w.length, w.offsets, w.num_classes)
    assert co.tolist() == po and cw.tolist() == pw and ct == pt


def test_c_oracle_batched_empty_segments():
    p, l, off = fuzz_segments([0, 3, 0, 0, 5, 1, 0], seed=9, classes=3)
    po, pw, pt = schedule_batched(p, l, off, 3)
    co, cw, ct = c_oracle_batched(p, l, off, 3)
    assert co.tolist() == po and cw.tolist() == pw and ct == pt


@pytest.mark.parametrize("log_n", [17, 18])
def test_totals_need_128_bits(log_n):
    n = 1 << log_n
    L = (1 << 31) - 1
    p = np.zeros(n, np.uint8)
    l = np.full(n, L, np.int32)
    expect = L * n * (n - 1) // 2
    assert expect > (1 << 63) - 1
    if log_n == 17:
        assert expect == 18446603327631327232
    co, cw, ct = c_oracle_queue(p, l)
    assert ct[0] == ct[1] == expect
    assert cw[-1] == (n - 1) * L
    _, pw, pt = schedule_queue(p, l, 1)
    assert pt[0] == expect and pw[-1] == (n - 1) * L


def test_c_oracle_range_errors():
    with pytest.raises(OracleRangeError):
        c_oracle_queue(np.array([0, 1], np.uint8), np.array([3, -1], np.int32))
    with pytest.raises(OracleRangeError):
        c_oracle_batched(np.array([0, 5], np.uint8), np.array([3, 1], np.int32),
                         np.array([0, 2]), 4)


def test_parallel_batched_equals_serial():
    # the OpenMP baseline spreads whole queues over threads: same results
    from oracle import c_oracle_batched, c_oracle_batched_parallel
    from workloads import fuzz_segments
    sizes = np.random.default_rng(9).integers(0, 900, 400)
    p, l, off = fuzz_segments(sizes, seed=10, classes=6, max_len=2000)
    o1, w1, t1 = c_oracle_batched(p, l, off, 6)
    o2, w2, t2, used = c_oracle_batched_parallel(p, l, off, 6)
    assert used >= 1
    assert np.array_equal(o1, o2) and np.array_equal(w1, w2) and t1 == t2
