"""GPU parity of sem_insert (arrivals merged into an earlier schedule).

The earlier schedule handed to the GPU is the oracle's (no input comes from
the HIP path); the expected result is the oracle's insert_queue, i.e. the
schedule of all requests. Everything is integer: bit-exact comparisons.
"""

import numpy as np
import pytest

from oracle import c_oracle_insert, c_oracle_queue
from tests._lib import assert_same, ensure_built, gpu_available
from workloads import fuzz_queue

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]


@pytest.fixture(scope="module", autouse=True)
def _built():
    ensure_built()


def gpu_insert(p, l, n_old, o_old, w_old):
    import torch

    import paper_2506_12204_amd as ss
    dev = torch.device("cuda")
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a, dtype=dt)).to(dev)
    order, wait, totals = ss.insert(t(p, np.uint8), t(l, np.int32), n_old,
                                    t(o_old, np.int32), t(w_old, np.int64))
    return order.cpu().numpy(), wait.cpu().numpy(), totals


def check(p, l, n_old, label):
    print(f"[gpu] insert {label}: n_old={n_old} m={len(p) - n_old}", flush=True)
    o_old, w_old, _ = c_oracle_queue(p[:n_old], l[:n_old])
    want = c_oracle_insert(p, l, n_old, o_old, w_old)
    assert_same(gpu_insert(p, l, n_old, o_old, w_old), want, label)


@pytest.mark.parametrize("n_old,m", [(0, 0), (0, 5), (5, 0), (1, 1), (100, 7), (1000, 1000),
                                     (16384, 1), (20000, 300), (100003, 70000),
                                     (300000, 20000), (5000, 40000)])
def test_insert_sizes(n_old, m):
    p, l = fuzz_queue(n_old + m, seed=n_old * 7 + m, classes=6, max_len=3000, tie_frac=0.3)
    check(p, l, n_old, f"{n_old}+{m}")


def test_arrivals_all_more_urgent_or_all_less():
    rng = np.random.default_rng(41)
    n_old, m = 50000, 3000
    l = rng.integers(1, 1000, n_old + m).astype(np.int32)
    p = np.concatenate([rng.integers(1, 4, n_old), np.zeros(m, np.int64)]).astype(np.uint8)
    check(p, l, n_old, "arrivals-first")
    p = np.concatenate([rng.integers(0, 3, n_old), np.full(m, 3)]).astype(np.uint8)
    check(p, l, n_old, "arrivals-last")


def test_arrivals_tie_every_earlier_key():
    rng = np.random.default_rng(42)
    n_old = 30000
    p_old = rng.integers(0, 4, n_old).astype(np.uint8)
    l_old = rng.integers(0, 50, n_old).astype(np.int32)
    pick = rng.integers(0, n_old, 10000)
    p = np.concatenate([p_old, p_old[pick]])
    l = np.concatenate([l_old, l_old[pick]])
    check(p, l, n_old, "ties")


def test_chained_inserts_equal_one_schedule():
    p, l = fuzz_queue(200000, seed=43, classes=5, max_len=32768, tie_frac=0.2)
    cuts = [0, 60000, 60001, 150000, 200000]
    o, w = np.zeros(0, np.int32), np.zeros(0, np.int64)
    for a, b in zip(cuts, cuts[1:]):
        print(f"[gpu] chained insert {a}->{b}", flush=True)
        o, w, t = gpu_insert(p[:b], l[:b], a, o, w)
    assert_same((o, w, t), c_oracle_queue(p, l), "chained")


def test_large_queue_small_arrival_batch():
    rng = np.random.default_rng(44)
    n_old, m = 1 << 22, 1 << 16
    p = rng.integers(0, 5, n_old + m).astype(np.uint8)
    l = rng.integers(1, 32769, n_old + m).astype(np.int32)
    check(p, l, n_old, "4M+64K")


def test_arrival_range_error():
    import paper_2506_12204_amd as ss
    p, l = fuzz_queue(5000, seed=45)
    l[4500] = -1
    o_old, w_old, _ = c_oracle_queue(p[:4000], l[:4000])
    with pytest.raises(ss.SemschedRangeError):
        gpu_insert(p, l, 4000, o_old, w_old)
