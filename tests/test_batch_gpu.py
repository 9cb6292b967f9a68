"""GPU parity of stage-aware batch selection (sem_select_batch, Algorithm 2)
and priority-based eviction (sem_evict, Algorithms 3-4) against the oracle's
heap simulations (oracle/batch_oracle.py, pinned in
tests/test_oracle_batch.py). Ids and counts: exact comparisons.
"""

import numpy as np
import pytest

from oracle import evict, select_batch
from tests._lib import ensure_built, gpu_available

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]


@pytest.fixture(scope="module", autouse=True)
def _built():
    ensure_built()


def dev(a, dt):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=dt)).cuda()


def instance(seed, n_ids, nh, nu, no, classes=5, max_len=4000, decode_frac=0.5):
    rng = np.random.default_rng(seed)
    p = rng.integers(0, classes, n_ids).astype(np.uint8)
    l = rng.integers(0, max_len, n_ids).astype(np.int32)
    stage = (rng.random(n_ids) < decode_frac).astype(np.uint8)
    ids = rng.permutation(n_ids)
    waiting = ids[:nh]
    heap = waiting[np.lexsort((waiting, l[waiting], p[waiting]))]
    buf = ids[nh:nh + nu]
    ong = ids[nh + nu:nh + nu + no]
    return p, l, stage, heap, buf, ong


def run_select(p, l, stage, heap, buf, ong, b):
    import paper_2506_12204_amd as ss
    bt, pu = ss.select_batch(dev(p, np.uint8), dev(l, np.int32), dev(stage, np.uint8),
                             dev(heap, np.int32), dev(buf, np.int32), dev(ong, np.int32), b)
    return bt.cpu().numpy().tolist(), pu.cpu().numpy().tolist()


@pytest.mark.parametrize("case", [
    (1, 0, 0, 0, 1), (10, 5, 2, 3, 4), (1000, 500, 100, 50, 64), (1 << 20, 200000, 3000, 256, 256),
    (1 << 20, 100000, 4096, 4096, 4096), (50000, 3, 4096, 10, 4096), (50000, 20000, 0, 4096, 1),
    (50000, 20000, 0, 0, 0), (50000, 0, 0, 300, 128), (9000, 4000, 4096, 0, 4096)])
@pytest.mark.parametrize("decode_frac", [0.0, 0.5, 1.0])
def test_select_batch(case, decode_frac):
    n_ids, nh, nu, no, b = case
    print(f"[gpu] select n_ids={n_ids} heap={nh} buffer={nu} ongoing={no} b={b}", flush=True)
    p, l, stage, heap, buf, ong = instance(sum(case) + int(10 * decode_frac), n_ids, nh, nu, no,
                                           decode_frac=decode_frac)
    want = select_batch(p.tolist(), l.tolist(), stage.tolist(), heap.tolist(), buf.tolist(),
                        ong.tolist(), b)
    assert run_select(p, l, stage, heap, buf, ong, b) == want


# Beyond one workgroup's LDS (b, buffer or ongoing above 4096): the lists are
# sorted in 8192-entry chunks and merged in the workspace.
@pytest.mark.parametrize("case", [
    (1 << 20, 40000, 10000, 5000, 16384), (200000, 16384, 0, 16384, 16384),
    (100000, 5000, 5000, 0, 4097), (100000, 0, 4097, 0, 100), (100000, 100, 0, 4097, 50),
    (300000, 70000, 20000, 30000, 60000), (50000, 20000, 0, 0, 8193)])
@pytest.mark.parametrize("decode_frac", [0.0, 0.5, 1.0])
def test_select_batch_beyond_lds(case, decode_frac):
    n_ids, nh, nu, no, b = case
    print(f"[gpu] select (merged in the workspace) n_ids={n_ids} heap={nh} buffer={nu} "
          f"ongoing={no} b={b}", flush=True)
    p, l, stage, heap, buf, ong = instance(sum(case) + int(10 * decode_frac), n_ids, nh, nu, no,
                                           decode_frac=decode_frac)
    want = select_batch(p.tolist(), l.tolist(), stage.tolist(), heap.tolist(), buf.tolist(),
                        ong.tolist(), b)
    assert run_select(p, l, stage, heap, buf, ong, b) == want


def test_select_batch_beyond_lds_ties():
    # few distinct keys across 40000 candidates: the merge rounds must keep
    # equal (rank, length) pairs in id order across chunks
    n = 200000
    rng = np.random.default_rng(8)
    p = rng.integers(0, 2, n).astype(np.uint8)
    l = rng.integers(0, 3, n).astype(np.int32)
    stage = (rng.random(n) < 0.5).astype(np.uint8)
    ids = rng.permutation(n)
    w = ids[:30000]
    heap = w[np.lexsort((w, l[w], p[w]))]
    buf, ong = ids[30000:40000], ids[40000:50000]
    print("[gpu] select (merged in the workspace), ties", flush=True)
    want = select_batch(p.tolist(), l.tolist(), stage.tolist(), heap.tolist(), buf.tolist(),
                        ong.tolist(), 12000)
    assert run_select(p, l, stage, heap, buf, ong, 12000) == want


def test_select_batch_ties_and_inversion():
    # many equal keys (ties go to the lower id) and an urgent decoding request
    n = 20000
    rng = np.random.default_rng(5)
    p = rng.integers(0, 2, n).astype(np.uint8)
    l = rng.integers(0, 3, n).astype(np.int32)
    stage = (rng.random(n) < 0.5).astype(np.uint8)
    ids = rng.permutation(n)
    heap = ids[:9000][np.lexsort((ids[:9000], l[ids[:9000]], p[ids[:9000]]))]
    buf, ong = ids[9000:12000], ids[12000:12100]
    p[ong[0]], l[ong[0]], stage[ong[0]] = 0, 0, 1  # the most urgent request is decoding
    want = select_batch(p.tolist(), l.tolist(), stage.tolist(), heap.tolist(), buf.tolist(),
                        ong.tolist(), 2000)
    assert run_select(p, l, stage, heap, buf, ong, 2000) == want


@pytest.mark.parametrize("n_cached,n_dem", [(0, 0), (0, 3), (1, 1), (100, 7), (5000, 300),
                                            (8192, 4000), (8192, 0), (3000, 2500)])
def test_evict(n_cached, n_dem):
    import paper_2506_12204_amd as ss
    rng = np.random.default_rng(n_cached * 31 + n_dem)
    n_ids = 1 << 18
    p = rng.integers(0, 5, n_ids).astype(np.uint8)
    l = rng.integers(0, 100, n_ids).astype(np.int32)  # small range: many ties
    cached = rng.permutation(n_ids)[:n_cached].astype(np.int32)
    kv = rng.integers(0, 1 << 30, n_cached).astype(np.int64)
    kv[: n_cached // 10] = 0
    demands = rng.integers(0, 1 << 31, n_dem).astype(np.int64)
    usage = int(kv.sum()) + 12345
    for capacity in (usage + int(demands.sum()) + 1, usage, usage // 2, 0):
        print(f"[gpu] evict cached={n_cached} demands={n_dem} capacity={capacity}", flush=True)
        want_v, want_u = evict(p.tolist(), l.tolist(), cached.tolist(), kv.tolist(), usage,
                               capacity, demands.tolist())
        v, u = ss.evict(dev(p, np.uint8), dev(l, np.int32), dev(cached, np.int32),
                        dev(kv, np.int64), usage, capacity, dev(demands, np.int64))
        assert v.cpu().numpy().tolist() == want_v
        assert u.cpu().numpy().tolist() == want_u


@pytest.mark.parametrize("n_cached,n_dem", [(8193, 10), (65536, 16384), (100000, 0),
                                            (65536, 1), (20000, 70000)])
def test_evict_beyond_lds(n_cached, n_dem):
    import paper_2506_12204_amd as ss
    rng = np.random.default_rng(n_cached + 7 * n_dem)
    n_ids = 1 << 20
    p = rng.integers(0, 5, n_ids).astype(np.uint8)
    l = rng.integers(0, 100, n_ids).astype(np.int32)  # small range: many ties
    cached = rng.permutation(n_ids)[:n_cached].astype(np.int32)
    kv = rng.integers(0, 1 << 30, n_cached).astype(np.int64)
    kv[: n_cached // 10] = 0
    demands = rng.integers(0, 1 << 20, n_dem).astype(np.int64)
    usage = int(kv.sum()) + 12345
    for capacity in (usage + int(demands.sum()) + 1, usage // 2, 0):
        print(f"[gpu] evict (merged in the workspace) cached={n_cached} demands={n_dem} "
              f"capacity={capacity}", flush=True)
        want_v, want_u = evict(p.tolist(), l.tolist(), cached.tolist(), kv.tolist(), usage,
                               capacity, demands.tolist())
        v, u = ss.evict(dev(p, np.uint8), dev(l, np.int32), dev(cached, np.int32),
                        dev(kv, np.int64), usage, capacity, dev(demands, np.int64))
        assert v.cpu().numpy().tolist() == want_v
        assert u.cpu().numpy().tolist() == want_u


def test_errors_beyond_lds():
    import paper_2506_12204_amd as ss
    n = 50000
    p = dev(np.zeros(n, np.uint8), np.uint8)
    l = dev(np.arange(n, dtype=np.int32), np.int32)
    st = dev(np.ones(n, np.uint8), np.uint8)
    buf = np.arange(5000, dtype=np.int32)
    buf[4321] = n + 3  # an id outside [0, n_ids)
    with pytest.raises(ss.SemschedError):
        ss.select_batch(p, l, st, None, dev(buf, np.int32), None, 4500)
    cached = np.arange(9000, dtype=np.int32)
    kv = np.ones(9000, np.int64)
    kv[8999] = -1
    with pytest.raises(ss.SemschedRangeError):
        ss.evict(p, l, dev(cached, np.int32), dev(kv, np.int64), 5, 1, dev(np.array([1]), np.int64))
    # later good calls are not affected
    buf[4321] = 4321
    bt, pu = ss.select_batch(p, l, st, None, dev(buf, np.int32), None, 4500)
    assert bt.cpu().tolist() == list(range(4500)) and pu.cpu().tolist() == []
    kv[8999] = 1
    v, u = ss.evict(p, l, dev(cached, np.int32), dev(kv, np.int64), 9000, 9000,
                    dev(np.array([2]), np.int64))
    assert u.cpu().tolist() == [2] and v.cpu().tolist() == [8999, 8998]


def test_errors():
    import paper_2506_12204_amd as ss
    p = dev(np.zeros(10, np.uint8), np.uint8)
    l = dev(np.ones(10, np.int32), np.int32)
    st = dev(np.zeros(10, np.uint8), np.uint8)
    with pytest.raises(ss.SemschedError):
        ss.select_batch(p, l, st, dev(np.array([1, 12]), np.int32), None, None, 2)
    with pytest.raises(ss.SemschedRangeError):
        ss.evict(p, l, dev(np.array([1, 2]), np.int32), dev(np.array([3, -1]), np.int64), 5, 1,
                 dev(np.array([1]), np.int64))
    with pytest.raises(ss.SemschedError):
        ss.evict(p, l, dev(np.array([1, 99]), np.int32), dev(np.array([3, 1]), np.int64), 5, 1,
                 dev(np.array([1]), np.int64))
    # a later good call is not affected
    v, u = ss.evict(p, l, dev(np.array([1, 2]), np.int32), dev(np.array([3, 4]), np.int64), 7, 7,
                    dev(np.array([1]), np.int64))
    assert u.cpu().tolist() == [1]


def test_full_range_keys_and_ids():
    # every key field at full width: ranks 0..255, lengths up to 2^31 - 1
    # (both ends present), ids up to 2^27, and equal (rank, length) pairs, so
    # that the sort runs a pass on every varying byte of the id and the key
    import paper_2506_12204_amd as ss
    rng = np.random.default_rng(77)
    n_ids = 1 << 27
    p = np.zeros(n_ids, np.uint8)
    l = np.zeros(n_ids, np.int32)
    ids = rng.choice(n_ids, 4096 * 3 + 8192, replace=False).astype(np.int32)
    ids[0], ids[1] = 0, n_ids - 1
    p[ids] = rng.integers(0, 256, ids.size)
    l[ids] = rng.integers(0, 2**31 - 1, ids.size, endpoint=True)
    l[ids[:2]] = (0, 2**31 - 1)
    l[ids[2:400]] = 12345  # ties on (rank, length) across ids
    p[ids[2:400]] = 7
    stage = (rng.random(n_ids) < 0.5).astype(np.uint8)
    waiting = ids[:4096]
    heap = waiting[np.lexsort((waiting, l[waiting], p[waiting]))]
    buf, ong = ids[4096:8192], ids[8192:12288]
    print("[gpu] select, full-range keys", flush=True)
    want = select_batch(p, l, stage, heap.tolist(), buf.tolist(), ong.tolist(), 4096)
    assert run_select(p, l, stage, heap, buf, ong, 4096) == want
    cached = ids[-8192:]
    kv = rng.integers(0, 1 << 20, cached.size).astype(np.int64)
    demands = rng.integers(0, 1 << 24, 500).astype(np.int64)
    usage = int(kv.sum())
    print("[gpu] evict, full-range keys", flush=True)
    want_v, want_u = evict(p, l, cached.tolist(), kv.tolist(), usage, usage // 3, demands.tolist())
    v, u = ss.evict(dev(p, np.uint8), dev(l, np.int32), dev(cached, np.int32), dev(kv, np.int64),
                    usage, usage // 3, dev(demands, np.int64))
    assert v.cpu().numpy().tolist() == want_v
    assert u.cpu().numpy().tolist() == want_u


def test_packed_key_spans():
    # keys whose varying bits fit one u64 once packed (the sorts' packed form):
    # lengths 2^20 + [0, 5000) and ranks 64 + [0, 6) (constant bits above
    # the spans of both words, which the keys get back after the passes), ids
    # that are multiples of 16 (a span starting at bit 4), ties on the key
    import paper_2506_12204_amd as ss
    rng = np.random.default_rng(78)
    n_ids = 1 << 22
    p = np.full(n_ids, 64, np.uint8)
    l = np.full(n_ids, 1 << 20, np.int32)
    ids = (16 * rng.choice(n_ids // 16, 4096 * 3 + 8192, replace=False)).astype(np.int32)
    p[ids] = 64 + rng.integers(0, 6, ids.size)
    l[ids] = (1 << 20) + rng.integers(0, 5000, ids.size)
    l[ids[:300]] = (1 << 20) + 77  # ties on (rank, length) across ids
    p[ids[:300]] = 65
    stage = (rng.random(n_ids) < 0.5).astype(np.uint8)
    waiting = ids[:4096]
    heap = waiting[np.lexsort((waiting, l[waiting], p[waiting]))]
    buf, ong = ids[4096:8192], ids[8192:12288]
    print("[gpu] select, packed key spans", flush=True)
    want = select_batch(p, l, stage, heap.tolist(), buf.tolist(), ong.tolist(), 4096)
    assert run_select(p, l, stage, heap, buf, ong, 4096) == want
    cached = ids[-8192:]
    kv = rng.integers(0, 1 << 20, cached.size).astype(np.int64)
    demands = rng.integers(0, 1 << 24, 500).astype(np.int64)
    usage = int(kv.sum())
    print("[gpu] evict, packed key spans", flush=True)
    want_v, want_u = evict(p, l, cached.tolist(), kv.tolist(), usage, usage // 3, demands.tolist())
    v, u = ss.evict(dev(p, np.uint8), dev(l, np.int32), dev(cached, np.int32), dev(kv, np.int64),
                    usage, usage // 3, dev(demands, np.int64))
    assert v.cpu().numpy().tolist() == want_v
    assert u.cpu().numpy().tolist() == want_u
