"""Shared test helpers: load (building if needed) the HIP library and run it."""

import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2506_12204_amd", "libsemsched.so")


def ensure_built():
    if not os.path.exists(LIB):
        subprocess.check_call([sys.executable, os.path.join(ROOT, "paper_2506_12204_amd", "build.py")],
                              cwd=ROOT)


def gpu_available() -> bool:
    import torch
    return torch.cuda.is_available()


def to_gpu(*arrays):
    import torch
    return [torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in arrays]


def gpu_queue(p: np.ndarray, l: np.ndarray):
    """Schedule one queue on the GPU through the C ABI; numpy results."""
    import paper_2506_12204_amd as ss
    tp, tl = to_gpu(p.astype(np.uint8), l.astype(np.int32))
    order, wait, totals = ss.schedule(tp, tl)
    return order.cpu().numpy(), wait.cpu().numpy(), totals


def gpu_batched(p, l, offsets, num_classes, blocking=False, long_requests=None):
    """Batched schedule through the C ABI: the asynchronous call (workspace
    room for ``long_requests`` requests of long queues, default all) or the
    blocking one."""
    import paper_2506_12204_amd as ss
    tp, tl, to = to_gpu(p.astype(np.uint8), l.astype(np.int32), offsets.astype(np.int64))
    order, wait, totals = ss.schedule_batched(tp, tl, to, num_classes, blocking=blocking,
                                              long_requests=long_requests)
    return order.cpu().numpy(), wait.cpu().numpy(), totals


def assert_same(got, want, label=""):
    go, gw, gt = got
    wo, ww, wt = want
    wo = np.asarray(wo, dtype=np.int64)
    ww = np.asarray(ww, dtype=np.int64)
    assert go.shape == wo.shape, f"{label}: order size {go.shape} vs {wo.shape}"
    bad = np.flatnonzero(go.astype(np.int64) != wo)
    assert bad.size == 0, f"{label}: order differs at {bad[:8]} ({bad.size} positions)"
    bad = np.flatnonzero(gw.astype(np.int64) != ww)
    assert bad.size == 0, f"{label}: wait differs at {bad[:8]} ({bad.size} positions)"
    assert list(gt) == list(wt), f"{label}: totals differ"


def check_queue_by_definition(p, l, order, wait, totals):
    """The schedule's definition checked directly, for queues the oracle would
    take minutes on: order is a permutation of the ids and strictly
    increasing in the unique key (rank, length, id), so it is the one sorted
    order; every wait is the sum of the lengths before it; the totals are the
    exact sums of the waits, overall and per rank (Eq. 1)."""
    n = p.shape[0]
    assert order.shape == (n,) and wait.shape == (n,)
    if n == 0:
        assert all(t == 0 for t in totals)
        return
    assert order.min() >= 0 and order.max() < n
    seen = np.zeros(n, np.bool_)
    seen[order] = True
    assert seen.all(), "order is not a permutation"
    del seen
    po = p[order]
    lo = l[order]
    dp = np.diff(po.astype(np.int16))
    dl = np.diff(lo.astype(np.int64))
    di = np.diff(order.astype(np.int64))
    assert (dp >= 0).all(), "ranks decrease"
    assert (dl[dp == 0] >= 0).all(), "lengths decrease within a rank"
    assert (di[(dp == 0) & (dl == 0)] > 0).all(), "ids decrease within a key"
    del dp, dl, di
    assert wait[0] == 0
    assert np.array_equal(np.diff(wait), lo[:-1].astype(np.int64)), "waits"

    def exact_sum(v):  # int64 values >= 0, summed exactly in two 32-bit halves
        u = v.astype(np.uint64)
        return (int((u >> np.uint64(32)).sum()) << 32) + int((u & np.uint64(0xffffffff)).sum())

    assert totals[0] == exact_sum(wait), "grand total"
    present = np.bincount(po, minlength=256)
    for c in range(256):
        want = exact_sum(wait[po == c]) if present[c] else 0
        assert totals[1 + c] == want, f"class {c} total"
