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


def gpu_batched(p, l, offsets, num_classes, max_segment=None):
    import paper_2506_12204_amd as ss
    tp, tl, to = to_gpu(p.astype(np.uint8), l.astype(np.int32), offsets.astype(np.int64))
    order, wait, totals = ss.schedule_batched(tp, tl, to, num_classes, max_segment)
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
