"""CPU oracle package (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package. The product library never imports it
and shares no code with it.

* ``semsched_oracle``: the pure-Python oracle (the plain definition).
* ``cost_oracle``: the cost model of Section 3.4 (service times, the cache
  and recompute decisions of an eviction) in exact integers.
* ``batch_oracle``: stage-aware batch selection and priority-based eviction
  (Algorithms 2-4) as literal heap simulations.
* ``c_oracle_*``: ctypes wrappers of ``oracle.c``, the same definition in
  plain C for large queues and for the timed CPU baseline.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from .batch_oracle import evict, eviction_order, select_batch  # noqa: F401
from .cost_oracle import (  # noqa: F401
    CostModel,
    evict_plan,
    keep_prefill_cache,
    schedule_cost,
    service_times,
    tokens_to_save,
)
from .semsched_oracle import (  # noqa: F401
    MAX_CLASSES,
    POLICIES,
    POLICY_FCFS,
    POLICY_HPJF,
    POLICY_SEMANTIC,
    POLICY_SJF,
    OracleRangeError,
    insert_queue,
    schedule_batched,
    schedule_policy,
    schedule_queue,
)

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

ORACLE_OK = 0
ORACLE_EINVAL = -1
ORACLE_ERANGE = -2


def build_c_oracle() -> str:
    """Compile oracle.c into liboracle.so (plain gcc; every oracle function is
    single-threaded except the OpenMP segment-parallel batched baseline)."""
    tmp = _LIB + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-shared", "-fPIC",
                           "-o", tmp, _SRC])
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build_c_oracle()
    lib = ctypes.CDLL(_LIB)
    vp = ctypes.c_void_p
    i64 = ctypes.c_int64
    lib.oracle_schedule.argtypes = [vp, vp, i64, vp, vp, vp, vp]
    lib.oracle_schedule.restype = ctypes.c_int
    lib.oracle_schedule_batched.argtypes = [vp, vp, vp, i64, ctypes.c_int32,
                                            vp, vp, vp, vp]
    lib.oracle_schedule_batched.restype = ctypes.c_int
    lib.oracle_schedule_batched_parallel.argtypes = [vp, vp, vp, i64, ctypes.c_int32,
                                                     vp, vp, vp, vp, vp]
    lib.oracle_schedule_batched_parallel.restype = ctypes.c_int
    lib.oracle_schedule_policy.argtypes = [ctypes.c_int, vp, vp, i64, vp, vp, vp, vp]
    lib.oracle_schedule_policy.restype = ctypes.c_int
    lib.oracle_service_times.argtypes = [vp, vp, vp, i64, vp, vp]
    lib.oracle_service_times.restype = ctypes.c_int
    lib.oracle_evict_plan.argtypes = [vp, vp, i64, vp, vp, vp]
    lib.oracle_evict_plan.restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


def _join128(lo: np.ndarray, hi: np.ndarray) -> list:
    return [int(h) << 64 | int(l) for l, h in zip(lo.tolist(), hi.tolist())]


def c_oracle_queue(p: np.ndarray, l: np.ndarray):
    """Single queue through oracle.c: (order i32, wait i64, totals[257] ints)."""
    p = np.ascontiguousarray(p, dtype=np.uint8)
    l = np.ascontiguousarray(l, dtype=np.int32)
    n = p.shape[0]
    order = np.empty(n, np.int32)
    wait = np.empty(n, np.int64)
    lo = np.zeros(257, np.uint64)
    hi = np.zeros(257, np.uint64)
    rc = _load().oracle_schedule(_ptr(p), _ptr(l), n, _ptr(order), _ptr(wait),
                                 _ptr(lo), _ptr(hi))
    if rc == ORACLE_ERANGE:
        raise OracleRangeError("length < 0 or priority out of range")
    if rc != ORACLE_OK:
        raise ValueError(f"oracle_schedule failed: {rc}")
    return order, wait, _join128(lo, hi)


def c_oracle_policy(p: np.ndarray, l: np.ndarray, policy: int):
    """Single queue under a comparison policy through oracle.c."""
    p = np.ascontiguousarray(p, dtype=np.uint8)
    l = np.ascontiguousarray(l, dtype=np.int32)
    n = p.shape[0]
    order = np.empty(n, np.int32)
    wait = np.empty(n, np.int64)
    lo = np.zeros(257, np.uint64)
    hi = np.zeros(257, np.uint64)
    rc = _load().oracle_schedule_policy(int(policy), _ptr(p), _ptr(l), n, _ptr(order),
                                        _ptr(wait), _ptr(lo), _ptr(hi))
    if rc == ORACLE_ERANGE:
        raise OracleRangeError("length < 0 or priority out of range")
    if rc != ORACLE_OK:
        raise ValueError(f"oracle_schedule_policy failed: {rc}")
    return order, wait, _join128(lo, hi)


def _coeffs(cm) -> np.ndarray:
    return np.array([cm.alpha1, cm.alpha2, cm.beta, cm.gamma1, cm.gamma2], dtype=np.uint64)


def c_oracle_service_times(prompt, output, decoded, cm) -> np.ndarray:
    """``service_times`` through oracle.c (int32 array)."""
    prompt = np.ascontiguousarray(prompt, dtype=np.int32)
    output = np.ascontiguousarray(output, dtype=np.int32)
    dec = None if decoded is None else np.ascontiguousarray(decoded, dtype=np.int32)
    n = prompt.shape[0]
    out = np.empty(n, np.int32)
    c = _coeffs(cm)
    rc = _load().oracle_service_times(_ptr(prompt), _ptr(output),
                                      ctypes.c_void_p(0) if dec is None else _ptr(dec), n,
                                      _ptr(c), _ptr(out))
    if rc == ORACLE_ERANGE:
        raise OracleRangeError("negative token count")
    if rc != ORACLE_OK:
        raise ValueError(f"oracle_service_times failed: {rc}")
    return out


def c_oracle_evict_plan(prompt, decoded, cm):
    """``evict_plan`` through oracle.c: (keep uint8, save int32)."""
    prompt = np.ascontiguousarray(prompt, dtype=np.int32)
    dec = np.ascontiguousarray(decoded, dtype=np.int32)
    n = prompt.shape[0]
    keep = np.empty(n, np.uint8)
    save = np.empty(n, np.int32)
    c = _coeffs(cm)
    rc = _load().oracle_evict_plan(_ptr(prompt), _ptr(dec), n, _ptr(c), _ptr(keep), _ptr(save))
    if rc == ORACLE_ERANGE:
        raise OracleRangeError("negative token count")
    if rc != ORACLE_OK:
        raise ValueError(f"oracle_evict_plan failed: {rc}")
    return keep, save


def c_oracle_batched(p: np.ndarray, l: np.ndarray, offsets: np.ndarray,
                     num_classes: int):
    """Batched queues through oracle.c; totals are S*(1+C) Python ints."""
    p = np.ascontiguousarray(p, dtype=np.uint8)
    l = np.ascontiguousarray(l, dtype=np.int32)
    offsets = np.ascontiguousarray(offsets, dtype=np.int64)
    n = p.shape[0]
    s = offsets.shape[0] - 1
    order = np.empty(n, np.int32)
    wait = np.empty(n, np.int64)
    lo = np.zeros(max(1, s * (1 + num_classes)), np.uint64)
    hi = np.zeros_like(lo)
    rc = _load().oracle_schedule_batched(_ptr(p), _ptr(l), _ptr(offsets), s,
                                         num_classes, _ptr(order), _ptr(wait),
                                         _ptr(lo), _ptr(hi))
    if rc == ORACLE_ERANGE:
        raise OracleRangeError("length < 0 or priority out of range")
    if rc != ORACLE_OK:
        raise ValueError(f"oracle_schedule_batched failed: {rc}")
    return order, wait, _join128(lo[: s * (1 + num_classes)],
                                 hi[: s * (1 + num_classes)])


def c_oracle_batched_parallel(p: np.ndarray, l: np.ndarray, offsets: np.ndarray,
                              num_classes: int):
    """c_oracle_batched with the queues spread over the host's threads
    (OpenMP); the per-queue arithmetic is the same. Returns (order, wait,
    totals, threads used)."""
    p = np.ascontiguousarray(p, dtype=np.uint8)
    l = np.ascontiguousarray(l, dtype=np.int32)
    offsets = np.ascontiguousarray(offsets, dtype=np.int64)
    n = p.shape[0]
    s = offsets.shape[0] - 1
    order = np.empty(n, np.int32)
    wait = np.empty(n, np.int64)
    lo = np.zeros(max(1, s * (1 + num_classes)), np.uint64)
    hi = np.zeros_like(lo)
    used = np.zeros(1, np.int32)
    rc = _load().oracle_schedule_batched_parallel(_ptr(p), _ptr(l), _ptr(offsets), s,
                                                  num_classes, _ptr(order), _ptr(wait),
                                                  _ptr(lo), _ptr(hi), _ptr(used))
    if rc == ORACLE_ERANGE:
        raise OracleRangeError("length < 0 or priority out of range")
    if rc != ORACLE_OK:
        raise ValueError(f"oracle_schedule_batched_parallel failed: {rc}")
    return order, wait, _join128(lo[: s * (1 + num_classes)],
                                 hi[: s * (1 + num_classes)]), int(used[0])


def c_oracle_insert(p: np.ndarray, l: np.ndarray, n_old: int,
                    order_old: np.ndarray, wait_old: np.ndarray):
    """Large-size ``insert_queue`` through oracle.c: checks that the earlier
    schedule is that of the first ``n_old`` requests, then schedules all."""
    o, w, _ = c_oracle_queue(p[:n_old], l[:n_old])
    if not (np.array_equal(o, order_old) and np.array_equal(w, wait_old)):
        raise ValueError("order_old / wait_old are not the schedule of the first n_old requests")
    return c_oracle_queue(p, l)
