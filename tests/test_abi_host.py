"""The C ABI library loads, exports every declared entry point, and rejects
bad arguments on the host (no GPU is touched by any call here)."""

import ctypes
import os
import re

import pytest

from tests._lib import LIB, ROOT, ensure_built

HEADER = os.path.join(ROOT, "include", "semsched.h")


@pytest.fixture(scope="module")
def ss():
    ensure_built()
    import paper_2506_12204_amd as mod
    return mod


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sem_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(ss):
    names = declared_functions()
    assert "sem_schedule" in names and "sem_schedule_batched" in names
    lib = ctypes.CDLL(LIB)
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(ss.SYMBOLS)


def test_strerror(ss):
    for code in (0, -1, -2, -3, -4, -5):
        assert ss.strerror(code)
    assert ss.strerror(-99) == "unknown error"


def test_workspace_sizes(ss):
    big = ss.workspace_bytes(1 << 20, 1)
    assert big > 24 * (1 << 20)  # two u64 key buffers + two u32 id buffers
    assert ss.workspace_bytes(0, 1) >= 256
    assert ss.workspace_bytes(-1, 1) == 0


def test_queue_argument_errors(ss):
    L = ss.lib
    nul = ctypes.c_void_p(0)
    fake = ctypes.c_void_p(1 << 40)  # never dereferenced: the call fails first
    assert L.sem_schedule(fake, fake, -1, fake, fake, fake) == ss.SEM_EINVAL
    assert L.sem_schedule(fake, fake, 1 << 31, fake, fake, fake) == ss.SEM_EINVAL
    assert L.sem_schedule(nul, fake, 5, fake, fake, fake) == ss.SEM_EINVAL
    assert L.sem_schedule(fake, fake, 5, fake, nul, fake) == ss.SEM_EINVAL
    assert L.sem_schedule(fake, fake, 5, fake, fake, nul) == ss.SEM_EINVAL
    # async: workspace missing, too small or misaligned
    assert L.sem_schedule_async(fake, fake, 5, fake, fake, fake, nul, 4096, nul) == ss.SEM_EINVAL
    assert L.sem_schedule_async(fake, fake, 1 << 20, fake, fake, fake, fake, 256,
                                nul) == ss.SEM_EINVAL
    assert L.sem_schedule_async(fake, fake, 5, fake, fake, fake, ctypes.c_void_p((1 << 40) + 8),
                                4096, nul) == ss.SEM_EINVAL


def test_batched_argument_errors(ss):
    L = ss.lib
    nul = ctypes.c_void_p(0)
    fake = ctypes.c_void_p(1 << 40)
    assert L.sem_schedule_batched(fake, fake, fake, -1, 4, fake, fake, fake) == ss.SEM_EINVAL
    assert L.sem_schedule_batched(fake, fake, fake, 3, 0, fake, fake, fake) == ss.SEM_EINVAL
    assert L.sem_schedule_batched(fake, fake, fake, 3, 257, fake, fake, fake) == ss.SEM_EINVAL
    assert L.sem_schedule_batched(fake, fake, nul, 3, 4, fake, fake, fake) == ss.SEM_EINVAL
    assert L.sem_schedule_batched(fake, fake, fake, 3, 4, fake, fake, nul) == ss.SEM_EINVAL
    A = L.sem_schedule_batched_async
    fixed = ss.workspace_bytes(0, 3)
    assert fixed > 256  # header and work lists
    # workspace missing, too small for the fixed part, or misaligned
    assert A(fake, fake, fake, 3, 4, fake, fake, fake, nul, fixed, nul) == ss.SEM_EINVAL
    assert A(fake, fake, fake, 3, 4, fake, fake, fake, fake, fixed - 1, nul) == ss.SEM_EINVAL
    assert A(fake, fake, fake, 3, 4, fake, fake, fake, ctypes.c_void_p((1 << 40) + 8), fixed,
             nul) == ss.SEM_EINVAL
    assert A(fake, fake, fake, 1 << 31, 4, fake, fake, fake, fake, 1 << 40, nul) == ss.SEM_EINVAL
    assert A(fake, fake, nul, 3, 4, fake, fake, fake, fake, fixed, nul) == ss.SEM_EINVAL


def test_batched_workspace_sizes(ss):
    # room for long queues grows with the bound on their requests
    base = ss.workspace_bytes(0, 1000)
    assert base >= 256 + 4 * 4 * 1000
    assert ss.workspace_bytes(100000, 1000) > base + 24 * 100000
    assert ss.workspace_bytes(-1, 1000) == 0
    assert ss.workspace_bytes(10, -1) == 0
    # one queue: enough for either call
    assert ss.workspace_bytes(1 << 20, 1) >= max(ss.workspace_bytes(1 << 20, 2) - 16,
                                                24 * (1 << 20))
    assert ss.lib.sem_check(ctypes.c_void_p(0), ctypes.c_void_p(0)) == ss.SEM_EINVAL


def test_binding_type_checks(ss):
    import torch
    p = torch.zeros(4, dtype=torch.uint8)
    l = torch.zeros(4, dtype=torch.int32)
    with pytest.raises(TypeError):
        ss.schedule(p, l)  # CPU tensors are refused: there is no CPU path
    with pytest.raises(TypeError):
        ss.schedule(p.to(torch.int32), l)


def test_insert_argument_errors(ss):
    L = ss.lib
    fake = ctypes.c_void_p(1 << 40)  # never dereferenced: the call fails first
    base = 1 << 40
    o_old = ctypes.c_void_p(base)
    w_old = ctypes.c_void_p(base + (1 << 20))
    assert L.sem_insert(fake, fake, -1, 5, o_old, w_old, fake, fake, fake) == ss.SEM_EINVAL
    assert L.sem_insert(fake, fake, 5, -1, o_old, w_old, fake, fake, fake) == ss.SEM_EINVAL
    assert L.sem_insert(fake, fake, 1 << 30, 1 << 30, o_old, w_old, fake, fake,
                        fake) == ss.SEM_EINVAL
    assert L.sem_insert(fake, fake, 5, 5, ctypes.c_void_p(0), w_old, fake, fake,
                        fake) == ss.SEM_EINVAL
    # outputs overlapping the earlier schedule
    assert L.sem_insert(fake, fake, 100, 5, o_old, w_old, ctypes.c_void_p(base + 8),
                        ctypes.c_void_p(base + (1 << 30)), fake) == ss.SEM_EINVAL
    assert L.sem_insert(fake, fake, 100, 5, o_old, w_old, ctypes.c_void_p(base + (1 << 30)),
                        ctypes.c_void_p(base + (1 << 20) + 16), fake) == ss.SEM_EINVAL
    assert ss.lib.sem_insert_workspace_bytes(-1, 3) == 0
    assert ss.lib.sem_insert_workspace_bytes(1000, 100) >= 256 + 16 * 100


def test_policy_argument_errors(ss):
    L = ss.lib
    nul = ctypes.c_void_p(0)
    fake = ctypes.c_void_p(1 << 40)  # never dereferenced: the call fails first
    for policy in (ss.POLICY_SEMANTIC, ss.POLICY_FCFS, ss.POLICY_SJF, ss.POLICY_HPJF):
        assert L.sem_schedule_policy(policy, fake, fake, -1, fake, fake, fake) == ss.SEM_EINVAL
        assert L.sem_schedule_policy(policy, nul, fake, 5, fake, fake, fake) == ss.SEM_EINVAL
        assert L.sem_schedule_policy(policy, fake, fake, 5, fake, fake, nul) == ss.SEM_EINVAL
        assert L.sem_policy_workspace_bytes(policy, 1 << 20) >= 256
        assert L.sem_schedule_policy_async(policy, fake, fake, 1 << 20, fake, fake, fake, fake,
                                           256, nul) == ss.SEM_EINVAL
    for bad in (-1, 4, 99):
        assert L.sem_schedule_policy(bad, fake, fake, 5, fake, fake, fake) == ss.SEM_EINVAL
        assert L.sem_policy_workspace_bytes(bad, 5) == 0
    assert L.sem_policy_workspace_bytes(ss.POLICY_SEMANTIC, 1 << 20) == ss.workspace_bytes(1 << 20)
    assert L.sem_policy_workspace_bytes(ss.POLICY_FCFS, -1) == 0


def test_cost_argument_errors(ss):
    L = ss.lib
    nul = ctypes.c_void_p(0)
    fake = ctypes.c_void_p(1 << 40)  # never dereferenced: the call fails first
    cm = ss.CostModelC(1, 2, 3, 4, 5)
    ref = ctypes.byref(cm)
    nocm = ctypes.cast(None, ctypes.POINTER(ss.CostModelC))
    assert L.sem_service_times(fake, fake, nul, -1, ref, fake) == ss.SEM_EINVAL
    assert L.sem_service_times(fake, fake, nul, 1 << 31, ref, fake) == ss.SEM_EINVAL
    assert L.sem_service_times(nul, fake, nul, 5, ref, fake) == ss.SEM_EINVAL
    assert L.sem_service_times(fake, fake, nul, 5, nocm, fake) == ss.SEM_EINVAL
    assert L.sem_service_times(fake, fake, nul, 5, ref, nul) == ss.SEM_EINVAL
    assert L.sem_evict_plan(fake, nul, 5, ref, fake, fake) == ss.SEM_EINVAL
    assert L.sem_evict_plan(fake, fake, 5, ref, fake, nul) == ss.SEM_EINVAL
    assert L.sem_schedule_cost(fake, fake, fake, nul, 5, ref, fake, fake, nul,
                               nul) == ss.SEM_EINVAL
    assert L.sem_schedule_cost(nul, fake, fake, nul, 5, ref, fake, fake, fake,
                               nul) == ss.SEM_EINVAL
    assert L.sem_cost_workspace_bytes(-1) == 0
    assert L.sem_cost_workspace_bytes(1 << 20) >= ss.workspace_bytes(1 << 20) + 4 * (1 << 20)
    assert L.sem_schedule_cost_async(fake, fake, fake, nul, 1 << 20, ref, fake, fake, fake, nul,
                                     fake, 256, nul) == ss.SEM_EINVAL


def test_select_and_evict_argument_errors(ss):
    L = ss.lib
    nul = ctypes.c_void_p(0)
    fake = ctypes.c_void_p(1 << 40)  # never dereferenced: the call fails first
    S = L.sem_select_batch
    assert S(fake, fake, fake, -1, fake, 5, nul, 0, nul, 0, 2, fake, fake, fake) == ss.SEM_EINVAL
    assert S(fake, fake, fake, 10, fake, 5, nul, 0, nul, 0, -1, fake, fake, fake) == ss.SEM_EINVAL
    # beyond the LDS sizes the lists are merged in the workspace, up to WIDE_MAX entries
    assert S(fake, fake, fake, 10, fake, ss.WIDE_MAX, nul, 0, fake, 1, ss.WIDE_MAX, fake, fake,
             fake) == ss.SEM_ENOTIMPL
    assert S(fake, fake, fake, 10, fake, 5, fake, ss.WIDE_MAX, fake, 1, 2, fake, fake,
             fake) == ss.SEM_ENOTIMPL
    SW = L.sem_select_workspace_bytes
    assert SW(5, 10, 10, 2) == 256 and SW(-1, 0, 0, 0) == 0
    big = SW(10000, ss.SELECT_CAP + 1, 100, 20000)
    assert big >= 256 + 24 * (10000 + ss.SELECT_CAP + 1 + 100)
    A = L.sem_select_batch_async
    assert A(fake, fake, fake, 10, fake, 10000, fake, ss.SELECT_CAP + 1, fake, 100, 20000, fake,
             fake, fake, fake, big - 1, nul) == ss.SEM_EINVAL
    assert S(fake, fake, nul, 10, fake, 5, nul, 0, nul, 0, 2, fake, fake, fake) == ss.SEM_EINVAL
    assert S(fake, fake, fake, 10, nul, 5, nul, 0, nul, 0, 2, fake, fake, fake) == ss.SEM_EINVAL
    assert S(fake, fake, fake, 10, fake, 5, nul, 0, nul, 0, 2, fake, fake, nul) == ss.SEM_EINVAL
    E = L.sem_evict
    assert E(fake, fake, 10, fake, fake, -1, 0, 0, fake, 1, fake, fake) == ss.SEM_EINVAL
    assert E(fake, fake, 10, fake, fake, ss.WIDE_MAX + 1, 0, 0, fake, 1, fake,
             fake) == ss.SEM_ENOTIMPL
    EW = L.sem_evict_workspace_bytes
    assert EW(ss.EVICT_CAP) == 256 and EW(-1) == 0
    assert EW(ss.EVICT_CAP + 1) >= 256 + 36 * (ss.EVICT_CAP + 1)
    assert L.sem_evict_async(fake, fake, 10, fake, fake, ss.EVICT_CAP + 1, 0, 0, fake, 1, fake,
                             fake, fake, EW(ss.EVICT_CAP + 1) - 1, nul) == ss.SEM_EINVAL
    assert E(fake, fake, 10, fake, nul, 5, 0, 0, fake, 1, fake, fake) == ss.SEM_EINVAL
    assert E(fake, fake, 10, fake, fake, 5, 0, 0, nul, 1, fake, fake) == ss.SEM_EINVAL
    assert L.sem_evict_async(fake, fake, 10, fake, fake, 5, 0, 0, fake, 1, fake, fake, nul, 256,
                             nul) == ss.SEM_EINVAL


def test_static_entry_point_host_checks(ss):
    L = ss.lib
    nul = ctypes.c_void_p(0)
    fake = ctypes.c_void_p(1 << 40)  # never dereferenced: the call fails first
    # the scratch holds the workspace of the largest size it accepts
    assert ss.workspace_bytes(ss.STATIC_MAX_N, 1) <= ss.STATIC_SCRATCH_BYTES
    assert L.sem_schedule_static(fake, fake, ss.STATIC_MAX_N + 1, fake, fake, fake, fake,
                                 nul) == ss.SEM_ENOMEM
    assert L.sem_schedule_static(fake, fake, 5, fake, fake, fake, nul, nul) == ss.SEM_EINVAL
    assert L.sem_schedule_static(fake, fake, -1, fake, fake, fake, fake, nul) == ss.SEM_EINVAL
    assert L.sem_schedule_static(nul, fake, 5, fake, fake, fake, fake, nul) == ss.SEM_EINVAL
