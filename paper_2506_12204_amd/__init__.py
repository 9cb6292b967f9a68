"""MI355X (gfx950) semantic-scheduling hot path: Python binding.

This module only marshals arguments: it allocates outputs and workspaces as
torch ROCm tensors and calls the C ABI of ``libsemsched.so`` (declared in
``include/semsched.h``) on torch's current stream. Every step of the schedule
runs in the library's HIP kernels; there is no CPU fallback. Importing the
package fails loudly if the library has not been built
(``python paper_2506_12204_amd/build.py``).

What is computed (Section 3.2, Eq. 1 and Eq. 2 with all arrivals at time 0;
Algorithm 1's (f_e, f_t) min-heap order): requests sorted by (priority,
length, id), each request's wait as the exclusive prefix sum of the lengths
ahead of it, and the exact total and per-class waits.
"""

from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsemsched.so")

SEM_OK = 0
SEM_EINVAL = -1
SEM_ERANGE = -2
SEM_ENOMEM = -3
SEM_EDEVICE = -4
SEM_ENOTIMPL = -5
MAX_CLASSES = 256
SEGMENT_CAP = 16384

SYMBOLS = (
    "sem_schedule",
    "sem_schedule_batched",
    "sem_workspace_bytes",
    "sem_schedule_async",
    "sem_schedule_batched_async",
    "sem_set_stream",
    "sem_check",
    "sem_strerror",
    "sem_trace_stage",
    "sem_insert",
    "sem_insert_workspace_bytes",
    "sem_insert_async",
    "sem_schedule_policy",
    "sem_policy_workspace_bytes",
    "sem_schedule_policy_async",
    "sem_service_times",
    "sem_evict_plan",
    "sem_schedule_cost",
    "sem_cost_workspace_bytes",
    "sem_schedule_cost_async",
    "sem_select_batch",
    "sem_select_workspace_bytes",
    "sem_select_batch_async",
    "sem_evict",
    "sem_evict_workspace_bytes",
    "sem_evict_async",
    "sem_schedule_static",
)
STATIC_MAX_N = 1048576
STATIC_SCRATCH_BYTES = 33554432
SELECT_CAP = 4096  # selection sizes in one workgroup's LDS
EVICT_CAP = 8192   # cached requests in one workgroup's LDS
WIDE_MAX = 1 << 30
PREFILL, DECODE = 0, 1
STAGE_HIST, STAGE_FIRST, STAGE_FINAL, STAGE_MERGE, STAGE_POLICY, STAGE_COST, STAGE_MID = range(7)
# comparison policies (Section 4): the key fields before the id
POLICY_SEMANTIC, POLICY_FCFS, POLICY_SJF, POLICY_HPJF = 0, 1, 2, 3


class CostModelC(ctypes.Structure):
    """sem_cost_model: Q32.32 constants (time unit x 2^32 per token, per token^2
    for alpha1)."""
    _fields_ = [(name, ctypes.c_uint64)
                for name in ("alpha1", "alpha2", "beta", "gamma1", "gamma2")]


def cost_model(model) -> CostModelC:
    """Any object with integer attributes alpha1, alpha2, beta, gamma1, gamma2."""
    return CostModelC(*(int(getattr(model, k)) for k in ("alpha1", "alpha2", "beta",
                                                          "gamma1", "gamma2")))


class SemschedError(RuntimeError):
    """A library call returned a non-zero status."""

    def __init__(self, code: int, what: str):
        self.code = code
        super().__init__(f"{what}: {strerror(code)} ({code})")


class SemschedRangeError(SemschedError, ValueError):
    """Some length < 0 or some priority >= num_classes."""


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python paper_2506_12204_amd/build.py`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    lib.sem_schedule.argtypes = [vp, vp, i64, vp, vp, vp]
    lib.sem_schedule_batched.argtypes = [vp, vp, vp, i64, i32, vp, vp, vp]
    lib.sem_workspace_bytes.argtypes = [i64, i64]
    lib.sem_workspace_bytes.restype = sz
    lib.sem_schedule_async.argtypes = [vp, vp, i64, vp, vp, vp, vp, sz, vp]
    lib.sem_schedule_batched_async.argtypes = [vp, vp, vp, i64, i32, vp, vp, vp, vp, sz, vp]
    lib.sem_set_stream.argtypes = [vp]
    lib.sem_check.argtypes = [vp, vp]
    lib.sem_trace_stage.argtypes = [ctypes.c_int, vp, vp]
    lib.sem_trace_stage.restype = ctypes.c_int
    lib.sem_insert.argtypes = [vp, vp, i64, i64, vp, vp, vp, vp, vp]
    lib.sem_insert_workspace_bytes.argtypes = [i64, i64]
    lib.sem_insert_workspace_bytes.restype = sz
    lib.sem_insert_async.argtypes = [vp, vp, i64, i64, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.sem_schedule_policy.argtypes = [ctypes.c_int, vp, vp, i64, vp, vp, vp]
    lib.sem_policy_workspace_bytes.argtypes = [ctypes.c_int, i64]
    lib.sem_policy_workspace_bytes.restype = sz
    lib.sem_schedule_policy_async.argtypes = [ctypes.c_int, vp, vp, i64, vp, vp, vp, vp, sz, vp]
    cm = ctypes.POINTER(CostModelC)
    lib.sem_service_times.argtypes = [vp, vp, vp, i64, cm, vp]
    lib.sem_evict_plan.argtypes = [vp, vp, i64, cm, vp, vp]
    lib.sem_schedule_cost.argtypes = [vp, vp, vp, vp, i64, cm, vp, vp, vp, vp]
    lib.sem_cost_workspace_bytes.argtypes = [i64]
    lib.sem_cost_workspace_bytes.restype = sz
    lib.sem_schedule_cost_async.argtypes = [vp, vp, vp, vp, i64, cm, vp, vp, vp, vp, vp, sz, vp]
    lib.sem_select_batch.argtypes = [vp, vp, vp, i64, vp, i64, vp, i64, vp, i64, i64, vp, vp, vp]
    lib.sem_select_batch_async.argtypes = [vp, vp, vp, i64, vp, i64, vp, i64, vp, i64, i64, vp,
                                           vp, vp, vp, sz, vp]
    lib.sem_select_workspace_bytes.argtypes = [i64, i64, i64, i64]
    lib.sem_select_workspace_bytes.restype = sz
    lib.sem_evict_workspace_bytes.argtypes = [i64]
    lib.sem_evict_workspace_bytes.restype = sz
    lib.sem_evict.argtypes = [vp, vp, i64, vp, vp, i64, i64, i64, vp, i64, vp, vp]
    lib.sem_evict_async.argtypes = [vp, vp, i64, vp, vp, i64, i64, i64, vp, i64, vp, vp, vp, sz,
                                    vp]
    lib.sem_schedule_static.argtypes = [vp, vp, i64, vp, vp, vp, vp, vp]
    lib.sem_strerror.argtypes = [ctypes.c_int]
    lib.sem_strerror.restype = ctypes.c_char_p
    for name in ("sem_schedule", "sem_schedule_batched", "sem_schedule_async",
                 "sem_schedule_batched_async", "sem_set_stream", "sem_check", "sem_insert",
                 "sem_insert_async", "sem_schedule_policy", "sem_schedule_policy_async",
                 "sem_service_times", "sem_evict_plan", "sem_schedule_cost",
                 "sem_schedule_cost_async", "sem_select_batch", "sem_select_batch_async",
                 "sem_evict", "sem_evict_async", "sem_schedule_static"):
        getattr(lib, name).restype = ctypes.c_int
    return lib


lib = _load()


def strerror(code: int) -> str:
    return lib.sem_strerror(code).decode()


def _raise(code: int, what: str) -> None:
    if code == SEM_OK:
        return
    if code == SEM_ERANGE:
        raise SemschedRangeError(code, what)
    raise SemschedError(code, what)


def _ptr(t: Optional[torch.Tensor]):
    return ctypes.c_void_p(t.data_ptr() if t is not None and t.numel() else 0)


def _stream_handle(device: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _check_inputs(priority: torch.Tensor, length: torch.Tensor) -> None:
    if priority.dtype != torch.uint8 or length.dtype != torch.int32:
        raise TypeError("priority must be uint8 and length int32")
    if priority.device.type != "cuda" or length.device != priority.device:
        raise TypeError("priority and length must live on the same GPU")
    if priority.dim() != 1 or priority.shape != length.shape:
        raise ValueError("priority and length must be 1-D and the same size")
    if not (priority.is_contiguous() and length.is_contiguous()):
        raise ValueError("inputs must be contiguous")


def totals_to_ints(t: torch.Tensor) -> List[int]:
    """Decode an int64 [..., 2] (lo, hi) tensor of sem_i128 values."""
    flat = t.reshape(-1, 2).cpu().tolist()
    return [(hi << 64) | (lo & 0xFFFFFFFFFFFFFFFF) for lo, hi in flat]


def trace_stage(stage: int, before: int, after: int) -> None:
    """Arm one-shot hipEvent_t handles around one stage of the next long-queue call."""
    _raise(lib.sem_trace_stage(stage, ctypes.c_void_p(before), ctypes.c_void_p(after)),
           "sem_trace_stage")


def workspace_bytes(n: int, num_segments: int = 1) -> int:
    return int(lib.sem_workspace_bytes(n, num_segments))


class Scheduler:
    """Reusable single-queue schedule of a fixed size n on one device.

    Outputs and the workspace are allocated once; ``run`` enqueues the whole
    schedule on the current stream without synchronising, ``check`` waits
    and raises on a device-detected error.
    """

    def __init__(self, n: int, device="cuda"):
        self.n = int(n)
        self.device = torch.device(device)
        self.order = torch.empty(self.n, dtype=torch.int32, device=self.device)
        self.wait = torch.empty(self.n, dtype=torch.int64, device=self.device)
        self.totals = torch.empty((1 + MAX_CLASSES, 2), dtype=torch.int64, device=self.device)
        self.ws_bytes = workspace_bytes(self.n, 1)
        self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.device)

    def run(self, priority: torch.Tensor, length: torch.Tensor) -> None:
        _check_inputs(priority, length)
        if priority.numel() != self.n:
            raise ValueError("size differs from the Scheduler's n")
        rc = lib.sem_schedule_async(_ptr(priority), _ptr(length), self.n, _ptr(self.order),
                                    _ptr(self.wait), _ptr(self.totals), _ptr(self.workspace),
                                    self.ws_bytes, _stream_handle(self.device))
        _raise(rc, "sem_schedule_async")

    def check(self) -> None:
        _raise(lib.sem_check(_ptr(self.workspace), _stream_handle(self.device)), "sem_check")


def schedule(priority: torch.Tensor, length: torch.Tensor
             ) -> Tuple[torch.Tensor, torch.Tensor, List[int]]:
    """Schedule one queue. Returns (order int32, wait int64, totals[257] ints)."""
    _check_inputs(priority, length)
    s = Scheduler(priority.numel(), priority.device)
    s.run(priority, length)
    s.check()
    return s.order, s.wait, totals_to_ints(s.totals)


def schedule_static(priority: torch.Tensor, length: torch.Tensor,
                    out: Optional[Tuple[torch.Tensor, torch.Tensor, torch.Tensor, torch.Tensor]]
                    = None) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor, torch.Tensor]:
    """Schedule one queue through the allocation-free entry point (the library's
    static scratch stands in for the workspace; n <= STATIC_MAX_N).

    ``out`` = (order int32[n], wait int64[n], totals int64[257, 2], status
    int32[1]) preallocated by the caller; without it they are allocated here.
    Enqueues on the current stream without synchronising and returns the four
    tensors; status[0] holds SEM_OK or the device-detected error once the
    stream reaches it.
    """
    _check_inputs(priority, length)
    n = priority.numel()
    dev = priority.device
    if out is None:
        out = (torch.empty(n, dtype=torch.int32, device=dev),
               torch.empty(n, dtype=torch.int64, device=dev),
               torch.empty((1 + MAX_CLASSES, 2), dtype=torch.int64, device=dev),
               torch.empty(1, dtype=torch.int32, device=dev))
    order, wait, totals, status = out
    rc = lib.sem_schedule_static(_ptr(priority), _ptr(length), n, _ptr(order), _ptr(wait),
                                 _ptr(totals), _ptr(status), _stream_handle(dev))
    _raise(rc, "sem_schedule_static")
    return order, wait, totals, status


def schedule_batched(priority: torch.Tensor, length: torch.Tensor, offsets: torch.Tensor,
                     num_classes: int, blocking: bool = False,
                     long_requests: Optional[int] = None
                     ) -> Tuple[torch.Tensor, torch.Tensor, List[int]]:
    """Schedule independent queues laid out back to back.

    Returns (order int32 with queue-local ids, wait int64, totals as
    num_segments*(1+num_classes) ints, queue-major). By default the
    asynchronous call runs on the current stream (queues of any length, no
    host read of the offsets) and one check follows; ``long_requests`` bounds
    the requests in queues longer than SEGMENT_CAP (default: all of them) and
    sizes the workspace. ``blocking=True`` takes the blocking call instead.
    """
    _check_inputs(priority, length)
    if offsets.dtype != torch.int64 or offsets.device != priority.device or offsets.dim() != 1:
        raise TypeError("offsets must be a 1-D int64 tensor on the inputs' GPU")
    offsets = offsets.contiguous()
    s = offsets.numel() - 1
    if s < 0:
        raise ValueError("offsets needs at least one entry")
    n = priority.numel()
    dev = priority.device
    order = torch.empty(n, dtype=torch.int32, device=dev)
    wait = torch.empty(n, dtype=torch.int64, device=dev)
    totals = torch.empty((max(s, 1), 1 + num_classes, 2), dtype=torch.int64, device=dev)
    stream = _stream_handle(dev)
    if not blocking:
        lr = n if long_requests is None else int(long_requests)
        ws_bytes = int(lib.sem_workspace_bytes(lr, s))
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
        rc = lib.sem_schedule_batched_async(_ptr(priority), _ptr(length), _ptr(offsets), s,
                                            num_classes, _ptr(order), _ptr(wait), _ptr(totals),
                                            _ptr(ws), ws_bytes, stream)
        _raise(rc, "sem_schedule_batched_async")
        _raise(lib.sem_check(_ptr(ws), stream), "sem_check")
    else:
        lib.sem_set_stream(stream)
        rc = lib.sem_schedule_batched(_ptr(priority), _ptr(length), _ptr(offsets), s,
                                      num_classes, _ptr(order), _ptr(wait), _ptr(totals))
        _raise(rc, "sem_schedule_batched")
    return order, wait, totals_to_ints(totals[:s]) if s else []


class Inserter:
    """Reusable insertion of m arrivals into a schedule of n_old requests.

    ``run`` enqueues sem_insert_async on the current stream into this
    object's outputs (order, wait, totals of all n_old + m requests); ``check``
    waits and raises on a device-detected error.
    """

    def __init__(self, n_old: int, m: int, device="cuda"):
        self.n_old, self.m = int(n_old), int(m)
        self.device = torch.device(device)
        n = self.n_old + self.m
        self.order = torch.empty(n, dtype=torch.int32, device=self.device)
        self.wait = torch.empty(n, dtype=torch.int64, device=self.device)
        self.totals = torch.empty((1 + MAX_CLASSES, 2), dtype=torch.int64, device=self.device)
        self.ws_bytes = int(lib.sem_insert_workspace_bytes(self.n_old, self.m))
        self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.device)

    def run(self, priority: torch.Tensor, length: torch.Tensor, order_old: torch.Tensor,
            wait_old: torch.Tensor) -> None:
        _check_inputs(priority, length)
        if priority.numel() != self.n_old + self.m:
            raise ValueError("priority/length must hold n_old + m requests")
        if (order_old.dtype != torch.int32 or wait_old.dtype != torch.int64
                or order_old.numel() != self.n_old or wait_old.numel() != self.n_old
                or order_old.device != priority.device or wait_old.device != priority.device
                or not (order_old.is_contiguous() and wait_old.is_contiguous())):
            raise TypeError("order_old (int32) and wait_old (int64) must hold n_old entries "
                            "on the inputs' GPU")
        rc = lib.sem_insert_async(_ptr(priority), _ptr(length), self.n_old, self.m,
                                  _ptr(order_old), _ptr(wait_old), _ptr(self.order),
                                  _ptr(self.wait), _ptr(self.totals), _ptr(self.workspace),
                                  self.ws_bytes, _stream_handle(self.device))
        _raise(rc, "sem_insert_async")

    def check(self) -> None:
        _raise(lib.sem_check(_ptr(self.workspace), _stream_handle(self.device)), "sem_check")


def insert(priority: torch.Tensor, length: torch.Tensor, n_old: int, order_old: torch.Tensor,
           wait_old: torch.Tensor) -> Tuple[torch.Tensor, torch.Tensor, List[int]]:
    """Insert requests n_old.. into the schedule (order_old, wait_old) of the
    first n_old; returns the schedule of all (order, wait, totals[257] ints)."""
    s = Inserter(n_old, priority.numel() - int(n_old), priority.device)
    s.run(priority, length, order_old, wait_old)
    s.check()
    return s.order, s.wait, totals_to_ints(s.totals)


class PolicyScheduler:
    """Reusable single-queue schedule of size n under a comparison policy
    (POLICY_FCFS, POLICY_SJF, POLICY_HPJF or POLICY_SEMANTIC); ``run`` enqueues
    sem_schedule_policy_async on the current stream, ``check`` waits and raises
    on a device-detected error."""

    def __init__(self, n: int, policy: int, device="cuda"):
        self.n, self.policy = int(n), int(policy)
        self.device = torch.device(device)
        self.order = torch.empty(self.n, dtype=torch.int32, device=self.device)
        self.wait = torch.empty(self.n, dtype=torch.int64, device=self.device)
        self.totals = torch.empty((1 + MAX_CLASSES, 2), dtype=torch.int64, device=self.device)
        self.ws_bytes = int(lib.sem_policy_workspace_bytes(self.policy, self.n))
        if self.ws_bytes == 0:
            raise SemschedError(SEM_EINVAL, "sem_policy_workspace_bytes")
        self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.device)

    def run(self, priority: torch.Tensor, length: torch.Tensor) -> None:
        _check_inputs(priority, length)
        if priority.numel() != self.n:
            raise ValueError("size differs from the PolicyScheduler's n")
        rc = lib.sem_schedule_policy_async(self.policy, _ptr(priority), _ptr(length), self.n,
                                           _ptr(self.order), _ptr(self.wait), _ptr(self.totals),
                                           _ptr(self.workspace), self.ws_bytes,
                                           _stream_handle(self.device))
        _raise(rc, "sem_schedule_policy_async")

    def check(self) -> None:
        _raise(lib.sem_check(_ptr(self.workspace), _stream_handle(self.device)), "sem_check")


def schedule_policy(priority: torch.Tensor, length: torch.Tensor, policy: int
                    ) -> Tuple[torch.Tensor, torch.Tensor, List[int]]:
    """Schedule one queue under ``policy``; returns (order, wait, totals[257] ints)."""
    _check_inputs(priority, length)
    s = PolicyScheduler(priority.numel(), policy, priority.device)
    s.run(priority, length)
    s.check()
    return s.order, s.wait, totals_to_ints(s.totals)


def _check_counts(*arrays: Optional[torch.Tensor]) -> int:
    ref = next(a for a in arrays if a is not None)
    for a in arrays:
        if a is None:
            continue
        if a.dtype != torch.int32 or a.device != ref.device or a.device.type != "cuda":
            raise TypeError("token counts must be int32 tensors on one GPU")
        if a.dim() != 1 or a.numel() != ref.numel() or not a.is_contiguous():
            raise ValueError("token counts must be contiguous 1-D tensors of one size")
    return ref.numel()


def service_times(prompt: torch.Tensor, output: torch.Tensor, decoded: Optional[torch.Tensor],
                  model) -> torch.Tensor:
    """Remaining computation time of every request under the cost model (int32)."""
    n = _check_counts(prompt, output, decoded)
    out = torch.empty(n, dtype=torch.int32, device=prompt.device)
    lib.sem_set_stream(_stream_handle(prompt.device))
    cm = cost_model(model)
    _raise(lib.sem_service_times(_ptr(prompt), _ptr(output), _ptr(decoded), n, ctypes.byref(cm),
                                 _ptr(out)), "sem_service_times")
    return out


def evict_plan(prompt: torch.Tensor, decoded: torch.Tensor, model
               ) -> Tuple[torch.Tensor, torch.Tensor]:
    """Per evicted request: keep its prefill cache (uint8 0/1) and how many of
    its decoded tokens' cache to save (int32)."""
    n = _check_counts(prompt, decoded)
    keep = torch.empty(n, dtype=torch.uint8, device=prompt.device)
    save = torch.empty(n, dtype=torch.int32, device=prompt.device)
    lib.sem_set_stream(_stream_handle(prompt.device))
    cm = cost_model(model)
    _raise(lib.sem_evict_plan(_ptr(prompt), _ptr(decoded), n, ctypes.byref(cm), _ptr(keep),
                              _ptr(save)), "sem_evict_plan")
    return keep, save


class CostScheduler:
    """Reusable schedule of n requests by (priority, cost-model service time,
    id); ``run`` enqueues sem_schedule_cost_async on the current stream and
    leaves the service times in ``service``."""

    def __init__(self, n: int, model, device="cuda"):
        self.n = int(n)
        self.device = torch.device(device)
        self.model = cost_model(model)
        self.order = torch.empty(self.n, dtype=torch.int32, device=self.device)
        self.wait = torch.empty(self.n, dtype=torch.int64, device=self.device)
        self.service = torch.empty(self.n, dtype=torch.int32, device=self.device)
        self.totals = torch.empty((1 + MAX_CLASSES, 2), dtype=torch.int64, device=self.device)
        self.ws_bytes = int(lib.sem_cost_workspace_bytes(self.n))
        self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.device)

    def run(self, priority: torch.Tensor, prompt: torch.Tensor, output: torch.Tensor,
            decoded: Optional[torch.Tensor] = None) -> None:
        if priority.dtype != torch.uint8 or priority.numel() != self.n:
            raise TypeError("priority must be uint8 with n entries")
        if _check_counts(prompt, output, decoded) != self.n:
            raise ValueError("size differs from the CostScheduler's n")
        rc = lib.sem_schedule_cost_async(_ptr(priority), _ptr(prompt), _ptr(output),
                                         _ptr(decoded), self.n, ctypes.byref(self.model),
                                         _ptr(self.order), _ptr(self.wait), _ptr(self.totals),
                                         _ptr(self.service), _ptr(self.workspace), self.ws_bytes,
                                         _stream_handle(self.device))
        _raise(rc, "sem_schedule_cost_async")

    def check(self) -> None:
        _raise(lib.sem_check(_ptr(self.workspace), _stream_handle(self.device)), "sem_check")


def schedule_cost(priority: torch.Tensor, prompt: torch.Tensor, output: torch.Tensor,
                  decoded: Optional[torch.Tensor], model):
    """Schedule by (priority, service time, id); returns (order, wait,
    totals[257] ints, service times)."""
    s = CostScheduler(priority.numel(), model, priority.device)
    s.run(priority, prompt, output, decoded)
    s.check()
    return s.order, s.wait, totals_to_ints(s.totals), s.service


def _ids(t: Optional[torch.Tensor], device) -> Optional[torch.Tensor]:
    if t is None:
        return None
    if t.dtype != torch.int32 or t.device != device or t.dim() != 1 or not t.is_contiguous():
        raise TypeError("id lists must be contiguous 1-D int32 tensors on the inputs' GPU")
    return t


def select_batch(priority: torch.Tensor, length: torch.Tensor, stage: torch.Tensor,
                 heap_order: torch.Tensor, buffer: Optional[torch.Tensor],
                 ongoing: Optional[torch.Tensor], b: int) -> Tuple[torch.Tensor, torch.Tensor]:
    """Algorithm 2: (next batch, pushed-back requests), both in key order."""
    _check_inputs(priority, length)
    dev = priority.device
    if stage.dtype != torch.uint8 or stage.shape != priority.shape or stage.device != dev:
        raise TypeError("stage must be uint8 with one entry per request")
    heap_order, buffer, ongoing = (_ids(heap_order, dev), _ids(buffer, dev), _ids(ongoing, dev))
    nh = heap_order.numel() if heap_order is not None else 0
    nb = buffer.numel() if buffer is not None else 0
    no = ongoing.numel() if ongoing is not None else 0
    batch = torch.empty(max(int(b), 1), dtype=torch.int32, device=dev)
    pushed = torch.empty(max(int(b) + no, 1), dtype=torch.int32, device=dev)
    counts = torch.zeros(2, dtype=torch.int64, device=dev)
    lib.sem_set_stream(_stream_handle(dev))
    _raise(lib.sem_select_batch(_ptr(priority), _ptr(length), _ptr(stage), priority.numel(),
                                _ptr(heap_order), nh, _ptr(buffer), nb, _ptr(ongoing), no, int(b),
                                _ptr(batch), _ptr(pushed), _ptr(counts)), "sem_select_batch")
    nbat, npush = counts.tolist()
    return batch[:nbat], pushed[:npush]


def evict(priority: torch.Tensor, length: torch.Tensor, cached: torch.Tensor, kv: torch.Tensor,
          usage: int, capacity: int, demands: torch.Tensor) -> Tuple[torch.Tensor, torch.Tensor]:
    """Algorithms 3-4: (victims in eviction order, victims after each incoming
    request)."""
    _check_inputs(priority, length)
    dev = priority.device
    cached = _ids(cached, dev)
    if kv.dtype != torch.int64 or kv.shape != cached.shape or kv.device != dev:
        raise TypeError("kv must be int64 with one entry per cached request")
    if demands.dtype != torch.int64 or demands.device != dev or demands.dim() != 1:
        raise TypeError("demands must be a 1-D int64 tensor")
    kv, demands = kv.contiguous(), demands.contiguous()
    victims = torch.empty(max(cached.numel(), 1), dtype=torch.int32, device=dev)
    upto = torch.empty(max(demands.numel(), 1), dtype=torch.int64, device=dev)
    lib.sem_set_stream(_stream_handle(dev))
    _raise(lib.sem_evict(_ptr(priority), _ptr(length), priority.numel(), _ptr(cached), _ptr(kv),
                         cached.numel(), int(usage), int(capacity), _ptr(demands),
                         demands.numel(), _ptr(victims), _ptr(upto)), "sem_evict")
    upto = upto[:demands.numel()]
    k = int(upto[-1]) if demands.numel() else 0
    return victims[:k], upto
