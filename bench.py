#!/usr/bin/env python3
"""Benchmark of the semantic-scheduling hot path on one MI355X.

One step = one complete schedule of a single queue of n = 2^26 requests
(5 urgency classes uniform, predicted lengths uniform in [1, 32768]):
order, every request's wait, and exact total and per-class waits, with the
inputs already resident in HBM. Prints ONE JSON line.

  python bench.py [--steps K] [--warmup W] [--no-cpu-baseline] [--op insert]

Besides whole-step throughput it reports, for the dominant kernel, the
achieved bandwidth from its algorithmic bytes and its average duration
(HIP events recorded by the library around that kernel, on its stream), and
the CPU oracle timed on this host as a baseline.
"""

from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "scheduled requests/sec + achieved HBM GB/s, single queue n=2^26, 1 GPU"
HBM_PEAK_GBPS = 8000.0
# Algorithmic bytes per request moved by each stage of the long-queue path.
# The n = 2^26 queue takes the compact layout (u32 elements between the
# passes); SEMSCHED_NO_COMPACT=1 forces the u64 element layout.
if os.environ.get("SEMSCHED_NO_COMPACT") == "1":
    STAGE_BYTES = {
        "hist": 5,    # read priority (1 B) + length (4 B)
        "first": 13,  # read priority + length (5 B), write the packed u64 element (8 B)
        "final": 20,  # read the element (8 B), write order (4 B) + wait (8 B)
    }
else:
    STAGE_BYTES = {
        "hist": 5,    # read priority (1 B) + length (4 B)
        "first": 9,   # read priority + length (5 B), write the u32 element (4 B)
        "final": 16,  # read the element (4 B), write order (4 B) + wait (8 B)
    }
PATH_BYTES = 17  # the whole schedule's own inputs + outputs per request
# Peak rate of 32-bit integer VALU work on MI355X: 256 CUs x 4 SIMDs x 16
# lanes per clock (a wave64 instruction takes 4 clocks on a SIMD) x 2.4 GHz,
# in lane operations per second.
VALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12
COUNTERS = os.path.join(ROOT, "profiles", "c3_step_counters.md")
CSRC = os.path.join(ROOT, "paper_2506_12204_amd", "csrc")
# the headers every kernel is built with: a counter measurement belongs to a
# kernel source together with these
COMMON = tuple(os.path.join(CSRC, h) for h in ("device_common.h", "block_common.h", "kernels.h"))
FINAL_SOURCE = (os.path.join(CSRC, "global_sort.hip"),) + COMMON
MERGE_COUNTERS = os.path.join(ROOT, "profiles", "insert_merge_c3_counters.md")
MERGE_SOURCE = (os.path.join(CSRC, "insert.hip"),) + COMMON
WORKLOAD_TEXT = {
    "c3": "single queue n=2^26, 5 urgency classes uniform, lengths uniform int32 in [1,32768], "
          "seed 2",
    "c2": "single queue n=2^20, 10 Zipf(1.2) classes, lognormal lengths, seed 1",
    "c4": "65,536 queues x 256 requests, 4 urgency classes uniform, lognormal lengths, seed 3",
    "c5": "16,384 queues of sizes U[1,4096], 8 classes (70 % in class 7), Pareto lengths "
          "with 30 % copied from the left neighbour, seed 4",
    "long": "16 queues x 2^20 requests, 5 urgency classes uniform, lengths uniform in "
            "[1,32768], 20 % copying an earlier request's class and length, seed 3",
}


def long_queue_workload():
    """16 queues of 2^20 requests: every queue is longer than one workgroup's
    LDS holds, so the whole batch goes through the segmented sort of long
    queues (the queues are cut into tiles of the batch, ranked per queue)."""
    from workloads import Workload, fuzz_segments
    p, l, off = fuzz_segments([1 << 20] * 16, seed=3, classes=5, max_len=32768)
    return Workload(name="long", priority=p, length=l, offsets=off, num_classes=5,
                    meta={"queues": 16, "queue_size": 1 << 20, "seed": 3})
POLICY_COUNTERS = os.path.join(ROOT, "profiles", "policy_c3_counters.md")
POLICY_SOURCE = (os.path.join(CSRC, "policy.hip"),) + COMMON
# The pass each policy's roofline is taken on: its name, the algorithmic
# bytes per request (FCFS and HPJF: rank and length read, order and wait
# written; SJF's final sort pass: its compact element read, order and wait
# written), the stage whose events bracket it, the source file its counters
# belong to.
POLICY_PASS = {
    "fcfs": ("f_write: identity order and waits", 17, "policy", POLICY_SOURCE),
    "hpjf": ("h_scatter: stable scatter by rank", 17, "policy", POLICY_SOURCE),
    "sjf": ("g_final_pay: final pass of the sort by (length, id), ranks carried "
            "(order, waits, class totals)", 16, "final", FINAL_SOURCE),
}


class HipEvents:
    """hipEvent_t handles from the HIP runtime already loaded by torch."""

    def __init__(self):
        self.rt = ctypes.CDLL("libamdhip64.so.7", mode=os.RTLD_NOLOAD | os.RTLD_GLOBAL)
        self.rt.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.rt.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float),
                                                ctypes.c_void_p, ctypes.c_void_p]
        self.rt.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self) -> int:
        ev = ctypes.c_void_p()
        if self.rt.hipEventCreate(ctypes.byref(ev)) != 0:
            raise RuntimeError("hipEventCreate failed")
        return ev.value

    def elapsed_ms(self, a: int, b: int) -> float:
        ms = ctypes.c_float()
        if self.rt.hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(a),
                                       ctypes.c_void_p(b)) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(ms.value)

    def destroy(self, ev: int) -> None:
        self.rt.hipEventDestroy(ctypes.c_void_p(ev))


def code_sha(paths) -> str:
    """SHA-256 of C++ sources (a path or a sequence of paths, in order) with
    their // comments and blank lines removed: what identifies the kernel a
    counter measurement belongs to."""
    if isinstance(paths, str):
        paths = (paths,)
    lines = []
    for path in paths:
        lines.append("// " + os.path.basename(path))
        with open(path) as f:
            for line in f:
                code = line.split("//", 1)[0].rstrip()
                if code:
                    lines.append(code)
    return hashlib.sha256("\n".join(lines).encode()).hexdigest()


def host_info() -> dict:
    """The host the CPU baselines ran on: usable threads and CPU model."""
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count()
    return {"nproc": usable, "cpu_count": os.cpu_count(), "cpu_model": model}


def median_of_runs(fn, runs: int = 3):
    """Median wall time (s) of `runs` calls of fn, and the first call's result."""
    import statistics
    times, first = [], None
    for k in range(runs):
        t = time.perf_counter()
        r = fn()
        times.append(time.perf_counter() - t)
        if k == 0:
            first = r
    return statistics.median(times), first


def time_steps(step, steps: int):
    """Run `steps` steps on torch's current stream with an event before each
    and after the last: per-step times, their median and mean (ms). The
    device is synchronised before the first event and after the last."""
    import statistics
    import torch
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    ev[0].record()
    for k in range(steps):
        step(k)
        ev[k + 1].record()
    torch.cuda.synchronize()
    per = [ev[k].elapsed_time(ev[k + 1]) for k in range(steps)]
    return per, statistics.median(per), ev[0].elapsed_time(ev[-1]) / steps


def profile_values(path: str, source: str, keys, n: int):
    """`key: value` figures of a committed rocprofv3 summary, or None when it
    was taken on another version of `source` (comments aside) or another n."""
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith(("|", "#", " ")):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip().strip("`")
    if kv.get("code_sha256") != code_sha(source) or kv.get("n") != str(n):
        return None
    try:
        return {k: float(kv[k]) for k in keys}
    except (KeyError, ValueError):
        return None


def counter_traffic(n: int, counters: str = COUNTERS, source: str = FINAL_SOURCE,
                    prefix: str = ""):
    """HBM bytes per launch of a kernel from committed rocprofv3 counters.

    The summary file carries `key: value` lines (n, code_sha256,
    hbm_bytes_per_launch). Null when the counters were taken on a different
    version of the kernel source (comments aside) or another request count.
    """
    if not os.path.exists(counters):
        return None
    kv = {}
    with open(counters) as f:
        for line in f:
            if ":" in line and not line.startswith(("|", "#", " ")):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip().strip("`")
    sha = kv.get(prefix + "code_sha256", kv.get("code_sha256"))  # (a kernel may have its own)
    if sha != code_sha(source) or kv.get("n") != str(n):
        return None
    key = prefix + "hbm_bytes_per_launch"
    return float(kv[key]) if key in kv else None


def copy_probe() -> int:
    """Plain 1 GiB device-to-device copy: the calibration run for the byte
    counters (FETCH_SIZE / WRITE_SIZE of a copy of known size)."""
    import torch
    n = 1 << 28  # int32 elements
    a = torch.ones(n, dtype=torch.int32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    s = torch.cuda.Event(enable_timing=True)
    e = torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(10):
        b.copy_(a)
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / 10
    print(json.dumps({"copy_bytes": 4 * n, "ms": ms, "read_plus_write_GBps": 8 * n / ms / 1e6}))
    return 0


INSERT_ARRIVALS = 1 << 16
# Algorithmic bytes of the insertion's merge pass: an earlier entry reads and
# writes its order (4 B) and wait (8 B); an arrival reads its order, wait and
# insertion point (4 + 8 + 4 B) and the earlier wait at that point (8 B), and
# writes 12 B.
MERGE_OLD_BYTES = 24
MERGE_NEW_BYTES = 36


def bench_insert(args) -> int:
    """Insert the last 2^16 requests of the n = 2^26 workload into the
    schedule of the others (sem_insert); one step = one insertion."""
    import numpy as np
    import torch
    import paper_2506_12204_amd as ss
    from workloads import generate

    w = generate("c3")
    n = w.n
    m = INSERT_ARRIVALS
    n_old = n - m
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    p = torch.from_numpy(w.priority).to(dev)
    l = torch.from_numpy(w.length).to(dev)
    old = ss.Scheduler(n_old, dev)
    old.run(p[:n_old], l[:n_old])
    old.check()
    ins = ss.Inserter(n_old, m, dev)
    print(f"[bench] insert {m} arrivals into a schedule of {n_old}; warmup {args.warmup}",
          file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        ins.run(p, l, old.order, old.wait)
    ins.check()
    hip = HipEvents()
    pairs = [(hip.create(), hip.create()) for _ in range(args.steps)]
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for k in range(args.steps):
        ss.trace_stage(ss.STAGE_MERGE, *pairs[k])
        ins.run(p, l, old.order, old.wait)
    t1.record()
    torch.cuda.synchronize()
    ins.check()
    ms_step = t0.elapsed_time(t1) / args.steps
    merge_ms = sum(hip.elapsed_ms(a, b) for a, b in pairs) / args.steps
    for a, b in pairs:
        hip.destroy(a)
        hip.destroy(b)
    print(f"[bench] {args.steps} inserts: {ms_step:.4f} ms each; merge pass {merge_ms:.4f} ms",
          file=sys.stderr, flush=True)
    merge_bytes = MERGE_OLD_BYTES * n_old + MERGE_NEW_BYTES * m
    achieved = merge_bytes / (merge_ms * 1e-3) / 1e9
    out = {
        "metric": "merged schedule requests/s, 2^16 arrivals into a queue of 2^26 - 2^16, 1 GPU",
        "value": n / (ms_step * 1e-3),
        "unit": "requests/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {
            "workload": ("insert the last 2^16 requests of the single queue n=2^26 "
                         "(5 urgency classes uniform, lengths uniform int32 in [1,32768], "
                         "seed 2) into the schedule of the others"),
            "n_old": n_old, "arrivals": m, "parallelism": "single GPU",
        },
        "roofline": {
            "bound": "hbm", "kernel": "insertion merge pass", "achieved": achieved,
            "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBPS,
            "traffic": counter_traffic(n, MERGE_COUNTERS, MERGE_SOURCE),
            "bytes_per_launch": merge_bytes, "avg_launch_ms": merge_ms,
        },
    }
    if not args.no_cpu_baseline:
        from oracle import c_oracle_insert
        o_old = old.order.cpu().numpy()
        w_old = old.wait.cpu().numpy()
        t = time.perf_counter()
        want = c_oracle_insert(w.priority, w.length, n_old, o_old, w_old)
        dt = time.perf_counter() - t
        same = (want[0].tobytes() == ins.order.cpu().numpy().tobytes()
                and want[1].tobytes() == ins.wait.cpu().numpy().tobytes()
                and list(want[2]) == ss.totals_to_ints(ins.totals))
        out["cpu_baseline"] = {
            "value": n / dt, "unit": "requests/s", "cores": 1, "kind": "oracle",
            "sample": (f"the full workload (n={n}): the plain C oracle checks the earlier "
                       f"schedule and schedules all requests (merge sort + running sum), "
                       f"single thread"),
        }
        out["parity"] = "bit-exact vs oracle" if same else "MISMATCH vs oracle"
        if not same:
            print(json.dumps(out))
            return 1
    print(json.dumps(out))
    return 0


def bench_policy(args) -> int:
    """One comparison policy (FCFS / SJF / HPJF) on the n = 2^26 workload;
    one step = the whole schedule under that policy."""
    import torch
    import paper_2506_12204_amd as ss
    from workloads import generate

    code = {"fcfs": ss.POLICY_FCFS, "sjf": ss.POLICY_SJF, "hpjf": ss.POLICY_HPJF}[args.policy]
    w = generate(args.workload)
    n = w.n
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    p = torch.from_numpy(w.priority).to(dev)
    l = torch.from_numpy(w.length).to(dev)
    sched = ss.PolicyScheduler(n, code, dev)
    print(f"[bench] policy {args.policy} workload {args.workload} n={n}; warmup {args.warmup}",
          file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        sched.run(p, l)
    sched.check()
    hip = HipEvents()
    pairs = [(hip.create(), hip.create()) for _ in range(args.steps)]
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    kernel, per_req, stage, source = POLICY_PASS[args.policy]
    for k in range(args.steps):
        ss.trace_stage(ss.STAGE_FINAL if stage == "final" else ss.STAGE_POLICY, *pairs[k])
        sched.run(p, l)
    t1.record()
    torch.cuda.synchronize()
    sched.check()
    ms_step = t0.elapsed_time(t1) / args.steps
    pass_ms = sum(hip.elapsed_ms(a, b) for a, b in pairs) / args.steps
    for a, b in pairs:
        hip.destroy(a)
        hip.destroy(b)
    print(f"[bench] {args.steps} schedules: {ms_step:.4f} ms each; {kernel}: {pass_ms:.4f} ms",
          file=sys.stderr, flush=True)
    pass_bytes = per_req * n
    achieved = pass_bytes / (pass_ms * 1e-3) / 1e9
    out = {
        "metric": f"scheduled requests/s under {args.policy.upper()}, single queue, 1 GPU",
        "value": n / (ms_step * 1e-3),
        "unit": "requests/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {"workload": WORKLOAD_TEXT[args.workload], "n": n,
                   "policy": args.policy, "parallelism": "single GPU"},
        "roofline": {
            "bound": "hbm", "kernel": kernel, "achieved": achieved,
            "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBPS,
            "traffic": counter_traffic(n, POLICY_COUNTERS, source, args.policy + "."),
            "bytes_per_launch": pass_bytes, "avg_launch_ms": pass_ms,
        },
    }
    if not args.no_cpu_baseline:
        from oracle import c_oracle_policy
        t = time.perf_counter()
        want = c_oracle_policy(w.priority, w.length, code)
        dt = time.perf_counter() - t
        same = (want[0].tobytes() == sched.order.cpu().numpy().tobytes()
                and want[1].tobytes() == sched.wait.cpu().numpy().tobytes()
                and list(want[2]) == ss.totals_to_ints(sched.totals))
        out["cpu_baseline"] = {
            "value": n / dt, "unit": "requests/s", "cores": 1, "kind": "oracle",
            "sample": (f"the full workload (n={n}): the plain C oracle's merge sort by the "
                       f"policy's key and running sum, single thread"),
        }
        out["parity"] = "bit-exact vs oracle" if same else "MISMATCH vs oracle"
        if not same:
            print(json.dumps(out))
            return 1
    print(json.dumps(out))
    return 0


# the A100 / Qwen1.5-7B constants of the paper's appendix (seconds per token or
# token^2: alpha1, alpha2, beta, gamma1, gamma2), used in microseconds. (The
# A100 / 4B prefill constant as printed, 1.466e-2 s per token^2, would put
# most service times at the 2^31 - 1 ceiling.)
COST_A100_7B = (5.135e-7, 1.481e-4, 1e-4, 1.349e-8, 1.330e-2)
COST_COUNTERS = os.path.join(ROOT, "profiles", "cost_c3_counters.md")


def bench_cost(args) -> int:
    """Schedule the n = 2^26 workload by (priority, cost-model service time,
    id): the service-time pass and the queue kernels; one step = one call."""
    import numpy as np
    import torch
    import paper_2506_12204_amd as ss
    from workloads import cost_tokens, generate

    class Model:  # Q32.32 microseconds, rounded to nearest
        pass
    model = Model()
    for name, v in zip(("alpha1", "alpha2", "beta", "gamma1", "gamma2"), COST_A100_7B):
        setattr(model, name, int(round(v / 1e-6 * (1 << 32))))
    w = generate(args.workload)
    n = w.n
    prompt, decoded = cost_tokens(w.length)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    p = torch.from_numpy(w.priority).to(dev)
    out_t = torch.from_numpy(w.length).to(dev)
    pr_t = torch.from_numpy(prompt).to(dev)
    de_t = torch.from_numpy(decoded).to(dev)
    sched = ss.CostScheduler(n, model, dev)
    print(f"[bench] cost-model schedule, workload {args.workload} n={n}; warmup {args.warmup}",
          file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        sched.run(p, pr_t, out_t, de_t)
    sched.check()
    hip = HipEvents()
    stages = [("cost", ss.STAGE_COST), ("hist", ss.STAGE_HIST), ("first", ss.STAGE_FIRST),
              ("mid", ss.STAGE_MID), ("final", ss.STAGE_FINAL)]
    pairs = {name: [(hip.create(), hip.create()) for _ in range(args.steps)]
             for name, _ in stages}
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for k in range(args.steps):
        for name, code in stages:
            ss.trace_stage(code, *pairs[name][k])
        sched.run(p, pr_t, out_t, de_t)
    t1.record()
    torch.cuda.synchronize()
    sched.check()
    ms_step = t0.elapsed_time(t1) / args.steps
    stage_ms = {name: sum(hip.elapsed_ms(a, b) for a, b in pairs[name]) / args.steps
                for name, _ in stages}
    for lst in pairs.values():
        for a, b in lst:
            hip.destroy(a)
            hip.destroy(b)
    print(f"[bench] {args.steps} steps: {ms_step:.4f} ms/step; stages {stage_ms}",
          file=sys.stderr, flush=True)
    # algorithmic bytes per request: the service pass reads three counts and
    # writes one; these keys (3 rank bits, about 29 service-time bits) and 26
    # id bits share one u64 element: the first pass reads 5 and writes 8
    # bytes, each of the two middle passes reads 8 to count and 8 to move and
    # writes 8, the final pass reads 8 and writes order and wait
    bytes_per_req = {"cost": 16, "hist": 5, "first": 13, "mid": 48, "final": 20}
    dom = max(stage_ms, key=stage_ms.get)
    achieved = bytes_per_req[dom] * n / (stage_ms[dom] * 1e-3) / 1e9
    out = {
        "metric": "requests/s scheduled by (urgency, cost-model service time), single queue, 1 GPU",
        "value": n / (ms_step * 1e-3),
        "unit": "requests/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {
            "workload": (WORKLOAD_TEXT[args.workload] + "; predicted output = those lengths, "
                         "prompt U[1,4096], 25 % part-way decoded (seed 5); A100 / "
                         "Qwen1.5-7B constants of the paper's appendix, microseconds"),
            "n": n, "parallelism": "single GPU",
        },
        "roofline": {
            "bound": "hbm", "kernel": f"{dom} pass", "achieved": achieved,
            "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBPS,
            "traffic": counter_traffic(n, COST_COUNTERS, FINAL_SOURCE, dom + "."),
            "bytes_per_request": bytes_per_req[dom], "avg_launch_ms": stage_ms[dom],
        },
        "stage_ms": stage_ms,
    }
    if not args.no_cpu_baseline:
        from oracle import c_oracle_queue, c_oracle_service_times
        from oracle import CostModel
        cm = CostModel(model.alpha1, model.alpha2, model.beta, model.gamma1, model.gamma2)
        t = time.perf_counter()
        s = c_oracle_service_times(prompt, w.length, decoded, cm)
        want = c_oracle_queue(w.priority, s)
        dt = time.perf_counter() - t
        same = (want[0].tobytes() == sched.order.cpu().numpy().tobytes()
                and want[1].tobytes() == sched.wait.cpu().numpy().tobytes()
                and list(want[2]) == ss.totals_to_ints(sched.totals)
                and s.tobytes() == sched.service.cpu().numpy().tobytes())
        out["cpu_baseline"] = {
            "value": n / dt, "unit": "requests/s", "cores": 1, "kind": "oracle",
            "sample": (f"the full workload (n={n}): the plain C oracle's service times "
                       f"(128-bit integers) and merge-sort schedule, single thread"),
        }
        out["parity"] = "bit-exact vs oracle" if same else "MISMATCH vs oracle"
        if not same:
            print(json.dumps(out))
            return 1
    print(json.dumps(out))
    return 0


BATCHED_SOURCE = (os.path.join(CSRC, "batched.hip"),) + COMMON


def bench_batched(args) -> int:
    """Batched independent queues through the asynchronous entry point:
    outputs and workspace allocated once, K calls enqueued back to back on
    torch's current stream, an event before every call. Bytes per request as
    in the single queue (rank and length read; order and wait written) plus
    each queue's offset and 128-bit totals."""
    import numpy as np
    import torch
    import paper_2506_12204_amd as ss
    from workloads import generate, workload_sha256

    w = long_queue_workload() if args.workload == "long" else generate(args.workload)
    n = w.n
    s = len(w.offsets) - 1
    c = int(w.num_classes)
    maxseg = int(np.diff(w.offsets).max())
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    p = torch.from_numpy(w.priority).to(dev)
    l = torch.from_numpy(w.length).to(dev)
    off = torch.from_numpy(w.offsets.astype(np.int64)).to(dev)
    order = torch.empty(n, dtype=torch.int32, device=dev)
    wait = torch.empty(n, dtype=torch.int64, device=dev)
    totals = torch.empty((s, 1 + c, 2), dtype=torch.int64, device=dev)
    # room for the requests of queues longer than the LDS cap (none in C4 and
    # C5), counted on the host before the timed region
    sizes = np.diff(w.offsets)
    long_requests = int(sizes[sizes > ss.SEGMENT_CAP].sum())
    ws_bytes = ss.workspace_bytes(long_requests, s)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    stream = ss._stream_handle(dev)

    def run(_k=0):
        rc = ss.lib.sem_schedule_batched_async(
            ss._ptr(p), ss._ptr(l), ss._ptr(off), s, c, ss._ptr(order),
            ss._ptr(wait), ss._ptr(totals), ss._ptr(ws), ws_bytes, stream)
        ss._raise(rc, "sem_schedule_batched_async")

    def check():
        ss._raise(ss.lib.sem_check(ss._ptr(ws), stream), "sem_check")

    print(f"[bench] workload {args.workload}: {s} queues, n={n}, longest {maxseg}; "
          f"warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        run()
    check()
    per, ms_step, ms_mean = time_steps(run, args.steps)
    check()
    alg_bytes = 17 * n + 8 * (s + 1) + 16 * s * (1 + c)
    gbps = alg_bytes / (ms_step * 1e-3) / 1e9
    print(f"[bench] {args.steps} calls: median {ms_step:.4f} ms (mean {ms_mean:.4f}), "
          f"{gbps:.0f} GB/s algorithmic", file=sys.stderr, flush=True)
    prof = profile_values(os.path.join(ROOT, "profiles", f"batched_{args.workload}_counters.md"),
                          BATCHED_SOURCE, ["hbm_bytes_per_call", "valu_insts_per_call"], n)
    traffic = prof["hbm_bytes_per_call"] if prof else None
    hbm = {"hbm_achieved_GBps": gbps, "hbm_peak_GBps": HBM_PEAK_GBPS,
           "hbm_frac": gbps / HBM_PEAK_GBPS, "bytes_per_request": 17,
           "counter_GBps": (traffic / (ms_step * 1e-3) / 1e9) if traffic else None}
    if prof:
        # the committed counters show the call's kernels bound by instruction
        # issue: VALU wave-instructions per call x 64 lanes over the call time
        valu_tops = prof["valu_insts_per_call"] * 64 / (ms_step * 1e-3) / 1e12
        roofline = {"bound": "alu", "kernel": "whole batched call", "achieved": valu_tops,
                    "peak": VALU_PEAK_TOPS, "unit": "TOP/s (32-bit integer VALU lane operations)",
                    "frac": valu_tops / VALU_PEAK_TOPS, "traffic": traffic, **hbm}
    else:
        roofline = {"bound": "hbm", "kernel": "whole batched call", "achieved": gbps,
                    "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": gbps / HBM_PEAK_GBPS,
                    "traffic": traffic, **hbm}
    out = {
        "metric": "scheduled requests/sec, batched independent queues, 1 GPU",
        "value": n / (ms_step * 1e-3),
        "unit": "requests/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "ms_per_step_mean": ms_mean,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {"workload": WORKLOAD_TEXT[args.workload], "n": n, "queues": s,
                   "parallelism": "single GPU", "input_sha256": workload_sha256(w)},
        "roofline": roofline,
    }
    if not args.no_cpu_baseline:
        from oracle import c_oracle_batched, c_oracle_batched_parallel
        dt, want = median_of_runs(lambda: c_oracle_batched(w.priority, w.length, w.offsets, c))
        dtp, wantp = median_of_runs(
            lambda: c_oracle_batched_parallel(w.priority, w.length, w.offsets, c))
        got = (order.cpu().numpy(), wait.cpu().numpy(), ss.totals_to_ints(totals))
        same = (want[0].tobytes() == got[0].tobytes() and want[1].tobytes() == got[1].tobytes()
                and list(want[2]) == got[2])
        host = host_info()
        out["cpu_baseline"] = {
            "value": n / dt, "unit": "requests/s", "cores": 1, "kind": "oracle",
            "sample": (f"the full workload (n={n}): the plain C oracle, queue by queue "
                       f"(merge sort + running sum), single thread, median of 3 runs"),
            **host,
        }
        out["cpu_baseline_parallel"] = {
            "value": n / dtp, "unit": "requests/s", "cores": wantp[3],
            "kind": "oracle, queues spread over OpenMP threads",
            "sample": f"the full workload (n={n}), median of 3 runs",
            **host,
        }
        out["parity"] = "bit-exact vs oracle" if same else "MISMATCH vs oracle"
        if not same:
            print(json.dumps(out))
            return 1
    print(json.dumps(out), flush=True)
    return 0


def bench_iteration(args) -> int:
    """One scheduling iteration of Algorithms 2 and 4 on the n = 2^26 queue:
    select the next batch (b = 256) from the schedule's head, a buffer of 4096
    arrivals and 256 ongoing requests, then evict for the selected batch's
    KV demands from 8192 cached requests. One step = both calls."""
    import numpy as np
    import torch
    import paper_2506_12204_amd as ss
    from workloads import generate

    b, nu, no, nr = 256, 4096, 256, 8192
    w = generate(args.workload)
    n = w.n
    rng = np.random.default_rng(6)
    stage = (rng.random(n) < 0.5).astype(np.uint8)
    ids = rng.permutation(n).astype(np.int32)
    buf, ong, cached = ids[:nu], ids[nu:nu + no], ids[nu + no:nu + no + nr]
    kv = (rng.integers(1, 4097, nr) * 131072).astype(np.int64)   # tokens x 128 KiB
    demands = (rng.integers(1, 4097, b) * 131072).astype(np.int64)
    usage = int(kv.sum())
    capacity = usage  # every incoming request must evict
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    t = lambda a: torch.from_numpy(a).to(dev)
    p, l, st = t(w.priority), t(w.length), t(stage)
    sched = ss.Scheduler(n, dev)
    sched.run(p, l)
    sched.check()
    heap = sched.order  # the waiting requests' schedule (only its head is read)
    tb, to, tc, tk, td = t(buf), t(ong), t(cached), t(kv), t(demands)
    batch = torch.empty(b, dtype=torch.int32, device=dev)
    pushed = torch.empty(b + no, dtype=torch.int32, device=dev)
    counts = torch.empty(2, dtype=torch.int64, device=dev)
    victims = torch.empty(nr, dtype=torch.int32, device=dev)
    upto = torch.empty(b, dtype=torch.int64, device=dev)
    ws1 = torch.empty(256, dtype=torch.uint8, device=dev)
    ws2 = torch.empty(256, dtype=torch.uint8, device=dev)
    stream = ss._stream_handle(dev)
    P = ss._ptr

    def step():
        rc = ss.lib.sem_select_batch_async(P(p), P(l), P(st), n, P(heap), n, P(tb), nu, P(to),
                                           no, b, P(batch), P(pushed), P(counts), P(ws1), 256,
                                           stream)
        ss._raise(rc, "sem_select_batch_async")
        rc = ss.lib.sem_evict_async(P(p), P(l), n, P(tc), P(tk), nr, usage, capacity, P(td), b,
                                    P(victims), P(upto), P(ws2), 256, stream)
        ss._raise(rc, "sem_evict_async")

    print(f"[bench] scheduling iteration: b={b} buffer={nu} ongoing={no} cached={nr}; "
          f"warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    ss._raise(ss.lib.sem_check(P(ws1), stream), "sem_check")
    ss._raise(ss.lib.sem_check(P(ws2), stream), "sem_check")
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for _ in range(args.steps):
        step()
    t1.record()
    torch.cuda.synchronize()
    ms_step = t0.elapsed_time(t1) / args.steps
    print(f"[bench] {args.steps} iterations: {ms_step * 1e3:.1f} us each", file=sys.stderr,
          flush=True)
    # algorithmic bytes: ids, keys and stages of the candidates and the
    # ongoing requests read, batch and pushed lists written; ids, keys and KV
    # sizes of the cached requests, demands read, victims written
    sel_bytes = (b + nu + no) * (4 + 1 + 4 + 1) + (b + no) * 4 * 2
    ev_bytes = nr * (4 + 1 + 4 + 8 + 4) + b * (8 + 8)
    achieved = (sel_bytes + ev_bytes) / (ms_step * 1e-3) / 1e9
    out = {
        "metric": "scheduling iterations/s (stage-aware selection + eviction), 1 GPU",
        "value": 1e3 / ms_step,
        "unit": "iterations/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {"workload": (f"the schedule of the single queue n=2^26 (seed 2) as the heap; "
                                f"b={b}, {nu} buffered arrivals, {no} ongoing, {nr} cached "
                                f"requests (KV 128 KiB per token, 1..4096 tokens), half of the "
                                f"requests decoding (seed 6)"),
                   "parallelism": "single GPU, one workgroup per call"},
        "roofline": {"bound": "hbm", "kernel": "b_select + b_evict", "achieved": achieved,
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": None, "bytes_per_launch": sel_bytes + ev_bytes,
                     "avg_launch_ms": ms_step},
    }
    if not args.no_cpu_baseline:
        from oracle import evict, select_batch
        heap_np = heap[: b].cpu().numpy().tolist()
        pl, ll, sl = w.priority, w.length, stage
        t_0 = time.perf_counter()
        reps = 0
        while True:
            want_sel = select_batch(pl, ll, sl, heap_np, buf.tolist(), ong.tolist(), b)
            want_ev = evict(pl, ll, cached.tolist(), kv.tolist(), usage, capacity,
                            demands.tolist())
            reps += 1
            if time.perf_counter() - t_0 > 2.0:
                break
        dt = (time.perf_counter() - t_0) / reps
        nb, npu = counts.cpu().tolist()
        same = (batch[:nb].cpu().tolist() == want_sel[0]
                and pushed[:npu].cpu().tolist() == want_sel[1]
                and upto.cpu().tolist() == want_ev[1]
                and victims[:want_ev[1][-1]].cpu().tolist() == want_ev[0])
        out["cpu_baseline"] = {
            "value": 1.0 / dt, "unit": "iterations/s", "cores": 1, "kind": "oracle",
            "sample": (f"the same iteration through the Python heap simulations "
                       f"(heapq), {reps} repetitions, single thread"),
        }
        out["parity"] = "bit-exact vs oracle" if same else "MISMATCH vs oracle"
        if not same:
            print(json.dumps(out))
            return 1
    print(json.dumps(out))
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="c3", choices=["c3", "c2", "c4", "c5", "long"],
                    help="c4, c5 and long are batched queues (the schedule op only)")
    ap.add_argument("--op", default="schedule", choices=["schedule", "insert", "policy", "cost", "iteration"],
                    help="schedule (default): the whole queue; insert: 2^16 arrivals "
                         "merged into the schedule of the rest; policy: the queue under "
                         "--policy; cost: ordered by cost-model service times; "
                         "iteration: one batch selection and eviction")
    ap.add_argument("--policy", default="fcfs", choices=["fcfs", "sjf", "hpjf"],
                    help="comparison policy timed by --op policy")
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the oracle leg (profiling runs)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only time a 1 GiB device copy (counter calibration)")
    args = ap.parse_args()
    if args.copy_probe:
        return copy_probe()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the schedule of one queue is not split "
              f"across GPUs in this build (asked for --gpus {args.gpus}).", file=sys.stderr)
        return 2
    if args.op == "insert":
        return bench_insert(args)
    if args.op == "policy":
        return bench_policy(args)
    if args.op == "cost":
        return bench_cost(args)
    if args.op == "iteration":
        return bench_iteration(args)
    if args.workload in ("c4", "c5", "long"):
        return bench_batched(args)

    return bench_queue(args)


STEP_COUNTERS = COUNTERS


def bench_queue(args) -> int:
    """The single-queue schedule (default: C3, n = 2^26). One step = one
    whole schedule; per-step events give the median; the library's stage
    events give the dominant pass's average duration."""
    import torch
    import paper_2506_12204_amd as ss
    from workloads import generate, workload_sha256

    w = generate(args.workload)
    n = w.n
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    p = torch.from_numpy(w.priority).to(dev)
    l = torch.from_numpy(w.length).to(dev)
    sched = ss.Scheduler(n, dev)
    print(f"[bench] workload {args.workload} n={n}; warmup {args.warmup}", file=sys.stderr,
          flush=True)

    for _ in range(args.warmup):
        sched.run(p, l)
    sched.check()

    hip = HipEvents()
    stages = [("hist", ss.STAGE_HIST), ("first", ss.STAGE_FIRST), ("final", ss.STAGE_FINAL)]
    pairs = {name: [(hip.create(), hip.create()) for _ in range(args.steps)]
             for name, _ in stages}

    def step(k):
        for name, code in stages:
            ss.trace_stage(code, *pairs[name][k])
        sched.run(p, l)

    per, ms_step, ms_mean = time_steps(step, args.steps)
    sched.check()
    stage_ms = {name: sum(hip.elapsed_ms(a, b) for a, b in pairs[name]) / args.steps
                for name, _ in stages}
    for lst in pairs.values():
        for a, b in lst:
            hip.destroy(a)
            hip.destroy(b)
    print(f"[bench] {args.steps} steps: median {ms_step:.4f} ms/step (mean {ms_mean:.4f}); "
          f"stages {stage_ms}", file=sys.stderr, flush=True)

    dom = max(stage_ms, key=stage_ms.get)
    hbm_achieved = STAGE_BYTES[dom] * n / (stage_ms[dom] * 1e-3) / 1e9
    traffic = counter_traffic(n) if dom == "final" else None
    prof = profile_values(STEP_COUNTERS, FINAL_SOURCE,
                          ["hbm_bytes_per_step", "final_valu_insts_per_launch"], n)
    step_bytes = prof["hbm_bytes_per_step"] if prof else None
    step_gbps = step_bytes / (ms_step * 1e-3) / 1e9 if step_bytes else None
    kernel = f"{dom} scatter pass" if dom != "hist" else "histogram pass"
    hbm = {
        # the dominant pass's algorithmic bytes per request over its launch time
        "hbm_achieved_GBps": hbm_achieved,
        "hbm_peak_GBps": HBM_PEAK_GBPS,
        "hbm_frac": hbm_achieved / HBM_PEAK_GBPS,
        "bytes_per_request": STAGE_BYTES[dom],
        "avg_launch_ms": stage_ms[dom],
        # the whole step: algorithmic bytes (17 per request) and the HBM
        # bytes the counters measured for one step, over the median step time
        "step_algorithmic_GBps": PATH_BYTES * n / (ms_step * 1e-3) / 1e9,
        "step_algorithmic_frac": PATH_BYTES * n / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        "step_counter_bytes": step_bytes,
        "step_counter_GBps": step_gbps,
        "step_frac": step_gbps / HBM_PEAK_GBPS if step_gbps else None,
    }
    if dom == "final" and prof:
        # The committed counters show the final pass bound by instruction
        # issue (VALU), not by HBM: its roofline is the integer VALU rate,
        # its VALU wave-instructions per launch (counters) x 64 lanes over the
        # launch time measured here.
        valu_tops = prof["final_valu_insts_per_launch"] * 64 / (stage_ms[dom] * 1e-3) / 1e12
        roofline = {"bound": "alu", "kernel": kernel, "achieved": valu_tops,
                    "peak": VALU_PEAK_TOPS, "unit": "TOP/s (32-bit integer VALU lane operations)",
                    "frac": valu_tops / VALU_PEAK_TOPS, "traffic": traffic, **hbm}
    else:
        roofline = {"bound": "hbm", "kernel": kernel, "achieved": hbm_achieved,
                    "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": hbm_achieved / HBM_PEAK_GBPS,
                    "traffic": traffic, **hbm}
    out = {
        "metric": METRIC,
        "value": n / (ms_step * 1e-3),
        "unit": "requests/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "ms_per_step_mean": ms_mean,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {
            "workload": WORKLOAD_TEXT[args.workload],
            "n": n,
            "parallelism": "single GPU",
            "input_sha256": workload_sha256(w),
        },
        "roofline": roofline,
        "stage_ms": stage_ms,
    }

    if not args.no_cpu_baseline:
        from oracle import c_oracle_queue
        order = sched.order.cpu().numpy()
        wait = sched.wait.cpu().numpy()
        totals = ss.totals_to_ints(sched.totals)
        dt, want = median_of_runs(lambda: c_oracle_queue(w.priority, w.length))
        same = (want[0].tobytes() == order.tobytes() and want[1].tobytes() == wait.tobytes()
                and list(want[2]) == list(totals))
        out["cpu_baseline"] = {
            "value": n / dt,
            "unit": "requests/s",
            "cores": 1,
            "kind": "oracle",
            "sample": f"the full workload (n={n}): the plain C oracle (merge sort + "
                      f"running sum, 128-bit totals), single thread, median of 3 runs",
            **host_info(),
        }
        out["parity"] = "bit-exact vs oracle" if same else "MISMATCH vs oracle"
        if not same:
            print(json.dumps(out))
            return 1
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
