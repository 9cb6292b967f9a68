"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Everything here is integer, so every comparison is bit-exact: order, every
wait and every 128-bit total. The oracle is the plain C oracle (oracle.c),
itself pinned to the pure-Python oracle and to the paper's optimisation
problem by the CPU tests.
"""

import os

import numpy as np
import pytest

from oracle import c_oracle_batched, c_oracle_queue
from tests._lib import (check_queue_by_definition, assert_same, ensure_built, gpu_available,
                        gpu_batched, gpu_queue, to_gpu)
from workloads import fuzz_queue, fuzz_segments, generate

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]


@pytest.fixture(scope="module", autouse=True)
def _built():
    ensure_built()


def say(*a):
    print(*a, flush=True)


def check_queue(p, l, label):
    say(f"[gpu] queue {label}: n={len(p)}")
    assert_same(gpu_queue(p, l), c_oracle_queue(p, l), label)


def check_batched(p, l, off, classes, label, forms=("async", "blocking"), want=None):
    if want is None:
        want = c_oracle_batched(p, l, off, classes)
    for form in forms:
        say(f"[gpu] batched {label} ({form}): n={len(p)} segments={len(off) - 1}")
        assert_same(gpu_batched(p, l, off, classes, blocking=form == "blocking"), want,
                    f"{label}-{form}")


# ---- the five workloads at full size -----------------------------------------

@pytest.mark.parametrize("name", ["c1", "c2", "c3"])
def test_workload_queue(name):
    w = generate(name)
    check_queue(w.priority, w.length, name)


@pytest.mark.parametrize("name", ["c4", "c5"])
def test_workload_batched(name):
    w = generate(name)
    check_batched(w.priority, w.length, w.offsets, w.num_classes, name)
    # the workspace without room for long queues (these workloads have none)
    say(f"[gpu] batched {name} (async, no long-queue room)")
    assert_same(gpu_batched(w.priority, w.length, w.offsets, w.num_classes, long_requests=0),
                c_oracle_batched(w.priority, w.length, w.offsets, w.num_classes), name)


def test_batched_repeat_many_workgroups_per_cu():
    # Regression: a barrier that let waves pass with LDS loads in flight let
    # another wave's counter reset overwrite staged elements, intermittently,
    # only when many workgroups shared a CU. Repeat the crowded launch.
    w = generate("c5")
    want = c_oracle_batched(w.priority, w.length, w.offsets, w.num_classes)
    for k in range(4):
        say(f"[gpu] c5 repeat {k}")
        assert_same(gpu_batched(w.priority, w.length, w.offsets, w.num_classes,
                                blocking=k % 2 == 1), want, f"c5-repeat{k}")


# ---- sizes around every tile and LDS-class boundary -----------------------------

SIZES = [0, 1, 2, 63, 64, 65, 255, 256, 257, 1023, 1024, 1025, 4095, 4096, 4097,
         16383, 16384, 16385, 24576, 24577, 65537, 100003]


@pytest.mark.parametrize("n", SIZES)
def test_fuzz_sizes(n):
    p, l = fuzz_queue(n, seed=n, classes=7, max_len=5000, tie_frac=0.3)
    check_queue(p, l, f"fuzz{n}")


@pytest.mark.parametrize("d0", ["8", "9", "10"])
@pytest.mark.parametrize("max_len", [2000, 32768])
def test_first_digit_widths(d0, max_len, monkeypatch):
    # max_len 2000 keeps the final digit under 256 values for every width
    # (compact layout); 32768 with 8 or 9 bits gives 640 or 320 (u64 layout)
    monkeypatch.setenv("SEMSCHED_D0", d0)
    p, l = fuzz_queue(200_000, seed=7, classes=5, max_len=max_len, tie_frac=0.2)
    check_queue(p, l, f"d0={d0},max_len={max_len}")


# ---- compact two-pass layout: id chunks and the sub-bucket search -------------

def test_compact_chunk_boundaries_inside_blocks():
    # 10M requests: 3 id chunks of 2^22 ids; the first pass's blocks hold
    # 49,152 ids, so both chunk boundaries fall inside a block
    p, l = fuzz_queue(10_000_000, seed=31, classes=5, max_len=32768, tie_frac=0.2)
    check_queue(p, l, "chunks-unaligned")


def test_compact_window_in_global_memory():
    # 99 % of the lengths are multiples of 1024 (first digit 0); the rest
    # spread over the other 1023 first digits, so the last blocks span
    # hundreds of buckets x 4 chunk slots: more sub-bucket starts than the
    # LDS window holds, and the search reads them from global memory
    rng = np.random.default_rng(32)
    n = 12_000_000
    p = rng.integers(0, 4, n).astype(np.uint8)
    l = (rng.integers(1, 8, n) * 1024).astype(np.int32)
    sprinkle = rng.random(n) < 0.01
    l[sprinkle] = rng.integers(1, 8192, int(sprinkle.sum()))
    check_queue(p, l, "window-global")


def test_compact_beyond_buffer_store_range():
    # 2^28 + 12,345 requests: past the size up to which the compact passes
    # store through buffer resources (2^28), so every block of the final pass
    # takes the kernel with plain stores; the largest queue tested (checked
    # against the definition: the oracle's merge sort takes minutes here)
    rng = np.random.default_rng(35)
    n = (1 << 28) + 12_345
    p = rng.integers(0, 5, n, dtype=np.uint8)
    l = rng.integers(1, 32769, n, dtype=np.int32)
    say(f"[gpu] queue 2^28+: n={n}")
    order, wait, totals = gpu_queue(p, l)
    check_queue_by_definition(p, l, order, wait, totals)


@pytest.mark.parametrize("n", [100_003, 5_000_000])
def test_u64_layout_when_compact_is_off(n, monkeypatch):
    monkeypatch.setenv("SEMSCHED_NO_COMPACT", "1")
    p, l = fuzz_queue(n, seed=33, classes=5, max_len=32768, tie_frac=0.2)
    check_queue(p, l, "no-compact")


# ---- degenerate and adversarial queues ----------------------------------------

@pytest.mark.parametrize("n", [300, 5000, 40000])
def test_all_keys_equal(n):
    check_queue(np.full(n, 3, np.uint8), np.full(n, 7, np.int32), "all-equal")


@pytest.mark.parametrize("n", [3000, 50000])
def test_reverse_sorted(n):
    p = np.repeat(np.arange(4, dtype=np.uint8)[::-1], n // 4 + 1)[:n]
    l = np.arange(n, 0, -1).astype(np.int32)
    check_queue(p, l, "reverse")


@pytest.mark.parametrize("n", [1000, 70000])
def test_one_class_and_zero_lengths(n):
    rng = np.random.default_rng(n)
    l = rng.integers(0, 3, n).astype(np.int32)
    check_queue(np.zeros(n, np.uint8), l, "one-class-zeros")


@pytest.mark.parametrize("classes,lo,hi,label", [
    (5, 0, 1 << 20, "one middle pass, 5 final digits"),
    (1, 0, 1 << 27, "one middle pass, lengths past 2^26, 128 final digits"),
    (5, 0, 1 << 29, "two middle passes, 3 final digits (the cost-model shape)"),
    (2, 1 << 26, (1 << 26) + (1 << 19), "two passes, lengths past 2^26"),
    (5, 0, 1 << 31, "34-bit keys: generic final pass"),
])
def test_wide_keys_with_few_final_digits(classes, lo, hi, label):
    # Keys of at most 32 bits (in the high word) with at most 256 final
    # digits but more than two passes or lengths of 2^26 and more: the wide
    # form of the big-tile final pass, reading the buffer of the pass before
    # it (either of the two)
    rng = np.random.default_rng(len(label))
    n = 300_000
    p = rng.integers(0, classes, n).astype(np.uint8)
    l = rng.integers(lo, hi, n, dtype=np.int64).astype(np.int32)
    l[:1000] = l[1000:2000]  # ties on (rank, length)
    check_queue(p, l, label)


@pytest.mark.parametrize("n", [2000, 50000])
def test_all_256_classes_full_length_range(n):
    # 256 classes x lengths up to 2^31-1: the widest keys; on the global path
    # this needs three middle passes.
    rng = np.random.default_rng(99)
    p = rng.integers(0, 256, n).astype(np.uint8)
    l = rng.integers(0, 2**31 - 1, n, dtype=np.int64).astype(np.int32)
    l[:5] = 2**31 - 1
    l[5:10] = 0
    check_queue(p, l, "256-classes")


def test_max_length_totals_beyond_2_64():
    n = 1 << 18
    p = np.zeros(n, np.uint8)
    l = np.full(n, 2**31 - 1, np.int32)
    got = gpu_queue(p, l)
    want = c_oracle_queue(p, l)
    assert_same(got, want, "int32-max")
    assert want[2][0] > 2**64


@pytest.mark.parametrize("n", [20000, 100003])
def test_forced_wide_layout(n, monkeypatch):
    monkeypatch.setenv("SEMSCHED_FORCE_WIDE", "1")
    p, l = fuzz_queue(n, seed=3, classes=9, max_len=100000, tie_frac=0.2)
    check_queue(p, l, "wide")
    rng = np.random.default_rng(5)
    p = rng.integers(0, 256, n).astype(np.uint8)
    l = rng.integers(0, 2**31 - 1, n, dtype=np.int64).astype(np.int32)
    check_queue(p, l, "wide-mid-passes")


@pytest.mark.parametrize("classes,hi", [(256, 2**31 - 1), (5, 1 << 29)])
def test_middle_passes_as_separate_launches(classes, hi, monkeypatch):
    # the per-phase launches of the middle passes (no grid barrier)
    monkeypatch.setenv("SEMSCHED_SPLIT_MID", "1")
    rng = np.random.default_rng(classes)
    n = 400_000
    p = rng.integers(0, classes, n).astype(np.uint8)
    l = rng.integers(0, hi, n, dtype=np.int64).astype(np.int32)
    l[:1000] = l[1000:2000]
    check_queue(p, l, f"split-mid-{classes}")


def test_repeatable_bit_for_bit():
    p, l = fuzz_queue(300_000, seed=11, classes=5, max_len=2000, tie_frac=0.5)
    first = gpu_queue(p, l)
    for _ in range(10):
        assert_same(gpu_queue(p, l), first, "repeat")


def _shifted(a, dtype):
    # a device copy that starts one element into its allocation
    import torch
    buf = np.concatenate([np.zeros(1, dtype), np.asarray(a, dtype)])
    return torch.from_numpy(buf).to("cuda")[1:]


@pytest.mark.parametrize("n", [5000, 100_003, 5_000_001])
def test_queue_unaligned_inputs(n):
    # lengths not 16-byte aligned, ranks not 4-byte aligned: the first
    # histogram pass then loads one request per lane instead of four (at 5M,
    # with the chunk counts of the compact layout); 5000 takes the LDS path
    import paper_2506_12204_amd as ss
    p, l = fuzz_queue(n, seed=51, classes=5, max_len=32768, tie_frac=0.2)
    tp, tl = _shifted(p, np.uint8), _shifted(l, np.int32)
    assert tl.data_ptr() % 16 != 0 and tp.data_ptr() % 4 != 0
    say(f"[gpu] queue unaligned: n={n}")
    order, wait, totals = ss.schedule(tp, tl)
    assert_same((order.cpu().numpy(), wait.cpu().numpy(), totals),
                c_oracle_queue(p, l), f"unaligned{n}")


def test_batched_unaligned_inputs():
    import paper_2506_12204_amd as ss
    sizes = [0, 7, 300, 4097, 16385, 70000, 1]
    p, l, off = fuzz_segments(sizes, seed=52, classes=6, max_len=3000)
    tp, tl = _shifted(p, np.uint8), _shifted(l, np.int32)
    to = _shifted(off, np.int64)
    assert tl.data_ptr() % 16 != 0 and tp.data_ptr() % 4 != 0
    say(f"[gpu] batched unaligned: n={len(p)}")
    order, wait, totals = ss.schedule_batched(tp, tl, to, 6)
    assert_same((order.cpu().numpy(), wait.cpu().numpy(), totals),
                c_oracle_batched(p, l, off, 6), "batched-unaligned")


# ---- batched inputs ------------------------------------------------------------

def test_batched_mixed_sizes_and_empty_queues():
    sizes = [0, 1, 0, 255, 256, 257, 1024, 1025, 4096, 4097, 0, 16384, 16385, 70000, 3]
    p, l, off = fuzz_segments(sizes, seed=21, classes=6, max_len=3000)
    check_batched(p, l, off, 6, "mixed")


def test_batched_long_and_many_small_queues():
    # queues of every size class, long ones among thousands of small ones
    rng = np.random.default_rng(24)
    sizes = rng.integers(0, 600, 5000)
    sizes[[0, 1, 2, 3, 4]] = [0, 1, 16384, 16385, 70000]
    sizes[[2500, 4999]] = [40000, 17000]
    rng.shuffle(sizes)
    p, l, off = fuzz_segments(sizes, seed=25, classes=5, max_len=32768)
    check_batched(p, l, off, 5, "long-and-small")


def test_batched_medium_queues_in_one_list_segment():
    # 2,400 queues: chunks of two queues on a 256-CU device, so the medium
    # queues (every pair whose chunk index is a multiple of 8) all fall into
    # one of the medium list's segments; the workgroups serving the other
    # segments find theirs empty and must help drain that one. Some of those
    # queues have keys too wide for a 32-bit element and are handed on.
    sizes = [300 + (i % 7) * 500 if (i // 2) % 8 == 0 else 10 for i in range(2400)]
    p, l, off = fuzz_segments(sizes, seed=29, classes=5, max_len=3000)
    for q in range(0, 2400, 160):
        l[off[q]:off[q + 1]] = np.random.default_rng(q).integers(0, 2**31 - 1, off[q + 1] - off[q])
    check_batched(p, l, off, 5, "one-segment")


@pytest.mark.parametrize("classes", [32, 33])
def test_batched_class_sums_at_the_copy_limit(classes):
    # the class sums of a queue are kept in eight copies while its classes
    # span at most 32 ranks, in one copy beyond that
    sizes = [5, 256, 257, 1000, 4096, 4097, 9000]
    p, l, off = fuzz_segments(sizes, seed=32 + classes, classes=classes, max_len=700)
    for q in range(len(sizes)):  # every queue spans the full range of ranks
        p[off[q]] = 0
        p[off[q + 1] - 1] = classes - 1
    check_batched(p, l, off, classes, f"classes-{classes}")


def test_batched_more_queues_than_planner_chunks():
    # 600,000 queues: more than the resident planner workgroups take in one
    # chunk of 256 each, so every planner workgroup plans several chunks
    rng = np.random.default_rng(30)
    sizes = rng.integers(0, 4, 600_000)
    sizes[::4999] = 300
    sizes[7::99991] = 5000
    p, l, off = fuzz_segments(sizes, seed=31, classes=3, max_len=2000)
    check_batched(p, l, off, 3, "many-chunks", forms=("async",))


def test_batched_many_long_queues():
    sizes = [16385 + 977 * k for k in range(24)] + [3, 0, 200000]
    p, l, off = fuzz_segments(sizes, seed=26, classes=8, max_len=100000)
    check_batched(p, l, off, 8, "many-long")


def test_batched_one_long_queue():
    p, l, off = fuzz_segments([300000], seed=27, classes=5, max_len=32768)
    check_batched(p, l, off, 5, "one-long")


@pytest.mark.parametrize("classes,max_len", [(2, 256), (4, 512), (3, 2**19), (5, 2**27),
                                             (200, 2**24)])
def test_batched_long_queue_key_widths(classes, max_len):
    # 9, 11, 21, 30 and 32 key bits: one pass, and splits of the key over two
    # to four passes that are not all of the widest digit
    sizes = [20000, 70000, 5, 300000]
    p, l, off = fuzz_segments(sizes, seed=40 + classes, classes=classes, max_len=max_len)
    check_batched(p, l, off, classes, f"long-keys-{classes}-{max_len}")


def test_batched_long_queue_tile_boundaries():
    # queues ending on and just past 8,192-request tile edges; 32 tiles (the
    # most whose digit offsets are one work item) and 33 (scanned in column
    # items of 16 digits); 600 tiles, past one 512-tile block of a column item
    t = 8192
    sizes = [2 * t, 2 * t + 1, 3 * t, 3 * t + 1, 32 * t, 32 * t + 1, 5, 600 * t - 3]
    p, l, off = fuzz_segments(sizes, seed=71, classes=6, max_len=50000)
    check_batched(p, l, off, 6, "long-tile-edges")


def test_batched_long_queue_key_and_index_beyond_64_bits():
    # 39 key bits (256 classes, lengths over the whole int32 range) and a
    # queue of more than 2^25 requests (26 index bits): the elements between
    # the passes keep the index apart from the key
    p, l, off = fuzz_segments([5, 2**25 + 3, 7], seed=61, classes=256, max_len=2**31 - 1)
    check_batched(p, l, off, 256, "long-keys-65-bits")


def test_batched_wide_keys_in_short_queues():
    # lengths over the whole int32 range: short queues whose key does not fit
    # a 32-bit element go to the 64-bit kernel, long ones to the segmented sort
    sizes = [5, 256, 300, 2000, 4096, 5000, 16384, 20000, 1]
    p, l, off = fuzz_segments(sizes, seed=28, classes=256, max_len=2**31 - 1)
    l[off[2]] = 0
    l[off[3]] = 2**31 - 1
    check_batched(p, l, off, 256, "wide-keys")


def test_batched_long_queue_totals_beyond_2_64():
    # one class, every length 2^31 - 1: the queue's total exceeds 2^64
    n = 200_000
    p = np.zeros(n + 10, np.uint8)
    l = np.full(n + 10, 2**31 - 1, np.int32)
    off = np.array([0, 10, n + 10], np.int64)
    want = c_oracle_batched(p, l, off, 1)
    assert want[2][2] > 2**64
    check_batched(p, l, off, 1, "long-128bit", want=want)


def test_batched_async_small():
    sizes = np.random.default_rng(1).integers(0, 700, 3000)
    p, l, off = fuzz_segments(sizes, seed=22, classes=4, max_len=400)
    check_batched(p, l, off, 4, "async-small")


def test_batched_single_class_count():
    p, l, off = fuzz_segments([5, 9, 2000], seed=23, classes=1, max_len=50)
    check_batched(p, l, off, 1, "one-class")


# ---- errors detected on the device ------------------------------------------------

@pytest.mark.parametrize("n", [100, 3000, 50000])
def test_negative_length_is_range_error(n):
    import paper_2506_12204_amd as ss
    p, l = fuzz_queue(n, seed=1)
    l[n // 2] = -5
    with pytest.raises(ss.SemschedRangeError):
        gpu_queue(p, l)


@pytest.mark.parametrize("sizes,where", [([10, 20, 30], 15), ([10, 300, 30], 200),
                                         ([10, 20000, 30], 12345), ([5, 5000, 7], 2000)])
def test_priority_out_of_range_in_batched(sizes, where):
    import paper_2506_12204_amd as ss
    p, l, off = fuzz_segments(sizes, seed=2, classes=4)
    p[where] = 4
    for blocking in (False, True):
        with pytest.raises(ss.SemschedRangeError):
            gpu_batched(p, l, off, 4, blocking=blocking)


def test_negative_length_in_long_batched_queue():
    import paper_2506_12204_amd as ss
    p, l, off = fuzz_segments([10, 20000, 30], seed=5, classes=4)
    l[9000] = -1
    for blocking in (False, True):
        with pytest.raises(ss.SemschedRangeError):
            gpu_batched(p, l, off, 4, blocking=blocking)


@pytest.mark.parametrize("sizes,where", [([10, 20, 30], 15), ([10, 300, 30], 200),
                                         ([5, 5000, 7], 2000)])
@pytest.mark.parametrize("bad_len", [-1, -2**31])
def test_negative_length_in_batched_queue(sizes, where, bad_len):
    # one queue of each size class below the segmented sort (one wave,
    # 256-thread and 1024-thread workgroups)
    import paper_2506_12204_amd as ss
    p, l, off = fuzz_segments(sizes, seed=7, classes=4)
    l[where] = bad_len
    for blocking in (False, True):
        with pytest.raises(ss.SemschedRangeError):
            gpu_batched(p, l, off, 4, blocking=blocking)


def test_bad_offsets():
    import paper_2506_12204_amd as ss
    p, l, off = fuzz_segments([10, 20, 30], seed=3, classes=4)
    bad = off.copy()
    bad[2] = 5  # decreasing
    for blocking in (False, True):
        with pytest.raises(ss.SemschedError):
            gpu_batched(p, l, bad, 4, blocking=blocking)
    bad = off.copy()
    bad[0] = 1  # not starting at 0
    for blocking in (False, True):
        with pytest.raises(ss.SemschedError):
            gpu_batched(p, l, bad, 4, blocking=blocking)


def test_long_queue_without_workspace_room():
    import paper_2506_12204_amd as ss
    p, l, off = fuzz_segments([10, 20000, 30], seed=6, classes=4)
    with pytest.raises(ss.SemschedError) as e:
        gpu_batched(p, l, off, 4, long_requests=0)
    assert e.value.code == ss.SEM_EINVAL
    with pytest.raises(ss.SemschedError):
        gpu_batched(p, l, off, 4, long_requests=15000)
    # exactly enough room
    check_batched(p, l, off, 4, "exact-room", forms=("async",))
    assert_same(gpu_batched(p, l, off, 4, long_requests=20000),
                c_oracle_batched(p, l, off, 4), "exact-room")


def test_after_error_next_call_is_clean():
    p, l = fuzz_queue(30000, seed=4)
    good = (p.copy(), l.copy())
    l[7] = -1
    with pytest.raises(Exception):
        gpu_queue(p, l)
    check_queue(*good, "after-error")


def test_middle_pass_barrier_give_up(monkeypatch):
    # SEMSCHED_MID_SPIN=0 makes the grid barrier of the middle passes give up
    # at its first wait, as it would if its workgroups were not all resident.
    # The asynchronous call then reports SEM_EDEVICE (and every kernel of the
    # schedule exits); the blocking call runs the schedule again with the
    # middle passes as separate launches and returns the right result; the
    # next call after either is clean.
    import torch
    import paper_2506_12204_amd as ss
    rng = np.random.default_rng(17)
    n = 1_500_000
    p = rng.integers(0, 256, n).astype(np.uint8)  # widest keys: three middle passes
    l = rng.integers(0, 2**31 - 1, n, dtype=np.int64).astype(np.int32)
    want = c_oracle_queue(p, l)
    monkeypatch.setenv("SEMSCHED_MID_SPIN", "0")
    say("[gpu] middle-pass barrier give-up (async)")
    with pytest.raises(ss.SemschedError) as e:
        gpu_queue(p, l)
    assert e.value.code == ss.SEM_EDEVICE
    say("[gpu] middle-pass barrier give-up (blocking, separate launches)")
    tp, tl = to_gpu(p, l)
    order = torch.empty(n, dtype=torch.int32, device="cuda")
    wait = torch.empty(n, dtype=torch.int64, device="cuda")
    totals = torch.empty((1 + ss.MAX_CLASSES, 2), dtype=torch.int64, device="cuda")
    torch.cuda.synchronize()
    rc = ss.lib.sem_schedule(ss._ptr(tp), ss._ptr(tl), n, ss._ptr(order), ss._ptr(wait),
                             ss._ptr(totals))
    assert rc == ss.SEM_OK, ss.strerror(rc)
    assert_same((order.cpu().numpy(), wait.cpu().numpy(), ss.totals_to_ints(totals)), want,
                "give-up-blocking")
    monkeypatch.delenv("SEMSCHED_MID_SPIN")
    check_queue(p, l, "after-give-up")
