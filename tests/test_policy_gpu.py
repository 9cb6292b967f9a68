"""GPU parity of the comparison policies (sem_schedule_policy*).

FCFS, SJF and HPJF schedules from the HIP path are compared element by
element with the C oracle's (``oracle_schedule_policy``, itself pinned in
tests/test_oracle_policies.py): order, waits and the 257 exact totals.
Everything is integer, so the comparison is bit-exact.
"""

import numpy as np
import pytest

from oracle import POLICY_FCFS, POLICY_HPJF, POLICY_SEMANTIC, POLICY_SJF, c_oracle_policy
from tests._lib import assert_same, ensure_built, gpu_available
from workloads import fuzz_queue, generate

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]

POLICIES = [POLICY_FCFS, POLICY_SJF, POLICY_HPJF]
NAMES = {POLICY_SEMANTIC: "semantic", POLICY_FCFS: "fcfs", POLICY_SJF: "sjf",
         POLICY_HPJF: "hpjf"}


@pytest.fixture(scope="module", autouse=True)
def _built():
    ensure_built()


def gpu_policy(p, l, policy):
    import torch

    import paper_2506_12204_amd as ss
    dev = torch.device("cuda")
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a, dtype=dt)).to(dev)
    order, wait, totals = ss.schedule_policy(t(p, np.uint8), t(l, np.int32), policy)
    return order.cpu().numpy(), wait.cpu().numpy(), totals


def check(p, l, policy, label):
    print(f"[gpu] policy {NAMES[policy]} {label}: n={len(p)}", flush=True)
    want = c_oracle_policy(p, l, policy)
    assert_same(gpu_policy(p, l, policy), want, f"{NAMES[policy]} {label}")


@pytest.mark.parametrize("policy", POLICIES)
@pytest.mark.parametrize("n", [1, 5, 63, 64, 65, 4095, 4096, 4097, 16385, 100003])
def test_policy_sizes(policy, n):
    p, l = fuzz_queue(n, seed=n + 17 * policy, classes=6, max_len=5000, tie_frac=0.2)
    check(p, l, policy, f"n={n}")


@pytest.mark.parametrize("policy", POLICIES)
@pytest.mark.parametrize("classes", [1, 64, 65, 256])
def test_policy_class_counts(policy, classes):
    # 65 and more ranks take the four-set lane tables
    p, l = fuzz_queue(30000, seed=classes, classes=classes, max_len=2000, tie_frac=0.1)
    check(p, l, policy, f"classes={classes}")


@pytest.mark.parametrize("policy", POLICIES)
def test_policy_zero_and_max_lengths(policy):
    rng = np.random.default_rng(9)
    n = 70000
    p = rng.integers(0, 5, n).astype(np.uint8)
    l = np.where(rng.random(n) < 0.5, 0, 2**31 - 1).astype(np.int32)
    check(p, l, policy, "lengths 0 / 2^31-1")


@pytest.mark.parametrize("policy", POLICIES)
def test_policy_workloads(policy):
    w = generate("c2")
    check(w.priority, w.length, policy, "c2")
    w = generate("c1")
    check(w.priority, w.length, policy, "c1")


@pytest.mark.parametrize("policy", POLICIES)
def test_policy_full_size_c3(policy):
    w = generate("c3")
    check(w.priority, w.length, policy, "c3")


def test_policy_empty_and_errors():
    import torch

    import paper_2506_12204_amd as ss
    dev = torch.device("cuda")
    e8 = torch.zeros(0, dtype=torch.uint8, device=dev)
    e32 = torch.zeros(0, dtype=torch.int32, device=dev)
    for policy in POLICIES + [POLICY_SEMANTIC]:
        o, w, t = ss.schedule_policy(e8, e32, policy)
        assert o.numel() == 0 and t == [0] * 257
        p = torch.tensor([0, 1, 2], dtype=torch.uint8, device=dev)
        l = torch.tensor([4, -1, 3], dtype=torch.int32, device=dev)
        with pytest.raises(ss.SemschedRangeError):
            ss.schedule_policy(p, l, policy)
    with pytest.raises(ss.SemschedError):
        ss.PolicyScheduler(10, 9, dev)


def test_semantic_policy_is_sem_schedule():
    p, l = fuzz_queue(50000, seed=3, classes=5, max_len=900, tie_frac=0.2)
    check(p, l, POLICY_SEMANTIC, "semantic")


@pytest.mark.parametrize("classes,max_len", [(4, 2**18 - 1), (5, 2**18 - 1), (8, 2**17 - 1),
                                             (9, 2**17 - 1), (256, 4095), (256, 4096)])
def test_sjf_carried_ranks_either_side_of_the_fit(classes, max_len):
    # A long SJF queue in the compact layout carries the ranks through the
    # sort when final-digit bits + rank bits fit above the 22 id bits
    # (4 ranks with 256 final digits fit, 5 do not; 8 ranks with 128 digits
    # fit, 9 do not; 256 ranks fit with 4 digits, lengths below 4096, not
    # with 5); otherwise
    # the class sums gather every position's rank. Both sides must agree
    # with the oracle.
    rng = np.random.default_rng(classes * 7 + max_len % 97)
    n = 70000
    p = rng.integers(0, classes, n).astype(np.uint8)
    p[0] = classes - 1  # the largest rank is present
    l = rng.integers(0, max_len + 1, n).astype(np.int32)
    l[1], l[2] = 0, max_len  # the full length range is present
    check(p, l, POLICY_SJF, f"classes={classes} max_len={max_len}")


def test_sjf_carried_ranks_window_in_global_memory():
    # As the queue test of the same name: 99 % of the lengths are multiples
    # of 1024, so the last blocks span more sub-bucket starts than the LDS
    # window holds; the final pass with carried ranks then takes its
    # global-window kernel.
    rng = np.random.default_rng(32)
    n = 12_000_000
    p = rng.integers(0, 4, n).astype(np.uint8)
    l = (rng.integers(1, 8, n) * 1024).astype(np.int32)
    sprinkle = rng.random(n) < 0.01
    l[sprinkle] = rng.integers(1, 8192, int(sprinkle.sum()))
    check(p, l, POLICY_SJF, "window-global")


@pytest.mark.parametrize("policy", POLICIES)
def test_policy_unaligned_inputs(policy):
    # inputs that start one element into their allocations: lengths not
    # 16-byte aligned, ranks not 4-byte aligned (the range kernels then load
    # one element per lane instead of four)
    import torch

    import paper_2506_12204_amd as ss
    p, l = fuzz_queue(100_001, seed=41 + policy, classes=6, max_len=5000, tie_frac=0.2)
    dev = torch.device("cuda")
    tp = torch.from_numpy(np.concatenate([[0], p]).astype(np.uint8)).to(dev)[1:]
    tl = torch.from_numpy(np.concatenate([[0], l]).astype(np.int32)).to(dev)[1:]
    assert tl.data_ptr() % 16 != 0 and tp.data_ptr() % 4 != 0
    print(f"[gpu] policy {NAMES[policy]} unaligned: n={len(p)}", flush=True)
    order, wait, totals = ss.schedule_policy(tp, tl, policy)
    assert_same((order.cpu().numpy(), wait.cpu().numpy(), totals),
                c_oracle_policy(p, l, policy), f"{NAMES[policy]} unaligned")
