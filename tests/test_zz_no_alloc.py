"""The allocation-free entry point (sem_schedule_static) against the
workspace-taking one it shares its kernels with (sem_schedule_async), call by
call, through the C ABI: the static scratch keeps each call's contents, so
consecutive calls of decreasing size (and one after a device-detected error)
must each give exactly the other entry point's schedule."""

import numpy as np
import pytest

from tests._lib import ensure_built, gpu_available

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ss():
    ensure_built()
    if not gpu_available():
        pytest.skip("no GPU")
    import paper_2506_12204_amd as mod
    return mod


def _inputs(n, seed, classes=5, max_len=32768):
    from workloads import fuzz_queue
    return fuzz_queue(n, seed=seed, classes=classes, max_len=max_len, tie_frac=0.2)


def _both(ss, p, l):
    import torch
    tp = torch.from_numpy(p.astype(np.uint8)).cuda()
    tl = torch.from_numpy(l.astype(np.int32)).cuda()
    order, wait, totals, status = ss.schedule_static(tp, tl)
    torch.cuda.synchronize()
    ref = ss.Scheduler(p.size, tp.device)
    ref.run(tp, tl)
    ref.check()
    return (order.cpu().numpy(), wait.cpu().numpy(), ss.totals_to_ints(totals),
            int(status.item())), (ref.order.cpu().numpy(), ref.wait.cpu().numpy(),
                                  ss.totals_to_ints(ref.totals))


def _assert_equal(got, want, label):
    go, gw, gt, st = got
    wo, ww, wt = want
    assert st == 0, f"{label}: status {st}"
    assert np.array_equal(go, wo), f"{label}: order differs"
    assert np.array_equal(gw, ww), f"{label}: wait differs"
    assert gt == wt, f"{label}: totals differ"


def test_static_matches_async_on_shrinking_calls(ss):
    # largest size first, then smaller ones on the global path, then the LDS path
    sizes = [ss.STATIC_MAX_N, 300_001, 16_385, 3_000, 0]
    for i, n in enumerate(sizes):
        p, l = _inputs(n, seed=100 + i)
        print(f"[static] call {i}: n={n}", flush=True)
        got, want = _both(ss, p, l)
        _assert_equal(got, want, f"n={n}")


def test_static_range_error_then_clean_call(ss):
    import torch
    p, l = _inputs(50_000, seed=7)
    l = l.copy()
    l[12_345] = -3
    tp = torch.from_numpy(p.astype(np.uint8)).cuda()
    tl = torch.from_numpy(l.astype(np.int32)).cuda()
    _, _, _, status = ss.schedule_static(tp, tl)
    torch.cuda.synchronize()
    assert int(status.item()) == ss.SEM_ERANGE
    # the next (smaller) call starts from a clean scratch
    p2, l2 = _inputs(40_000, seed=8)
    got, want = _both(ss, p2, l2)
    _assert_equal(got, want, "after a range error")


def test_static_rejects_oversize(ss):
    import torch
    n = ss.STATIC_MAX_N + 1
    tp = torch.zeros(n, dtype=torch.uint8, device="cuda")
    tl = torch.ones(n, dtype=torch.int32, device="cuda")
    with pytest.raises(ss.SemschedError) as e:
        ss.schedule_static(tp, tl)
    assert e.value.code == ss.SEM_ENOMEM
