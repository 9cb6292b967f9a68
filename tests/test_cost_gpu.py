"""GPU parity of the cost model (sem_service_times, sem_evict_plan,
sem_schedule_cost) against the C oracle (oracle.c, pinned to the
pure-Python definitions in tests/test_oracle_cost.py). All integer:
bit-exact comparisons.
"""

import random

import numpy as np
import pytest

from oracle import (CostModel, c_oracle_evict_plan, c_oracle_queue, c_oracle_service_times)
from tests._lib import assert_same, ensure_built, gpu_available
from workloads import cost_tokens, generate

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]

# the paper's appendix constants (seconds), in microseconds
A100_4B = CostModel.from_float(1.466e-2, 1.052e-4, 1e-4, 5.913e-9, 1.196e-2)
A5000_7B = CostModel.from_float(1.859e-9, 2.175e-4, 3e-4, 2.117e-6, 2.727e-2)
MAX64 = (1 << 64) - 1


@pytest.fixture(scope="module", autouse=True)
def _built():
    ensure_built()


def dev(a, dt):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=dt)).cuda()


def models():
    r = random.Random(7)
    yield "a100-4b", A100_4B
    yield "a5000-7b", A5000_7B
    yield "random", CostModel(*(r.randrange(1 << 40) for _ in range(5)))
    yield "extreme", CostModel(MAX64, MAX64, MAX64, MAX64, MAX64)
    yield "zero", CostModel(0, 0, 0, 0, 0)
    yield "no-gamma1", CostModel(5, 7, 1 << 36, 0, 3)
    yield "tiny-gamma1", CostModel(1, 1, MAX64, 1, 0)


@pytest.mark.parametrize("n", [1, 7, 256, 100003, 1 << 20])
def test_service_times(n):
    import paper_2506_12204_amd as ss
    rng = np.random.default_rng(n)
    prompt = rng.integers(0, 1 << 31, n).astype(np.int32)
    prompt[: n // 2] = rng.integers(0, 5000, n // 2)
    output = rng.integers(0, 1 << 31, n).astype(np.int32)
    output[: n // 2] = rng.integers(0, 5000, n // 2)
    decoded = np.where(rng.random(n) < 0.4, rng.integers(0, 1 << 31, n), 0).astype(np.int32)
    for label, cm in models():
        print(f"[gpu] service times n={n} model={label}", flush=True)
        for dec in (decoded, None):
            want = c_oracle_service_times(prompt, output, dec, cm)
            got = ss.service_times(dev(prompt, np.int32), dev(output, np.int32),
                                   None if dec is None else dev(dec, np.int32), cm)
            bad = np.flatnonzero(got.cpu().numpy() != want)
            assert bad.size == 0, f"{label}: differs at {bad[:8]}"


@pytest.mark.parametrize("n", [1, 5000, 200003])
def test_evict_plan(n):
    import paper_2506_12204_amd as ss
    rng = np.random.default_rng(n + 1)
    prompt = rng.integers(0, 1 << 20, n).astype(np.int32)
    prompt[: n // 3] = rng.integers(0, 50, n // 3)
    decoded = rng.integers(0, 2000, n).astype(np.int32)
    for label, cm in models():
        print(f"[gpu] evict plan n={n} model={label}", flush=True)
        keep, save = c_oracle_evict_plan(prompt, decoded, cm)
        gk, gs = ss.evict_plan(dev(prompt, np.int32), dev(decoded, np.int32), cm)
        assert np.array_equal(gk.cpu().numpy(), keep), label
        assert np.array_equal(gs.cpu().numpy(), save), label


@pytest.mark.parametrize("scale", [1 / 4096, 1 / 64, 1.0])
def test_schedule_cost_c3(scale):
    import paper_2506_12204_amd as ss
    w = generate("c3", scale=scale)
    prompt, decoded = cost_tokens(w.length)
    print(f"[gpu] schedule_cost n={w.n}", flush=True)
    s = c_oracle_service_times(prompt, w.length, decoded, A100_4B)
    want = c_oracle_queue(w.priority, s)
    o, wt, t, got_s = ss.schedule_cost(dev(w.priority, np.uint8), dev(prompt, np.int32),
                                       dev(w.length, np.int32), dev(decoded, np.int32), A100_4B)
    assert np.array_equal(got_s.cpu().numpy(), s)
    assert_same((o.cpu().numpy(), wt.cpu().numpy(), t), want, "schedule_cost")


def test_schedule_cost_small_and_empty():
    import torch

    import paper_2506_12204_amd as ss
    for n in (0, 1, 3, 16384, 16385):
        rng = np.random.default_rng(n)
        p = rng.integers(0, 5, n).astype(np.uint8)
        prompt = rng.integers(0, 3000, n).astype(np.int32)
        out = rng.integers(0, 3000, n).astype(np.int32)
        s = c_oracle_service_times(prompt, out, None, A5000_7B)
        want = c_oracle_queue(p, s)
        o, wt, t, gs = ss.schedule_cost(dev(p, np.uint8), dev(prompt, np.int32),
                                        dev(out, np.int32), None, A5000_7B)
        assert np.array_equal(gs.cpu().numpy(), s)
        assert_same((o.cpu().numpy(), wt.cpu().numpy(), t), want, f"n={n}")
    bad = dev(np.array([3, -1, 2], np.int32), np.int32)
    ok = dev(np.array([1, 1, 1], np.int32), np.int32)
    with pytest.raises(ss.SemschedRangeError):
        ss.service_times(ok, bad, None, A100_4B)
    with pytest.raises(ss.SemschedRangeError):
        ss.evict_plan(bad, ok, A100_4B)
    with pytest.raises(ss.SemschedRangeError):
        ss.schedule_cost(dev(np.zeros(3, np.uint8), np.uint8), bad, ok, None, A100_4B)
    # the error does not stick to the next call
    ss.schedule_cost(dev(np.zeros(3, np.uint8), np.uint8), ok, ok, None, A100_4B)
