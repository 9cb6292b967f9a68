"""Pins of the cost-model oracle (Section 3.4).

* Eq. 4 against the token-by-token sum it abbreviates: decoding tokens
  i = n+1 .. n+m at gamma1 * i + gamma2 each (a plain loop, no closed form).
* The remaining time of a request part-way through decoding against the same
  loop over the tokens still ahead, plus the prefill only before the first
  token.
* Eq. 5's integer minimiser against brute force over every number of saved
  tokens (largest among equal costs).
* Eq. 3 (read as: keep the prefill cache when reloading is cheaper than
  recomputing): properties instead of the formula retyped -- no cache is
  kept for an empty prompt, the decision is monotone in the prompt length
  (recomputation grows quadratically, reloading linearly), with beta = 0
  every non-empty prompt with a non-zero prefill cost keeps, and with
  alpha1 = 0 the decision is alpha2 > beta for every length.
* Fixed-point service times: unit constants give exact token counts,
  fractions floor, huge values saturate at 2^31 - 1.
* The C oracle against the Python one.
"""

import random

import numpy as np
import pytest

from oracle import (CostModel, OracleRangeError, c_oracle_evict_plan, c_oracle_service_times,
                    evict_plan, keep_prefill_cache, schedule_cost, schedule_queue,
                    service_times, tokens_to_save)
from oracle.cost_oracle import ONE, SERVICE_MAX, decode_cost, eviction_cost, remaining_cost


def rand_model(rng, scale=1 << 40):
    return CostModel(*(rng.randrange(scale) for _ in range(5)))


def test_eq4_is_the_token_sum():
    rng = random.Random(1)
    for _ in range(200):
        cm = rand_model(rng)
        n, m = rng.randrange(0, 300), rng.randrange(0, 300)
        want = 0
        for i in range(n + 1, n + m + 1):
            want += cm.gamma1 * i + cm.gamma2
        assert decode_cost(cm, n, m) == want


def test_remaining_cost_counts_the_tokens_ahead():
    rng = random.Random(2)
    for _ in range(300):
        cm = rand_model(rng)
        n, m, d = rng.randrange(0, 200), rng.randrange(0, 200), rng.randrange(0, 250)
        want = 0
        for i in range(n + d + 1, n + m + 1):  # empty once d >= m
            want += cm.gamma1 * i + cm.gamma2
        if d == 0:
            want += cm.alpha1 * n * n + cm.alpha2 * n
        assert remaining_cost(cm, n, m, d) == want


def test_eq5_minimiser_by_brute_force():
    rng = random.Random(3)
    for _ in range(400):
        cm = rand_model(rng, 1 << 20)
        n, mp = rng.randrange(0, 100), rng.randrange(0, 80)
        costs = [eviction_cost(cm, n, mp, x) for x in range(mp + 1)]
        best = min(costs)
        want = max(x for x in range(mp + 1) if costs[x] == best)
        assert tokens_to_save(cm, n, mp) == want


def test_eq5_extremes():
    # free reloading: save everything; reloading dearer than any recompute step: save nothing
    cm = CostModel(alpha1=1, alpha2=1, beta=0, gamma1=5, gamma2=7)
    assert tokens_to_save(cm, 10, 50) == 50
    cm = CostModel(alpha1=1, alpha2=1, beta=10**9, gamma1=5, gamma2=7)
    assert tokens_to_save(cm, 10, 50) == 0
    assert tokens_to_save(cm, 10, 0) == 0


def test_eq3_properties():
    rng = random.Random(4)
    for _ in range(100):
        cm = rand_model(rng, 1 << 24)
        assert not keep_prefill_cache(cm, 0)
        seen_keep = False
        for n in range(0, 400):
            k = keep_prefill_cache(cm, n)
            assert not (seen_keep and not k), "keep must be monotone in n"
            seen_keep |= k
    cm = CostModel(alpha1=3, alpha2=0, beta=0, gamma1=1, gamma2=1)
    assert all(keep_prefill_cache(cm, n) for n in range(1, 100))
    for a2, b in [(5, 3), (3, 5), (4, 4)]:
        cm = CostModel(alpha1=0, alpha2=a2, beta=b, gamma1=1, gamma2=1)
        assert all(keep_prefill_cache(cm, n) == (a2 > b) for n in range(1, 50))


def test_fixed_point_service_times():
    one_per_token = CostModel(alpha1=0, alpha2=0, beta=0, gamma1=0, gamma2=ONE)
    assert service_times([5, 0, 7], [10, 3, 0], [0, 1, 0], one_per_token) == [10, 2, 0]
    half = CostModel(alpha1=0, alpha2=ONE // 2, beta=0, gamma1=0, gamma2=0)
    assert service_times([3, 4], [0, 0], None, half) == [1, 2]  # 1.5 floors to 1
    huge = CostModel(alpha1=(1 << 64) - 1, alpha2=0, beta=0, gamma1=0, gamma2=0)
    assert service_times([1 << 20], [0], None, huge) == [SERVICE_MAX]
    with pytest.raises(OracleRangeError):
        service_times([1], [-1], None, one_per_token)


def test_paper_constants_order_long_prompts_later():
    # A5000, Qwen1.5-7B (appendix): decode 2.117e-6 / 2.727e-2, prefill 1.859e-9 /
    # 2.175e-4, cache 3e-4 per token; times in microseconds
    cm = CostModel.from_float(alpha1=1.859e-9, alpha2=2.175e-4, beta=3e-4,
                              gamma1=2.117e-6, gamma2=2.727e-2)
    s = service_times([100, 1000, 100], [50, 50, 500], None, cm)
    assert s[0] < s[1] < s[2]
    # about 50 tokens * 27 ms each, plus the small prefill
    assert 1.3e6 < s[0] < 1.45e6


def test_schedule_cost_is_the_schedule_of_the_service_times():
    rng = np.random.default_rng(5)
    n = 3000
    p = rng.integers(0, 5, n).astype(np.uint8)
    prompt = rng.integers(0, 4000, n).astype(np.int32)
    out = rng.integers(0, 2000, n).astype(np.int32)
    dec = np.where(rng.random(n) < 0.3, rng.integers(0, 2000, n), 0).astype(np.int32)
    cm = CostModel.from_float(1.466e-9, 1.052e-4, 1e-4, 5.913e-9, 1.196e-2)
    o, w, t, s = schedule_cost(p, prompt, out, dec, cm)
    assert (o, w, t) == schedule_queue(p, s)


@pytest.mark.parametrize("seed", range(3))
def test_c_oracle_matches_python(seed):
    rng = np.random.default_rng(seed)
    n = 5000
    prompt = rng.integers(0, 1 << 16, n).astype(np.int32)
    out = rng.integers(0, 1 << 16, n).astype(np.int32)
    dec = np.where(rng.random(n) < 0.5, rng.integers(0, 1 << 16, n), 0).astype(np.int32)
    r = random.Random(seed)
    for cm in (rand_model(r, 1 << 63), CostModel.from_float(1.859e-9, 2.175e-4, 3e-4,
                                                            2.117e-6, 2.727e-2)):
        assert c_oracle_service_times(prompt, out, dec, cm).tolist() == \
            service_times(prompt, out, dec, cm)
        assert c_oracle_service_times(prompt, out, None, cm).tolist() == \
            service_times(prompt, out, None, cm)
        small = rng.integers(0, 300, n).astype(np.int32)
        keep, save = c_oracle_evict_plan(prompt, small, cm)
        k2, s2 = evict_plan(prompt, small, cm)
        assert keep.tolist() == k2 and save.tolist() == s2
    with pytest.raises(OracleRangeError):
        c_oracle_service_times(np.array([-1], np.int32), np.array([1], np.int32), None, cm)
