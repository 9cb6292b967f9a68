"""CPU oracle of the cost model of Section 3.4 (pure Python, exact integers).

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it. It shares no code with the HIP
library.

The paper models the time of a request's stages with per-model constants:

* prefill of a prompt of n tokens: alpha1 * n^2 + alpha2 * n;
* reloading n tokens of offloaded KV cache: beta * n;
* decoding m tokens after a prompt of n (Eq. 4, the sum over tokens
  i = n+1 .. n+m of gamma1 * i + gamma2):
  gamma1 * (m^2/2 + n*m + m/2) + gamma2 * m.

Readings (the paper leaves these open or states them inconsistently):

* Fixed point. The constants are non-negative Q32.32 numbers (integers in
  units of 2^-32 of the chosen time unit per token, or per token^2 for
  alpha1); all arithmetic is exact on integers; a service time is the
  floor of the exact cost divided by 2^32, saturated at 2^31 - 1.
* Eq. 4 is taken as printed (token i costs gamma1 * i + gamma2). The
  sentence before it charges the m'-th token gamma1 * (n + m' - 1) + gamma2,
  which sums to gamma1 * m less; the printed sum is the paper's definition
  of the decoding cost, so it is the one used.
* Remaining time. A request that has decoded d of its m predicted tokens
  has gamma-cost for tokens n+d+1 .. n+m still ahead (none if d >= m) and
  its prefill still ahead only if d = 0.
* Eq. 3 direction. Keeping (offloading and reloading) the prefill cache of
  n tokens costs beta * n, recomputing it alpha1 * n^2 + alpha2 * n; the
  cache is kept when reloading is strictly cheaper. (As printed, Eq. 3
  says the opposite, which contradicts its own explanation.)
* Tokens to save after a decode-stage eviction (Eq. 5). With x of the m'
  decoded tokens saved and y = m' - x recomputed, the cost is
  beta * x + gamma1 * (y^2/2 + n*y + y/2) + gamma2 * y (Eq. 5, reading its
  m_* as m'_*). It is convex in y; the oracle takes the integer minimiser
  over 0 <= x <= m', and the largest x among equal costs. Eq. 6's closed
  form does not follow from Eq. 5 and is not used.

Pins (tests/test_oracle_cost.py): the token-by-token sums behind Eq. 4,
brute-force minimisation of Eq. 5 over every x, direct comparison for
Eq. 3, and the schedule with these service times against ``schedule_queue``.
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import List, Sequence, Tuple

from .semsched_oracle import OracleRangeError, schedule_queue

FRAC_BITS = 32
ONE = 1 << FRAC_BITS
SERVICE_MAX = (1 << 31) - 1


@dataclass(frozen=True)
class CostModel:
    """Q32.32 constants (integers, time units * 2^32 per token or token^2)."""
    alpha1: int
    alpha2: int
    beta: int
    gamma1: int
    gamma2: int

    @staticmethod
    def from_float(alpha1, alpha2, beta, gamma1, gamma2, unit=1e-6):
        """Constants given in seconds (as the paper's appendix lists them),
        converted to Q32.32 multiples of ``unit`` seconds (rounded to nearest)."""
        q = lambda v: int(round(v / unit * ONE))
        return CostModel(q(alpha1), q(alpha2), q(beta), q(gamma1), q(gamma2))

    def check(self):
        for v in (self.alpha1, self.alpha2, self.beta, self.gamma1, self.gamma2):
            if not 0 <= v < 1 << 64:
                raise ValueError("cost constants are unsigned 64-bit Q32.32")


def prefill_cost(cm: CostModel, n: int) -> int:
    """alpha1 * n^2 + alpha2 * n (Section 3.4), Q32.32."""
    return cm.alpha1 * n * n + cm.alpha2 * n


def decode_cost(cm: CostModel, n: int, m: int) -> int:
    """Eq. 4: gamma1 * (m^2/2 + n*m + m/2) + gamma2 * m, Q32.32 (exact:
    m^2 + m is even)."""
    return cm.gamma1 * ((m * m + m) // 2 + n * m) + cm.gamma2 * m


def remaining_cost(cm: CostModel, n: int, m: int, d: int) -> int:
    """Cost still ahead of a request with prompt n that has decoded d of its
    m predicted tokens: decoding tokens n+d+1 .. n+m (Eq. 4 shifted by d),
    plus its prefill when d = 0."""
    r = max(m - d, 0)
    c = decode_cost(cm, n + d, r)
    if d == 0:
        c += prefill_cost(cm, n)
    return c


def service_times(prompt: Sequence[int], output: Sequence[int],
                  decoded: Sequence[int] | None, cm: CostModel) -> List[int]:
    """Remaining computation time of every request in the time unit: the
    floor of the exact cost / 2^32, saturated at 2^31 - 1."""
    cm.check()
    n = len(prompt)
    if len(output) != n or (decoded is not None and len(decoded) != n):
        raise ValueError("arrays differ in size")
    out = []
    for i in range(n):
        a, m = int(prompt[i]), int(output[i])
        d = 0 if decoded is None else int(decoded[i])
        if a < 0 or m < 0 or d < 0:
            raise OracleRangeError(f"negative token count at {i}")
        out.append(min(remaining_cost(cm, a, m, d) >> FRAC_BITS, SERVICE_MAX))
    return out


def keep_prefill_cache(cm: CostModel, n: int) -> bool:
    """Eq. 3 read the intended way: keep the cache of n prefill tokens when
    reloading it (beta * n) is strictly cheaper than recomputing it."""
    return cm.beta * n < prefill_cost(cm, n)


def eviction_cost(cm: CostModel, n: int, mp: int, x: int) -> int:
    """Eq. 5: beta * x + gamma1 * (y^2/2 + n*y + y/2) + gamma2 * y with
    y = mp - x recomputed tokens, Q32.32 (exact: y^2 + y is even)."""
    y = mp - x
    return cm.beta * x + cm.gamma1 * ((y * y + y) // 2 + n * y) + cm.gamma2 * y


def tokens_to_save(cm: CostModel, n: int, mp: int) -> int:
    """Integer minimiser x in [0, mp] of Eq. 5; the largest x among ties.
    Cost(y + 1) - Cost(y) = gamma1 * (y + 1 + n) + gamma2 - beta grows with
    y, so the best y is the first one whose next step does not pay."""
    y = 0
    while y < mp and cm.gamma1 * (y + 1 + n) + cm.gamma2 < cm.beta:
        y += 1
    return mp - y


def evict_plan(prompt: Sequence[int], decoded: Sequence[int], cm: CostModel
               ) -> Tuple[List[int], List[int]]:
    """Per evicted request: 1 if its prefill cache is kept (Eq. 3, read as
    above), and how many of its decoded tokens' cache to save (Eq. 5)."""
    cm.check()
    keep, save = [], []
    for i in range(len(prompt)):
        a, d = int(prompt[i]), int(decoded[i])
        if a < 0 or d < 0:
            raise OracleRangeError(f"negative token count at {i}")
        keep.append(1 if keep_prefill_cache(cm, a) else 0)
        save.append(tokens_to_save(cm, a, d))
    return keep, save


def schedule_cost(priority: Sequence[int], prompt: Sequence[int], output: Sequence[int],
                  decoded: Sequence[int] | None, cm: CostModel):
    """The semantic schedule with the cost model's service times as f_t:
    (order, wait, totals, service times)."""
    s = service_times(prompt, output, decoded, cm)
    o, w, t = schedule_queue(priority, s)
    return o, w, t, s
