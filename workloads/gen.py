"""Generators for the five synthetic workloads and for fuzz queues.

The paper evaluates on an emergency-medical-services conversation set with
five ESI urgency levels (Section 3.1; Section 4) and on simulated arrival
spikes (Section 4.1). Neither the data nor the trained urgency/length
predictors are available, so these seeded generators stand in for them: each
request carries an urgency class (uint8, 0 = most urgent, the graded-poset
rank of Definition 1) and a predicted generation length in tokens (int32).

Recipes (numpy ``default_rng``; priorities drawn first, then lengths, then
duplicate masks):

* ``c1``  n = 1,000, seed 0. p ~ U{0..3}; len = clip(rint(lognormal(5, 1)), 1, 4096).
* ``c2``  n = 2^20, seed 1. 10 classes with Zipf(1.2) frequencies, class 0
  rarest (weight of class c proportional to (10 - c)^-1.2);
  len = clip(rint(lognormal(5.5, 1.2)), 1, 8192); 25 % of requests copy the
  length of a uniformly drawn request of the same class (drawn from the
  pre-copy lengths), which plants many exact (class, length) ties.
* ``c3``  n = 2^26, seed 2. p ~ U{0..4}; len ~ U{1..32768}.
* ``c4``  65,536 queues x 256 requests, seed 3. p ~ U{0..3};
  len = clip(rint(lognormal(5, 1)), 1, 4096).
* ``c5``  16,384 queues with sizes ~ U{1..4096}, seed 4. 70 % of requests in
  the least urgent class 7, the rest uniform over 0..6;
  len = clip(floor(pareto(1.5) + 1), 1, 65536) (numpy's pareto is the Lomax
  form, so +1 gives a classical Pareto with x_min = 1); 30 % of lengths copy
  the left neighbour in the same queue from the pre-copy array (a queue's
  first request copies its right neighbour; queues of size 1 are untouched).

Token counts for the cost model of Section 3.4 (``cost_tokens``), seed 5
unless given: prompt = U{1..4096}; output = the workload's predicted lengths;
25 % of the requests are part-way through decoding with decoded ~
U{1..output}, the rest have decoded nothing (decoded = 0).
"""

from __future__ import annotations

import hashlib
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

__all__ = [
    "CONFIGS",
    "Workload",
    "generate",
    "fuzz_queue",
    "fuzz_segments",
    "sha256_arrays",
    "workload_sha256",
    "cost_tokens",
]


@dataclass
class Workload:
    """One synthetic scheduling input.

    ``offsets`` is None for a single queue; otherwise it holds S+1 int64
    boundaries of S independent queues laid out back to back.
    """

    name: str
    priority: np.ndarray  # uint8 [N]
    length: np.ndarray  # int32 [N]
    offsets: Optional[np.ndarray] = None  # int64 [S+1] or None
    num_classes: int = 256
    meta: dict = field(default_factory=dict)

    @property
    def n(self) -> int:
        return int(self.priority.shape[0])

    @property
    def num_segments(self) -> int:
        return 1 if self.offsets is None else int(self.offsets.shape[0] - 1)


CONFIGS = {
    "c1": dict(kind="queue", n=1000, seed=0, classes=4),
    "c2": dict(kind="queue", n=1 << 20, seed=1, classes=10),
    "c3": dict(kind="queue", n=1 << 26, seed=2, classes=5),
    "c4": dict(kind="batched", segments=65536, seg_size=256, seed=3, classes=4),
    "c5": dict(kind="batched", segments=16384, max_seg=4096, seed=4, classes=8),
}


def _lognormal_len(rng, mu, sigma, n, hi):
    x = np.rint(rng.lognormal(mu, sigma, n))
    return np.clip(x, 1, hi).astype(np.int32)


def _gen_c1(rng, n):
    p = rng.integers(0, 4, n, dtype=np.uint8)
    ln = _lognormal_len(rng, 5.0, 1.0, n, 4096)
    return p, ln, None


def _gen_c2(rng, n):
    c = np.arange(10, dtype=np.float64)
    w = (10.0 - c) ** -1.2
    w /= w.sum()
    p = rng.choice(10, n, p=w).astype(np.uint8)
    ln = _lognormal_len(rng, 5.5, 1.2, n, 8192)
    mask = rng.random(n) < 0.25
    src_len = ln.copy()
    for cls in range(10):
        members = np.flatnonzero(p == cls)
        if members.size == 0:
            continue
        hit = members[mask[members]]
        pick = rng.integers(0, members.size, hit.size)
        ln[hit] = src_len[members[pick]]
    return p, ln, None


def _gen_c3(rng, n):
    p = rng.integers(0, 5, n, dtype=np.uint8)
    ln = rng.integers(1, 32769, n, dtype=np.int32)
    return p, ln, None


def _gen_c4(rng, segments, seg_size):
    total = segments * seg_size
    offsets = np.arange(segments + 1, dtype=np.int64) * seg_size
    p = rng.integers(0, 4, total, dtype=np.uint8)
    ln = _lognormal_len(rng, 5.0, 1.0, total, 4096)
    return p, ln, offsets


def _gen_c5(rng, segments, max_seg):
    sizes = rng.integers(1, max_seg + 1, segments).astype(np.int64)
    offsets = np.zeros(segments + 1, dtype=np.int64)
    np.cumsum(sizes, out=offsets[1:])
    total = int(offsets[-1])
    lowest = rng.random(total) < 0.7
    rest = rng.integers(0, 7, total)
    p = np.where(lowest, 7, rest).astype(np.uint8)
    ln = np.clip(np.floor(rng.pareto(1.5, total) + 1.0), 1, 65536).astype(np.int32)
    mask = rng.random(total) < 0.3
    src = ln.copy()
    idx = np.arange(total, dtype=np.int64)
    seg_of = np.repeat(np.arange(segments, dtype=np.int64), sizes)
    first = idx == offsets[seg_of]
    neighbour = np.where(first, idx + 1, idx - 1)
    usable = mask & (sizes[seg_of] > 1)
    ln[usable] = src[neighbour[usable]]
    return p, ln, offsets


def generate(name: str, scale: float = 1.0) -> Workload:
    """Build workload ``name`` (c1..c5).

    ``scale`` < 1 shrinks the request count (single queue) or the number of
    queues (batched) for quick tests; the value distributions are unchanged.
    The full-size arrays are reproduced bit for bit on any machine with the
    same numpy, which ``sha256_arrays`` checks.
    """
    cfg = CONFIGS[name]
    rng = np.random.default_rng(cfg["seed"])
    if name == "c1":
        n = max(1, int(cfg["n"] * scale))
        p, ln, off = _gen_c1(rng, n)
    elif name == "c2":
        n = max(1, int(cfg["n"] * scale))
        p, ln, off = _gen_c2(rng, n)
    elif name == "c3":
        n = max(1, int(cfg["n"] * scale))
        p, ln, off = _gen_c3(rng, n)
    elif name == "c4":
        s = max(1, int(cfg["segments"] * scale))
        p, ln, off = _gen_c4(rng, s, cfg["seg_size"])
    elif name == "c5":
        s = max(1, int(cfg["segments"] * scale))
        p, ln, off = _gen_c5(rng, s, cfg["max_seg"])
    else:
        raise KeyError(name)
    classes = cfg["classes"] if off is not None else 256
    return Workload(name=name, priority=p, length=ln, offsets=off,
                    num_classes=classes, meta=dict(cfg, scale=scale))


def fuzz_queue(n: int, seed: int, classes: int = 5, max_len: int = 1000,
               tie_frac: float = 0.0, min_len: int = 1) -> tuple:
    """Random single queue of n requests.

    ``tie_frac`` of the requests copy the (class, length) of an earlier
    request so that exact key ties occur and the id tie-break matters.
    """
    rng = np.random.default_rng(seed)
    p = rng.integers(0, classes, n, dtype=np.uint8)
    ln = rng.integers(min_len, max_len + 1, n, dtype=np.int64).astype(np.int32)
    if n > 1 and tie_frac > 0:
        mask = rng.random(n) < tie_frac
        mask[0] = False
        src = (rng.random(n) * np.arange(n)).astype(np.int64)
        p[mask] = p[src[mask]]
        ln[mask] = ln[src[mask]]
    return p, ln


def fuzz_segments(sizes, seed: int, classes: int = 4, max_len: int = 500,
                  tie_frac: float = 0.2) -> tuple:
    """Random batched input with the given per-queue sizes."""
    sizes = np.asarray(sizes, dtype=np.int64)
    offsets = np.zeros(sizes.size + 1, dtype=np.int64)
    np.cumsum(sizes, out=offsets[1:])
    p, ln = fuzz_queue(int(offsets[-1]), seed, classes, max_len, tie_frac)
    return p, ln, offsets


def workload_sha256(w: "Workload") -> str:
    """SHA-256 of a workload's arrays (priority, length, offsets if batched)."""
    if w.offsets is None:
        return sha256_arrays(w.priority, w.length)
    return sha256_arrays(w.priority, w.length, w.offsets)


def sha256_arrays(*arrays) -> str:
    h = hashlib.sha256()
    for a in arrays:
        if a is None:
            h.update(b"none")
            continue
        a = np.ascontiguousarray(a)
        h.update(str(a.dtype).encode())
        h.update(str(a.shape).encode())
        h.update(a.tobytes())
    return h.hexdigest()


def cost_tokens(output: np.ndarray, seed: int = 5) -> tuple:
    """(prompt, decoded) token counts for requests whose predicted output
    lengths are ``output`` (int32 arrays of the same size)."""
    rng = np.random.default_rng(seed)
    n = output.shape[0]
    prompt = rng.integers(1, 4097, n).astype(np.int32)
    started = rng.random(n) < 0.25
    dec = (rng.random(n) * output.astype(np.float64)).astype(np.int64) + 1
    decoded = np.where(started, np.minimum(dec, output), 0).astype(np.int32)
    return prompt, decoded
