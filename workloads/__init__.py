"""Seeded synthetic request queues shared by the oracle tests, the GPU parity
tests and the benchmark.

This package only draws random numbers. It holds none of the scheduling
arithmetic (no ordering, no prefix sums, no totals), so that the CPU oracle
and the HIP path can both consume its arrays without sharing any of the
method's code.
"""

from .gen import (  # noqa: F401
    CONFIGS,
    Workload,
    generate,
    fuzz_queue,
    fuzz_segments,
    sha256_arrays,
    workload_sha256,
    cost_tokens,
)
