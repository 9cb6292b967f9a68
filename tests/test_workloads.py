"""The synthetic workload generators: shapes, ranges and class mix."""

import numpy as np
import pytest

from workloads import CONFIGS, fuzz_segments, generate, sha256_arrays


def test_c1_shape_and_ranges():
    w = generate("c1")
    assert w.n == 1000 and w.offsets is None
    assert w.priority.dtype == np.uint8 and w.length.dtype == np.int32
    assert w.priority.max() <= 3 and 1 <= w.length.min() and w.length.max() <= 4096


def test_c2_zipf_and_duplicates():
    w = generate("c2", 1 / 16)
    freq = np.bincount(w.priority, minlength=10) / w.n
    assert freq[0] < freq[5] < freq[9]
    assert abs(freq[9] - 0.405) < 0.02 and abs(freq[0] - 0.026) < 0.01
    assert w.length.min() >= 1 and w.length.max() <= 8192
    keys = w.priority.astype(np.int64) << 32 | w.length
    assert np.unique(keys).size < 0.8 * w.n  # many exact (class, length) ties


def test_c3_small_scale_ranges():
    w = generate("c3", 1 / 1024)
    assert w.n == (1 << 26) // 1024
    assert w.priority.max() == 4 and w.length.min() >= 1 and w.length.max() <= 32768


def test_c4_c5_offsets():
    w4 = generate("c4", 1 / 256)
    assert np.all(np.diff(w4.offsets) == 256) and w4.offsets[-1] == w4.n
    w5 = generate("c5", 1 / 64)
    sizes = np.diff(w5.offsets)
    assert sizes.min() >= 1 and sizes.max() <= 4096 and w5.offsets[-1] == w5.n
    share7 = np.mean(w5.priority == 7)
    assert abs(share7 - 0.7) < 0.02  # the other 30 % spread over 0..6
    assert w5.length.min() >= 1 and w5.length.max() <= 65536


def test_deterministic():
    a = generate("c5", 1 / 128)
    b = generate("c5", 1 / 128)
    assert sha256_arrays(a.priority, a.length, a.offsets) == \
        sha256_arrays(b.priority, b.length, b.offsets)


def test_fuzz_segments_layout():
    p, l, off = fuzz_segments([0, 5, 1], seed=1)
    assert off.tolist() == [0, 0, 5, 6] and p.size == 6 and l.size == 6


@pytest.mark.parametrize("name", sorted(CONFIGS))
def test_config_names(name):
    assert name in ("c1", "c2", "c3", "c4", "c5")


@pytest.mark.parametrize("name", sorted(CONFIGS))
def test_recorded_sha256(name):
    # the full-size arrays hash to the values recorded by
    # tests/golden/write_workload_sha.py: the seeded generators are unchanged
    import json
    import os
    from workloads import workload_sha256
    with open(os.path.join(os.path.dirname(__file__), "golden", "workload_sha256.json")) as f:
        want = json.load(f)
    assert workload_sha256(generate(name)) == want[name]
