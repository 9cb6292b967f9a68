"""Host-side checks of bench.py's reading of committed counter summaries: a
summary counts only for the code it was taken on (the kernel source and the
common headers, comments aside) and for the same request count."""

import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def _write(path, text):
    with open(path, "w") as f:
        f.write(text)


def test_code_sha_ignores_comments_and_blank_lines(tmp_path):
    a = tmp_path / "a.hip"
    b = tmp_path / "b.h"
    _write(a, "int x = 1;\n")
    _write(b, "int y = 2;\n")
    base = bench.code_sha((str(a), str(b)))
    _write(a, "// a comment\n\nint x = 1;  // trailing\n")
    assert bench.code_sha((str(a), str(b))) == base
    _write(b, "int y = 3;\n")  # a header change is a kernel change
    assert bench.code_sha((str(a), str(b))) != base
    assert bench.code_sha(str(a)) != base  # the file set matters


def test_profile_values_only_for_matching_code_and_size(tmp_path):
    src = tmp_path / "k.hip"
    _write(src, "int k;\n")
    prof = tmp_path / "p.md"
    _write(prof, "# title\n\n| a | b |\n\nn: 64\ncode_sha256: %s\nhbm_bytes_per_step: 1234\n"
           % bench.code_sha(str(src)))
    assert bench.profile_values(str(prof), str(src), ["hbm_bytes_per_step"], 64) == {
        "hbm_bytes_per_step": 1234.0}
    assert bench.profile_values(str(prof), str(src), ["hbm_bytes_per_step"], 65) is None
    assert bench.profile_values(str(prof), str(src), ["missing_key"], 64) is None
    _write(src, "int k2;\n")
    assert bench.profile_values(str(prof), str(src), ["hbm_bytes_per_step"], 64) is None


@pytest.mark.parametrize("name, source", [
    ("c3_step_counters.md", "FINAL_SOURCE"),
    ("batched_c4_counters.md", "BATCHED_SOURCE"),
    ("batched_c5_counters.md", "BATCHED_SOURCE"),
    ("insert_merge_c3_counters.md", "MERGE_SOURCE"),
    ("policy_c3_counters.md", "POLICY_SOURCE"),
    ("cost_c3_counters.md", "FINAL_SOURCE"),
])
def test_committed_summaries_parse(name, source):
    """Every committed summary carries n and a code SHA in the format read."""
    path = os.path.join(ROOT, "profiles", name)
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith(("|", "#", " ")):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    assert int(kv["n"]) > 0
    assert len(kv["code_sha256"]) == 64
    assert isinstance(getattr(bench, source), tuple)
