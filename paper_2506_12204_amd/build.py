"""Build libsemsched.so (the HIP kernels and the C ABI) for gfx950, in-tree.

Usage: python paper_2506_12204_amd/build.py
(run by path: importing the package itself needs the built library)

Every source is compiled to an object of its own, in parallel, then the
objects are linked into the shared library.
"""

from __future__ import annotations

import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libsemsched.so")
SOURCES = ["abi.hip", "batched.hip", "global_sort.hip", "insert.hip", "policy.hip",
           "cost.hip", "batch.hip"]
ARCH = os.environ.get("SEMSCHED_ARCH", "gfx950")
NOISE = "is not a recognized feature for this target"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if cand and (os.path.isabs(cand) and os.path.exists(cand) or not os.path.isabs(cand)):
            return cand
    return "hipcc"


def flags() -> list:
    return [
        f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
        # no packed FP32 instructions anywhere in device code
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-I", INCLUDE, "-I", CSRC,
    ]


def command(out: str = LIB) -> list:
    """One-step build command (all sources at once)."""
    return [hipcc()] + flags() + ["-shared", "-o", out] + [os.path.join(CSRC, s) for s in SOURCES]


def _run(cmd: list) -> tuple:
    res = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(x for x in res.stderr.splitlines() if NOISE not in x)
    return res.returncode, err


def build(verbose: bool = False) -> str:
    jobs = max(1, min(len(SOURCES), int(os.environ.get("MAX_JOBS", os.cpu_count() or 4))))
    with tempfile.TemporaryDirectory(prefix="semsched_build_") as tmpdir:
        objs = [os.path.join(tmpdir, os.path.splitext(s)[0] + ".o") for s in SOURCES]
        cmds = [[hipcc()] + flags() + ["-c", os.path.join(CSRC, s), "-o", o]
                for s, o in zip(SOURCES, objs)]
        if verbose:
            for c in cmds:
                print(" ".join(c), flush=True)
        with ThreadPoolExecutor(max_workers=jobs) as ex:
            results = list(ex.map(_run, cmds))
        for s, (rc, err) in zip(SOURCES, results):
            if rc != 0:
                raise RuntimeError(f"hipcc failed on {s} ({rc}):\n{err}")
            if verbose and err.strip():
                print(err, file=sys.stderr)
        tmp = LIB + ".tmp"
        link = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
        if verbose:
            print(" ".join(link), flush=True)
        rc, err = _run(link)
        if rc != 0:
            raise RuntimeError(f"link failed ({rc}):\n{err}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
