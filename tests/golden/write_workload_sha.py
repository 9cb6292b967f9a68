"""Write the SHA-256 of every synthetic workload's arrays (C1-C5 at full size)
to workload_sha256.json beside this script.

The hashes pin the seeded generators of workloads/gen.py (priority, length
and offsets arrays, dtype and shape included): tests/test_workloads.py
regenerates each workload and compares, and bench.py reports the hash of the
input it timed.

Usage: python tests/golden/write_workload_sha.py
"""

import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from workloads import CONFIGS, generate, workload_sha256  # noqa: E402


def main() -> None:
    out = {name: workload_sha256(generate(name)) for name in sorted(CONFIGS)}
    with open(os.path.join(HERE, "workload_sha256.json"), "w") as f:
        json.dump(out, f, indent=2, sort_keys=True)
        f.write("\n")
    print(json.dumps(out, indent=2))


if __name__ == "__main__":
    main()
