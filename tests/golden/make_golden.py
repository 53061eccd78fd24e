"""Writes tests/golden/schedules.json from the oracle's schedule only (no GPU-library code).

Run from the repository root:  python tests/golden/make_golden.py
"""

import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import partition, schedule  # noqa: E402

CASES = [
    # (seed, sweep, rows, block_m, cols, block_n)
    (1, 0, 1000, 256, 1000, 256),
    (3, 0, 32768, 4096, 32768, 4096),
    (3, 4, 32768, 4096, 32768, 4096),
    (4, 0, 139255, 8192, 139255, 8192),
    (4, 1, 139255, 8192, 139255, 8192),
    (5, 0, 500000, 16384, 50000, 8192),
    (0xDEADBEEFCAFEF00D, 7, 100, 3, 50, 7),
    (2**64 - 1, 2**40, 9, 2, 12, 5),
]


def main():
    out = []
    for seed, t, m, bm, n, bn in CASES:
        R = partition.num_blocks(m, bm)
        C = partition.num_blocks(n, bn)
        out.append({
            "seed": str(seed), "sweep": t, "m": m, "block_m": bm, "n": n, "block_n": bn,
            "row_bounds": partition.bounds(m, bm), "col_bounds": partition.bounds(n, bn),
            "steps": schedule.sweep_schedule(seed, t, R, C, True),
        })
    path = os.path.join(ROOT, "tests", "golden", "schedules.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print("wrote", path)


if __name__ == "__main__":
    main()
