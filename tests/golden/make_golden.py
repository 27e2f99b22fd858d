"""Regenerate the stored budget vectors from the oracle allocator (run from the repo root).

    python tests/golden/make_golden.py

Calls only oracle/ and the workload configuration data.
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import alloc  # noqa: E402
from synth.workloads import B_MIN, pyramid_weights  # noqa: E402


def main():
    w = pyramid_weights(32)
    b512 = [int(x) for x in alloc.allocate(w, 32 * 512, B_MIN)]
    sweep = {str(avg): [int(x) for x in alloc.allocate(b512, 32 * avg, B_MIN)]
             for avg in (128, 256, 512, 1024, 2048)}
    out = {
        "_source": "oracle.alloc.allocate (Eq. 3 with the b_min clamp and largest-remainder "
                   "rounding, Section 3.3) on the 32-layer linear ramp 1024 -> 128; each sweep "
                   "point reuses the finished 512-average vector as its allocation weights at the "
                   "new total (the budget-sweep rule of Section 3.3), b_min still 48",
        "b_min": B_MIN,
        "pyramid_512": b512,
        "sweep": sweep,
    }
    with open(os.path.join(HERE, "budgets.json"), "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")


if __name__ == "__main__":
    main()
