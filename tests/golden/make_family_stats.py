"""Write family_stats.json: the family size, pair count, table cells and
relaxation count (the DP's unit of work) of every benchmark workload,
counted from the oracle's family with plain set operations
(tests/family_stats.py).  Run from the repository root:

    python tests/golden/make_family_stats.py
"""

import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from paper_1905_11722_amd import workloads as W  # noqa: E402
from tests.family_stats import family_stats  # noqa: E402

NAMES = ["chain16", "layered24", "resnet50", "densenet121", "unet", "ladder40",
         "resnet50_t10", "densenet121_t10", "unet_t10"]


def main():
    out = {}
    for name in NAMES:
        c = W.case(name)
        s = family_stats(c.graph, c.mode)
        s.pop("w")
        s["mode"] = c.mode
        out[name] = s
        print(name, s)
    with open(os.path.join(HERE, "family_stats.json"), "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)
        f.write("\n")


if __name__ == "__main__":
    main()
