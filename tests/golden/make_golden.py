"""Write tests/golden/cfg1_oracle.txt: the CPU oracle's outputs on the tiny
single-model configuration (4 lognormal classes, 128 bins over 0-200 ms,
batch sizes 1..16, 64 queued requests).

The paper prints no numeric worked example (its toy example in §4.2.2 is a
figure), so this fixture is a regression record of the oracle itself.  It
calls only the oracle and the seeded input generator.
"""
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
from paper_2209_00159_amd import workloads as W  # noqa: E402

OUT = os.path.join(HERE, "cfg1_oracle.txt")


def main():
    wl = W.make(1)
    o = oracle.score_workload(wl)
    with open(OUT, "w") as f:
        f.write("# oracle outputs for the tiny single-model configuration; "
                "written by tests/golden/make_golden.py\n")
        f.write(f"selection {o['sel_n'][0]} {o['sel_bs'][0]} {o['sel_score'][0]:.17g}\n")
        for k in ("expected_finish", "expected_latency_ms", "score", "finish_prob"):
            f.write(k + " " + " ".join(f"{v:.17g}" for v in o[k]) + "\n")


if __name__ == "__main__":
    main()
