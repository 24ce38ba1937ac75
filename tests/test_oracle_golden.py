"""The oracle still reproduces its recorded outputs on the tiny
configuration (tests/golden/make_golden.py wrote them)."""
import os

import numpy as np

import oracle
from paper_2209_00159_amd import workloads as W

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "cfg1_oracle.txt")


def test_cfg1_golden():
    rec = {}
    with open(GOLD) as f:
        for line in f:
            if line.startswith("#"):
                continue
            k, *vals = line.split()
            rec[k] = vals
    o = oracle.score_workload(W.make(1))
    n, b, s = rec["selection"]
    assert (int(n), int(b)) == (int(o["sel_n"][0]), int(o["sel_bs"][0]))
    assert abs(float(s) - o["sel_score"][0]) <= 1e-15
    for k in ("expected_finish", "expected_latency_ms", "score", "finish_prob"):
        ref = np.array([float(v) for v in rec[k]])
        assert np.allclose(o[k], ref, rtol=1e-14, atol=1e-300), k
