"""Random shapes through the HIP path against the oracle (hypothesis,
derandomised): bin counts 1..3000 (one or more panels, ragged tails), 1..6
classes, sparse and dense histograms, irregular batch-size sets, queues of
0..130 requests spanning dead, in-grid and beyond-grid deadlines, delay
rates 1e-6..1e-1, both prefix modes, optional miss costs, and both batch
laws (per-batch-size tables and the affine law c0 + c1 s l), with the
launch split into step chunks or not.  ORLOJ_SWEEP_EXAMPLES sets the number
of cases (default 80)."""
import dataclasses
import os
import sys

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
import parity
from paper_2209_00159_amd import orloj as O
from paper_2209_00159_amd import workloads as W

pytestmark = pytest.mark.gpu

SETTINGS = dict(max_examples=int(os.environ.get("ORLOJ_SWEEP_EXAMPLES", "80")), deadline=None,
                derandomize=True, database=None,
                suppress_health_check=[HealthCheck.too_slow, HealthCheck.function_scoped_fixture])


@pytest.fixture(scope="module")
def ctx():
    return O.Context()


@st.composite
def shapes(draw):
    K = draw(st.one_of(st.integers(1, 70), st.integers(900, 3000)))
    bs = sorted(set(draw(st.lists(st.integers(1, 70), min_size=1, max_size=6))))
    M = draw(st.integers(1, 3))
    return dict(seed=draw(st.integers(0, 10 ** 6)), n_models=M, n_classes=draw(st.integers(1, 6)),
                n_bins=K, batch_sizes=tuple(bs),
                queue_lens=draw(st.lists(st.integers(0, 130), min_size=M, max_size=M)),
                sparsity=draw(st.sampled_from([0.0, 0.3, 0.9])),
                tau_range=(-10.0, draw(st.sampled_from([20.0, 200.0, 5000.0]))),
                b_expo=10.0 ** draw(st.floats(-6.0, -1.0)))


@settings(**SETTINGS)
@given(case=shapes(), mode=st.sampled_from([0, 1]), costs=st.booleans(), affine=st.booleans(),
       chunk=st.sampled_from([-1, 0, 5]))
def test_random_shapes_match_oracle(ctx, case, mode, costs, affine, chunk):
    print("sweep", case, "mode", mode, "costs", costs, "affine", affine, "chunk", chunk,
          flush=True)
    sys.stdout.flush()
    wl = W.random_affine(**case) if affine else W.random_case(**case)
    if costs:
        r = np.random.default_rng(case["seed"])
        wl = dataclasses.replace(wl, cost=r.uniform(0.0, 3.0, size=wl.cls.size))
    ctx.set_score_chunk(chunk)
    try:
        got = O.Scorer(wl, ctx, prefix_mode=mode).run()
    finally:
        ctx.set_score_chunk(-1)
    ora = (oracle.score_workload_affine(wl, wl.c0_ms, wl.c1, prefix_mode=mode) if affine
           else oracle.score_workload(wl, prefix_mode=mode))
    parity.compare(wl, got, ora, mode=mode)
