"""Random shapes through orloj_iterate against the oracle (hypothesis,
derandomised): 1..300 bins, 1..80 classes, batch-size sets of a few sizes
or a run 1..n with n up to 140 (so first-bin tables on both sides of what
LDS stages), queues of up to 1600 requests (whole, or with the drop phase
in parts), dead / in-grid / beyond-grid deadlines, optional miss costs and
step cost functions, delay rates 1e-6..1e-1.  ORLOJ_ITERATE_SWEEP_EXAMPLES
sets the number of cases (default 60)."""
import dataclasses
import os
import sys

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
from paper_2209_00159_amd import orloj as O
from paper_2209_00159_amd import workloads as W
from test_gpu_iterate import check, random_steps

pytestmark = pytest.mark.gpu

SETTINGS = dict(max_examples=int(os.environ.get("ORLOJ_ITERATE_SWEEP_EXAMPLES", "60")),
                deadline=None, derandomize=True, database=None,
                suppress_health_check=[HealthCheck.too_slow, HealthCheck.function_scoped_fixture])


@pytest.fixture(scope="module")
def ctx():
    return O.Context()


@st.composite
def shapes(draw):
    if draw(st.booleans()):
        bs = tuple(sorted(set(draw(st.lists(st.integers(1, 70), min_size=1, max_size=6)))))
    else:
        lo = draw(st.integers(1, 3))
        bs = tuple(range(lo, lo + draw(st.integers(30, 140))))
    M = draw(st.integers(1, 3))
    lens = draw(st.lists(st.one_of(st.integers(0, 130), st.integers(500, 1600)),
                         min_size=M, max_size=M))
    return dict(seed=draw(st.integers(0, 10 ** 6)), n_models=M, n_classes=draw(st.integers(1, 80)),
                n_bins=draw(st.integers(1, 300)), batch_sizes=bs, queue_lens=lens,
                sparsity=draw(st.sampled_from([0.0, 0.3, 0.9])),
                tau_range=(-10.0, draw(st.sampled_from([20.0, 200.0, 5000.0]))),
                b_expo=10.0 ** draw(st.floats(-6.0, -1.0)))


@settings(**SETTINGS)
@given(case=shapes(), costs=st.booleans(), steps=st.booleans())
def test_random_iterations_match_oracle(ctx, case, costs, steps):
    print("iterate sweep", case, "costs", costs, "steps", steps, flush=True)
    sys.stdout.flush()
    wl = W.random_case(**case)
    if costs:
        r = np.random.default_rng(case["seed"])
        wl = dataclasses.replace(wl, cost=r.uniform(0.0, 3.0, size=wl.cls.size))
    # (step arrays for an empty queue array would be empty: NULL pointers,
    # which the ABI rejects as incomplete steps)
    st_ = random_steps(wl, case["seed"]) if steps and wl.cls.size else None
    it = O.Iterator(wl, ctx)
    it.set_queues(wl.queue_off, wl.cls, wl.deadline_ms, wl.now_ms, steps=st_)
    got = it.run()
    ora = oracle.iterate_workload(wl, steps=st_)
    check(wl, got, ora)
