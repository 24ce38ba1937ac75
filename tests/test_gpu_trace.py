"""The scheduling loop of configuration 5 driven through the C ABI: the
selections made along a trace are checked against the oracle, state by
state, on recorded decision states."""
import sys

import numpy as np
import pytest

import oracle
import parity
from paper_2209_00159_amd import orloj as O
from paper_2209_00159_amd import schedsim as S

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def test_trace_loop_selections_match_oracle():
    ctx = O.Context()
    models = list(range(8))
    say("config 5 loop: 8 models, 1500 arrivals")
    loop = S.config5_loop(1500, ctx=ctx, models=models, workers=8, record_every=1, record_limit=40)
    st = loop.run()
    say("  stats", st.as_dict())
    assert st.decisions >= 40 and len(st.recorded) == 40
    assert st.dispatched + st.dropped <= 1500
    assert st.on_time + st.late == st.dispatched
    wl = loop.wl
    bs = set(int(b) for b in wl.batch_sizes)
    for dec in st.recorded:
        assert dec.sel_bs in bs and 1 <= dec.sel_n <= min(dec.sel_bs, dec.cls.size)
        assert np.all(np.diff(dec.deadline_ms) >= 0)
        sub = wl.subset([dec.model]).with_queues([(dec.cls, dec.deadline_ms)], [dec.now_ms])
        ora = oracle.score_workload(sub)
        parity.check_selection(sub, 0, 0, ora["score"], (dec.sel_n, dec.sel_bs))
