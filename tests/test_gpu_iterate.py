"""The scheduler iteration (Algorithm 1 with the paper's own priority)
through the C ABI against the oracle: timed-out flags and candidate batch
sizes bit-exact, priorities within the score bar, and the popped batch a
valid top-s under the oracle's priorities (ties within the bar aside)."""
import os
import sys

import numpy as np
import pytest

import oracle
import parity
from paper_2209_00159_amd import orloj as O
from paper_2209_00159_amd import workloads as W

pytestmark = pytest.mark.gpu

TOL_ABS, TOL_REL = 1e-6, 1e-5


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def ctx():
    return O.Context()


def check(wl, got, ora):
    err = 0.0
    for q in range(wl.n_models):
        a, b = int(wl.queue_off[q]), int(wl.queue_off[q + 1])
        o = ora["per_model"][q]
        assert np.array_equal(got["timed_out"][a:b], o["timed_out"]), q
        assert int(got["cand_bs"][q]) == o["cand_bs"], (q, got["cand_bs"][q], o["cand_bs"])
        gs = got["score"][a:b].astype(np.float64)
        os_ = o["score"]
        d = np.abs(gs - os_)
        assert np.all(d <= TOL_ABS + TOL_REL * np.abs(os_)), (q, float(d.max()))
        err = max(err, float(d.max(initial=0.0)))
        s = o["cand_bs"]
        gb = got["batch"][q]
        if s == 0:
            assert np.all(gb == -1), q
            continue
        assert np.all(gb[s:] == -1) and np.all(gb[:s] >= 0), q
        sel = gb[:s]
        assert len(set(sel.tolist())) == s
        # ordered by the GPU's own priorities, earlier position first on ties
        g_sel = gs[sel]
        assert np.all((g_sel[:-1] > g_sel[1:]) | ((g_sel[:-1] == g_sel[1:]) & (sel[:-1] < sel[1:]))), q
        # a top-s set under the oracle's priorities, up to the bar
        kept = np.nonzero(os_ > 0)[0] if np.any(os_ > 0) else np.array([], int)
        thr = np.sort(os_[o["batch"]])[0]
        tol = TOL_ABS + TOL_REL * abs(thr)
        assert np.all(os_[sel] >= thr - tol), q
        rest = np.setdiff1d(np.arange(b - a), sel)
        in_q = rest[np.isin(rest, kept)]
        assert np.all(os_[in_q] <= thr + tol), q
    return err


ORACLE_THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


def run(wl, ctx, weights=None, b_expo=None):
    it = O.Iterator(wl, ctx, class_weights=weights)
    got = it.run(b_expo=b_expo)
    ora = oracle.iterate_workload(wl if b_expo is None else _with_b(wl, b_expo), weights=weights,
                                  threads=ORACLE_THREADS)
    return got, ora


def _with_b(wl, b):
    import dataclasses
    return dataclasses.replace(wl, b_expo=b)


CASES = [
    dict(seed=0),
    dict(seed=1, n_models=3, queue_lens=[0, 7, 13], batch_sizes=(1, 4, 16)),
    dict(seed=2, n_bins=1, batch_sizes=(1, 2)),
    dict(seed=3, n_bins=2, n_classes=1),
    dict(seed=4, n_bins=255, batch_sizes=(2, 3, 5, 7, 11, 13)),
    dict(seed=5, n_bins=257, queue_lens=[40, 1], batch_sizes=(1, 8, 32, 64)),
    dict(seed=6, n_bins=1023, n_classes=7, queue_lens=[65, 64], batch_sizes=(1, 63, 64, 65)),
    dict(seed=7, n_models=1, n_bins=4096, n_classes=5, queue_lens=[300], batch_sizes=(16, 64)),
    dict(seed=9, n_models=5, queue_lens=[0, 0, 0, 0, 0]),
    dict(seed=10, n_models=1, n_bins=100, queue_lens=[4096], batch_sizes=(128, 256, 1024)),
    dict(seed=11, n_bins=64, tau_range=(-50.0, -1.0)),
    dict(seed=12, n_bins=64, tau_range=(500.0, 900.0)),
    dict(seed=13, n_bins=300, sparsity=0.9, total=3),
    # 128-bit table accesses with the last thread chunks past the row's end
    dict(seed=14, n_bins=1000, n_classes=4, queue_lens=[40, 17], batch_sizes=(1, 5, 16)),
    dict(seed=15, n_models=1, n_bins=8192, n_classes=3, queue_lens=[30], batch_sizes=(4, 32)),
    # 128 batch sizes (two rows of lanes) with 64 classes (first-bin table
    # of 64 x 129 words, staged in LDS) and 66 classes (66 x 129 = 8514
    # words, past the 8448 staged: read from the support table)
    dict(seed=16, n_models=2, n_bins=40, n_classes=64, queue_lens=[200, 90],
         batch_sizes=tuple(range(1, 129))),
    dict(seed=17, n_models=2, n_bins=40, n_classes=66, queue_lens=[200, 90],
         batch_sizes=tuple(range(1, 129))),
    # a queue past 1024 requests (1024-thread workgroups) beside a short one
    # (rank counting) and an empty one, in the same launch
    dict(seed=18, n_models=3, n_bins=200, queue_lens=[1025, 3, 0], batch_sizes=(1, 7, 64, 512)),
    dict(seed=19, n_models=2, n_bins=60, n_classes=9, queue_lens=[2000, 600],
         batch_sizes=tuple(range(1, 129))),
    # many classes over 40 batch sizes: 200 x 41 words staged, 210 x 41 not
    dict(seed=22, n_models=2, n_bins=30, n_classes=200, queue_lens=[1500, 70],
         batch_sizes=tuple(range(1, 41))),
    dict(seed=23, n_models=1, n_bins=30, n_classes=210, queue_lens=[700],
         batch_sizes=tuple(range(1, 41))),
    # 256 batch sizes: four rows of lanes
    dict(seed=24, n_models=2, n_bins=50, n_classes=6, queue_lens=[1100, 300],
         batch_sizes=tuple(range(1, 257))),
    # batch sizes across the lanes at the edges of the keep test: one and
    # two bins, deadlines all past or all before, 33 / 65 / 129 batch sizes
    dict(seed=25, n_bins=1, queue_lens=[90, 33], batch_sizes=tuple(range(1, 34))),
    dict(seed=26, n_models=1, n_bins=2, n_classes=1, queue_lens=[70], batch_sizes=tuple(range(2, 67))),
    dict(seed=27, n_bins=64, tau_range=(-50.0, -1.0), queue_lens=[300, 70], batch_sizes=tuple(range(1, 130))),
    dict(seed=28, n_bins=64, tau_range=(500.0, 900.0), queue_lens=[300, 70], batch_sizes=tuple(range(1, 130))),
    dict(seed=29, n_bins=300, sparsity=0.9, total=3, queue_lens=[1200, 5], batch_sizes=tuple(range(1, 66))),
    # long queues on few models run the drop phase in parts of 256 requests
    # (the cases above with a queue past 1024); on 70 models the same
    # queues stay whole, one 1024-thread workgroup per model
    dict(seed=30, n_models=70, n_bins=40, n_classes=5, queue_lens=[1500] + [3] * 68 + [1025],
         batch_sizes=tuple(range(1, 41))),
    dict(seed=31, n_models=70, n_bins=40, n_classes=5, queue_lens=[0] * 69 + [2049],
         batch_sizes=(1, 4, 9, 30)),
    dict(seed=32, n_models=3, n_bins=70, n_classes=4, queue_lens=[1536, 1537, 0],
         batch_sizes=(2, 16, 500)),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"seed{c['seed']}")
def test_iterate_random_cases(ctx, case):
    say("iterate", case)
    wl = W.random_case(**case)
    got, ora = run(wl, ctx)
    say("  max |d score|", check(wl, got, ora))


@pytest.mark.parametrize("seed", [20, 21])
def test_iterate_class_weights(ctx, seed):
    wl = W.random_case(seed, n_models=3, queue_lens=[30, 12, 50], n_classes=5, n_bins=200,
                       batch_sizes=(1, 2, 4, 8, 16))
    r = np.random.default_rng(seed)
    weights = r.random((3, 5))
    weights[1, 2:] = 0.0
    got, ora = run(wl, ctx, weights=weights)
    check(wl, got, ora)


@pytest.mark.parametrize("b", [1e-6, 1e-2, 1e-1])
def test_iterate_delay_rate(ctx, b):
    wl = W.random_case(30, n_models=2, queue_lens=[40, 25], batch_sizes=(1, 2, 4, 8, 16, 32),
                       n_bins=512, tau_range=(0.0, 700.0))
    got, ora = run(wl, ctx, b_expo=b)
    check(wl, got, ora)


@pytest.mark.parametrize("cid,scale", [(1, 1.0), (1, 4.0), (2, 1.0), (2, 3.0), (3, 1.0), (3, 5.0),
                                       (4, 1.0), (4, 3.0), (5, 1.0), (5, 4.0)])
def test_iterate_configs(ctx, cid, scale):
    say(f"iterate config {cid} slo x{scale}")
    wl = parity.make_cached(cid, scale)
    got, ora = run(wl, ctx)
    say("  candidates", np.unique(got["cand_bs"]), "max |d score|", check(wl, got, ora))


def test_iterate_bad_weights_are_a_data_error(ctx):
    wl = W.random_case(40, n_models=2, queue_lens=[6, 3], n_classes=3)
    weights = np.ones((2, 3))
    weights[1] = 0.0
    it = O.Iterator(wl, ctx, class_weights=weights)
    it.build()
    with pytest.raises(O.OrlojError) as ei:
        ctx.sync()
    assert ei.value.code == O.ORLOJ_E_DATA


def test_iterate_queue_limit_is_unsupported(ctx):
    wl = W.random_case(41, n_models=1, queue_lens=[4097], batch_sizes=(1, 8))
    it = O.Iterator(wl, ctx)
    it.build()
    with pytest.raises(O.OrlojError) as ei:
        it.iterate()
    assert ei.value.code == O.ORLOJ_E_UNSUPPORTED


# ---------------------------------------------------------------- costs, step costs, profiler
def random_steps(wl, seed, max_steps=3):
    r = np.random.default_rng(seed)
    n = wl.cls.size
    k = r.integers(1, max_steps + 1, size=n)
    off = np.concatenate([[0], np.cumsum(k)]).astype(np.int64)
    dl, co = [], []
    for i in range(n):
        d = wl.deadline_ms[i] + np.concatenate([[0.0], np.cumsum(r.uniform(1.0, 40.0, size=k[i] - 1))])
        c = np.cumsum(r.uniform(0.1, 2.0, size=k[i]))
        dl.append(d)
        co.append(c)
    return off, np.concatenate(dl), np.concatenate(co)


@pytest.mark.parametrize("seed", [50, 51, 52])
def test_iterate_costs_and_steps(ctx, seed):
    import dataclasses
    wl = W.random_case(seed, n_models=3, queue_lens=[25, 9, 40], n_classes=4, n_bins=300,
                       batch_sizes=(1, 2, 4, 8), tau_range=(-5.0, 200.0))
    r = np.random.default_rng(seed)
    wl = dataclasses.replace(wl, cost=r.uniform(0.0, 3.0, size=wl.cls.size))
    steps = random_steps(wl, seed)
    it = O.Iterator(wl, ctx)
    it.set_queues(wl.queue_off, wl.cls, wl.deadline_ms, wl.now_ms, steps=steps)
    got = it.run()
    ora = oracle.iterate_workload(wl, steps=steps)
    check(wl, got, ora)


@pytest.mark.parametrize("seed,lens", [(54, [300, 9, 40]), (55, [1300, 9, 700])],
                         ids=["lanes-over-batch-sizes", "drop-in-parts"])
def test_iterate_costs_and_steps_wide(ctx, seed, lens):
    """Step cost functions where the drop phase runs across the batch sizes
    in the lanes (40 batch sizes), and split into parts (a 1300-request
    queue): the keep edge comes from each request's last step."""
    import dataclasses
    wl = W.random_case(seed, n_models=3, queue_lens=lens, n_classes=6, n_bins=200,
                       batch_sizes=tuple(range(1, 41)), tau_range=(-5.0, 150.0))
    r = np.random.default_rng(seed)
    wl = dataclasses.replace(wl, cost=r.uniform(0.0, 3.0, size=wl.cls.size))
    steps = random_steps(wl, seed)
    it = O.Iterator(wl, ctx)
    it.set_queues(wl.queue_off, wl.cls, wl.deadline_ms, wl.now_ms, steps=steps)
    got = it.run()
    ora = oracle.iterate_workload(wl, steps=steps)
    check(wl, got, ora)


def test_iterate_bad_steps_are_a_data_error(ctx):
    wl = W.random_case(53, n_models=1, queue_lens=[4], tau_range=(10.0, 40.0))
    off = np.array([0, 1, 3, 4, 5], np.int64)
    dl = np.array([wl.deadline_ms[0], wl.deadline_ms[1], wl.deadline_ms[1] - 1.0,
                   wl.deadline_ms[2], wl.deadline_ms[3]])
    co = np.array([1.0, 1.0, 2.0, 1.0, 1.0])
    it = O.Iterator(wl, ctx)
    it.set_queues(wl.queue_off, wl.cls, wl.deadline_ms, wl.now_ms, steps=(off, dl, co))
    it.build()
    it.iterate()
    with pytest.raises(O.OrlojError) as ei:
        ctx.sync()
    assert ei.value.code == O.ORLOJ_E_DATA


@pytest.mark.parametrize("n", [0, 1, 1000, 200_000])
def test_accumulate_matches_oracle(ctx, n):
    import torch
    r = np.random.default_rng(60 + n)
    M, B, C, K = 3, 4, 5, 257
    widths = np.array([0.5, 1.25, 2.0])
    counts = r.integers(0, 9, size=(M, B, C, K)).astype(np.uint32)
    mo = r.integers(0, M, size=n).astype(np.int32)
    bi = r.integers(0, B, size=n).astype(np.int32)
    cl = r.integers(0, C, size=n).astype(np.int32)
    lat = r.uniform(0.0, 1.2 * K, size=n) * widths[np.clip(mo, 0, M - 1)]
    bad = r.random(n)
    lat[bad < 0.01] = -3.0
    lat[(bad >= 0.01) & (bad < 0.02)] = np.nan
    lat[(bad >= 0.02) & (bad < 0.03)] = np.inf
    mo[(bad >= 0.03) & (bad < 0.035)] = M
    cl[(bad >= 0.035) & (bad < 0.04)] = -1
    ref = counts.copy()
    rej_ref = oracle.accumulate(ref, widths, mo, bi, cl, lat)
    dev = ctx.device
    d_counts = torch.from_numpy(counts.view(np.int32)).to(dev)
    d_w = torch.from_numpy(widths).to(dev)
    grid = O.make_grid(M, C, K, np.arange(1, B + 1), d_w)
    rej = O.accumulate(ctx, grid, d_counts, torch.from_numpy(mo).to(dev), torch.from_numpy(bi).to(dev),
                       torch.from_numpy(cl).to(dev), torch.from_numpy(lat).to(dev))
    got = d_counts.cpu().numpy().view(np.uint32)
    assert rej == rej_ref
    assert np.array_equal(got, ref)
