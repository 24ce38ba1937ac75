"""HIP path against the CPU oracle, element by element, through the C ABI.

Covers the CDF-table builder, scoring and selection on random ragged cases
(empty queues, dead and beyond-grid requests, odd bin counts, sparse
histograms, non-contiguous batch sizes, both prefix modes, a sweep of the
delay rate b), on configurations 1-4 at full size (as specified and with
relaxed SLOs), and on configuration 5 at full size in the launch the
benchmark times, every model compared.
"""
import os
import sys

import numpy as np
import pytest
import torch

import oracle
import parity
from paper_2209_00159_amd import orloj as O
from paper_2209_00159_amd import workloads as W

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def ctx():
    return O.Context()


def run_gpu(wl, ctx, mode=0, b_expo=None, trim=True):
    sc = O.Scorer(wl, ctx, prefix_mode=mode, trim=trim)
    out = sc.run(build=True, b_expo=b_expo)
    return sc, out


def assert_same_bits(a, b):
    for k in a:
        assert np.array_equal(a[k].view(np.uint8), b[k].view(np.uint8)), k


# ---------------------------------------------------------------- build_cdfs
@pytest.mark.parametrize("K", [1, 3, 37, 128, 1000, 1024, 4096, 8192])
def test_build_cdfs_matches_oracle(ctx, K):
    say(f"build_cdfs K={K}")
    r = np.random.default_rng(K)
    rows = 40
    counts = r.integers(0, 1 << 20, size=(rows, K), dtype=np.int64)
    counts[r.random(counts.shape) < 0.3] = 0
    counts[3] = 0
    counts[3, -1] = 5                                   # all mass in the last bin
    counts[4] = 0
    counts[4, 0] = 7                                    # all mass in the first bin
    counts[5] = (1 << 32) - 1 - r.integers(0, 3, size=K)  # 64-bit running sums
    counts[6] = 1                                       # F = (k+1)/K
    counts[counts.sum(axis=1) == 0, -1] = 1
    c32 = counts.astype(np.uint32)
    d = torch.from_numpy(c32.view(np.int32)).to(ctx.device)
    got = ctx.build_cdfs(d).cpu().numpy().astype(np.float64)
    ctx.sync()
    for i in range(rows):
        F = oracle.cdf(c32[i])[1:]
        ref = 1.0 - F                      # fp64; exact enough next to fp32
        g = got[i]
        assert np.all(g[F == 1.0] == 0.0), i
        assert np.all(g[F == 0.0] == 1.0), i
        # relative precision of the complement: one fp32 rounding (plus
        # the fp64 rounding of 1 - F on the oracle side)
        err = np.abs(g - ref)
        assert np.all(err <= 2.0 ** -24 * ref + 1e-15), (i, np.max(err / np.maximum(ref, 1e-300)))


@pytest.mark.parametrize("K", [1, 5, 64, 1000, 4096])
def test_build_cdfs_support(ctx, K):
    say(f"build_cdfs support K={K}")
    r = np.random.default_rng(100 + K)
    rows = 24
    counts = np.zeros((rows, K), np.uint32)
    for i in range(rows):
        lo = int(r.integers(0, K))
        hi = int(r.integers(lo, K))
        counts[i, lo:hi + 1] = r.integers(0, 9, size=hi - lo + 1)
        counts[i, lo] = counts[i, hi] = 3
    counts[0] = 0
    counts[0, K - 1] = 1                                 # only the last bin
    counts[1] = 0
    counts[1, 0] = 1                                     # only the first bin
    d = torch.from_numpy(counts.view(np.int32)).to(ctx.device)
    sup = torch.full((rows, 2), -7, dtype=torch.int32, device=ctx.device)
    ccdf = ctx.build_cdfs(d, support=sup).cpu().numpy()
    ctx.sync()
    sup = sup.cpu().numpy()
    for i in range(rows):
        nz = np.nonzero(counts[i])[0]
        assert sup[i, 0] == nz[0] and sup[i, 1] == nz[-1], i
        # the entries the scorer may skip hold exactly 1 and 0
        assert np.all(ccdf[i, :nz[0]] == 1.0) and np.all(ccdf[i, nz[-1]:] == 0.0), i


def test_build_cdfs_empty_histogram_is_a_data_error(ctx):
    c = torch.zeros((2, 16), dtype=torch.int32, device=ctx.device)
    c[0, 3] = 4
    out = ctx.build_cdfs(c)
    with pytest.raises(O.OrlojError) as ei:
        ctx.sync()
    assert ei.value.code == O.ORLOJ_E_DATA
    assert torch.isnan(out[1]).all()
    ctx.sync()                                           # the error was cleared


# ---------------------------------------------------------------- scoring
RANDOM_CASES = [
    dict(seed=0),
    dict(seed=1, n_models=3, queue_lens=[0, 7, 13], batch_sizes=(1, 4, 16)),
    dict(seed=2, n_bins=1, batch_sizes=(1, 2)),
    dict(seed=3, n_bins=2, n_classes=1),
    dict(seed=4, n_bins=255, batch_sizes=(2, 3, 5, 7, 11, 13)),
    dict(seed=5, n_bins=257, queue_lens=[40, 1], batch_sizes=(1, 8, 32, 64)),
    dict(seed=6, n_bins=1023, n_classes=7, queue_lens=[65, 64], batch_sizes=(1, 63, 64, 65)),
    dict(seed=7, n_models=1, n_bins=4096, n_classes=5, queue_lens=[70], batch_sizes=(16, 64)),
    dict(seed=8, n_bins=8192, n_classes=2, queue_lens=[20, 3], batch_sizes=(1, 20)),
    dict(seed=9, n_models=5, queue_lens=[0, 0, 0, 0, 0]),
    dict(seed=10, n_models=1, n_bins=100, queue_lens=[256], batch_sizes=(128, 256)),
    dict(seed=11, n_bins=64, tau_range=(-50.0, -1.0)),          # all dead
    dict(seed=12, n_bins=64, tau_range=(500.0, 900.0)),         # all beyond the grid
    dict(seed=13, n_bins=300, sparsity=0.9, total=3),
    dict(seed=14, n_bins=2048, queue_lens=[128, 100], batch_sizes=tuple(range(1, 129, 9))),
]


@pytest.mark.parametrize("case", RANDOM_CASES, ids=lambda c: f"seed{c['seed']}")
def test_random_cases(ctx, case):
    say("random case", case)
    wl = W.random_case(**case)
    sc, got = run_gpu(wl, ctx)
    ora = oracle.score_workload(wl)
    err = parity.compare(wl, got, ora)
    say("  max errors", err)


@pytest.mark.parametrize("case", [RANDOM_CASES[i] for i in (0, 5, 6, 8, 13, 14)],
                         ids=lambda c: f"seed{c['seed']}")
def test_support_trimming_changes_no_bits(ctx, case):
    say("trim on/off", case)
    wl = W.random_case(**case)
    _, on = run_gpu(wl, ctx, trim=True)
    _, off = run_gpu(wl, ctx, trim=False)
    assert_same_bits(on, off)


@pytest.mark.parametrize("seed", [20, 21, 22])
def test_rect_mode(ctx, seed):
    say("rect", seed)
    wl = W.random_case(seed, n_models=2, queue_lens=[9, 30], batch_sizes=(1, 4, 8), n_bins=200)
    sc, got = run_gpu(wl, ctx, mode=1)
    ora = oracle.score_workload(wl, prefix_mode=1)
    parity.compare(wl, got, ora, mode=1)


@pytest.mark.parametrize("b", [1e-6, 1e-4, 1e-2, 1e-1])
def test_delay_rate_sweep(ctx, b):
    say("b sweep", b)
    wl = W.random_case(30, n_models=2, queue_lens=[40, 25], batch_sizes=(1, 2, 4, 8, 16, 32),
                       n_bins=512, b_expo=b, tau_range=(0.0, 700.0))
    sc, got = run_gpu(wl, ctx)
    ora = oracle.score_workload(wl)
    parity.compare(wl, got, ora)


# Configuration 3's earliest-deadline prefixes (the first 128 of 4096 aged
# requests) can hardly finish at its nominal SLOs: x5 gives ~11 000 member
# slots with 0 < P.
@pytest.mark.parametrize("cid,scale", [(1, 1.0), (1, 4.0), (2, 1.0), (2, 3.0), (3, 1.0),
                                       (3, 5.0), (4, 1.0), (4, 3.0)])
def test_config_full_size(ctx, cid, scale):
    say(f"config {cid} slo x{scale}")
    wl = parity.make_cached(cid, scale)
    sc, got = run_gpu(wl, ctx)
    ora = oracle.score_workload(wl)
    err = parity.compare(wl, got, ora)
    say("  max errors", err)
    if scale > 1.0:     # relaxed SLOs: the comparison is not a trivial one
        P = got["finish_prob"]
        assert int((P > 0).sum()) >= min(1000, P.size // 2) and np.all(got["sel_n"] > 0)


ORACLE_THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


@pytest.fixture(scope="module")
def cfg5():
    say("generating config 5 (128 models x 64 batch sizes x 32 classes x 4096 bins)")
    return parity.make_cached(5)


# Configuration 5 at full size, in the launch the benchmark times, compared
# with the oracle on every one of its 128 models: as specified, and at x4
# SLOs, where most member slots have 0 < P < 1.
@pytest.mark.parametrize("scale", [1.0, 4.0])
def test_config5_full_launch_all_models(ctx, cfg5, scale):
    wl = parity.make_cached(5, scale)
    say(f"config 5 full launch, slo x{scale}, all {wl.n_models} models")
    sc, got = run_gpu(wl, ctx)
    ora = oracle.score_workload(wl, threads=ORACLE_THREADS)
    err = parity.compare(wl, got, ora)
    say("  max errors", err)
    P = got["finish_prob"]
    assert np.all((P >= 0) & (P <= 1))
    # the state is not a trivial one: members can finish, models pick batches
    assert (P > 0).mean() > 0.1 and (got["sel_n"] > 0).mean() > 0.9
    assert np.all(got["expected_latency_ms"] >= 0.5 * wl.bin_width_ms[0] * (1 - 1e-6))
    if scale > 1.0:
        assert ((P > 0) & (P < 1)).mean() > 0.3


def test_config5_trimmed_and_full_reads_agree(ctx, cfg5):
    wl = cfg5.subset(list(range(0, 128, 16)))
    say("config 5, 8 models, trim on/off")
    _, on = run_gpu(wl, ctx, trim=True)
    _, off = run_gpu(wl, ctx, trim=False)
    assert_same_bits(on, off)


# ---------------------------------------------------------------- errors and plumbing
def test_device_data_errors_are_reported(ctx):
    wl = W.random_case(40, n_models=1, queue_lens=[6])
    for mutate, _ in [(lambda w: w.cls.__setitem__(2, 99), "class"),
                      (lambda w: w.deadline_ms.__setitem__(3, np.nan), "nan"),
                      (lambda w: w.deadline_ms.__setitem__(1, w.deadline_ms[1] + 1e6), "order")]:
        w2 = W.random_case(40, n_models=1, queue_lens=[6])
        mutate(w2)
        sc = O.Scorer(w2, ctx)
        sc.build()
        sc.score()
        sc.select()
        with pytest.raises(O.OrlojError) as ei:
            ctx.sync()
        assert ei.value.code == O.ORLOJ_E_DATA
    ctx.sync()


def test_prefix_limit_is_unsupported(ctx):
    wl = W.random_case(41, n_models=1, queue_lens=[300], batch_sizes=(1, 300))
    sc = O.Scorer(wl, ctx)
    sc.build()
    with pytest.raises(O.OrlojError) as ei:
        sc.score()
    assert ei.value.code == O.ORLOJ_E_UNSUPPORTED


def test_side_stream(ctx):
    wl = W.random_case(42, n_models=2, queue_lens=[10, 12])
    s = torch.cuda.Stream()
    c2 = O.Context(stream=s)
    with torch.cuda.stream(s):
        sc = O.Scorer(wl, c2)
        got = sc.run()
    parity.compare(wl, got, oracle.score_workload(wl))


def test_native_library_is_loaded(ctx):
    with open("/proc/self/maps") as f:
        maps = f.read()
    assert os.path.basename(O.LIB_PATH) in maps


# ---------------------------------------------------------------- miss costs
@pytest.mark.parametrize("case", [RANDOM_CASES[i] for i in (0, 1, 5, 7, 14)],
                         ids=lambda c: f"seed{c['seed']}")
def test_cost_weighted_scores(ctx, case):
    import dataclasses
    say("costs", case)
    wl = W.random_case(**case)
    r = np.random.default_rng(100 + case["seed"])
    wl = dataclasses.replace(wl, cost=r.uniform(0.0, 4.0, size=wl.cls.size))
    sc, got = run_gpu(wl, ctx)
    parity.compare(wl, got, oracle.score_workload(wl))
    _, untrimmed = run_gpu(wl, ctx, trim=False)
    assert_same_bits(got, untrimmed)


def test_negative_cost_is_a_data_error(ctx):
    import dataclasses
    wl = W.random_case(43, n_models=1, queue_lens=[5])
    cost = np.ones(5)
    cost[2] = -1.0
    sc = O.Scorer(dataclasses.replace(wl, cost=cost), ctx)
    sc.build()
    sc.score()
    with pytest.raises(O.OrlojError) as ei:
        ctx.sync()
    assert ei.value.code == O.ORLOJ_E_DATA
