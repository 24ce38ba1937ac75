"""Affine batch-latency mode (§4.2.1 Eq. (3), (5); §4.2.2 Eq. (9)) on the GPU
against the CPU oracle, through the C ABI.

A batch of size s whose slowest member takes l runs c0 + c1 s l, so one
solo-latency table per class serves every batch size.  Random ragged cases
(the same shapes as the tabulated mode's), both prefix modes, a sweep of the
delay rate b, miss costs, configurations 1-4 at full size with their affine
constants, configuration 5's full launch with every model compared, the
reduction to the tabulated path at c0 = 0, c1 s = 1, and the data-error path.
"""
import ctypes
import dataclasses
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


def run_gpu(wl, ctx, mode=0, trim=True):
    sc = O.Scorer(wl, ctx, prefix_mode=mode, trim=trim)
    return sc, sc.run(build=True)


ORACLE_THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


def run_oracle(wl, mode=0, models=None, threads=1):
    sub = wl if models is None else wl.subset(models)
    return oracle.score_workload_affine(sub, sub.c0_ms, sub.c1, prefix_mode=mode, threads=threads)


def assert_same_bits(a, b):
    for k in a:
        assert np.array_equal(a[k].view(np.uint8), b[k].view(np.uint8)), k


CASES = [
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
    dict(seed=12, n_bins=64, tau_range=(5000.0, 9000.0)),       # all beyond the grid
    dict(seed=13, n_bins=300, sparsity=0.9, total=3),
    dict(seed=14, n_bins=2048, queue_lens=[128, 100], batch_sizes=tuple(range(1, 129, 9))),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"seed{c['seed']}")
def test_random_affine_cases(ctx, case):
    say("affine random case", case)
    wl = W.random_affine(**case)
    _, got = run_gpu(wl, ctx)
    err = parity.compare(wl, got, run_oracle(wl))
    say("  max errors", err)


def test_time_left_below_c0_is_dead(ctx):
    # every deadline lies after now but before c0: nothing can finish
    wl = W.random_affine(15, n_bins=50, tau_range=(0.5, 4.0), c0_range=(5.0, 6.0))
    _, got = run_gpu(wl, ctx)
    parity.compare(wl, got, run_oracle(wl))
    assert np.all(got["finish_prob"] == 0.0) and np.all(got["score"] == 0.0)
    assert np.all(got["sel_n"] == 0)


@pytest.mark.parametrize("case", [CASES[i] for i in (0, 5, 6, 8, 13, 14)],
                         ids=lambda c: f"seed{c['seed']}")
def test_support_trimming_changes_no_bits(ctx, case):
    say("affine trim on/off", case)
    wl = W.random_affine(**case)
    _, on = run_gpu(wl, ctx, trim=True)
    _, off = run_gpu(wl, ctx, trim=False)
    assert_same_bits(on, off)


@pytest.mark.parametrize("seed", [20, 21])
def test_rect_mode(ctx, seed):
    say("affine rect", seed)
    wl = W.random_affine(seed, n_models=2, queue_lens=[9, 30], batch_sizes=(1, 4, 8), n_bins=200)
    _, got = run_gpu(wl, ctx, mode=1)
    parity.compare(wl, got, run_oracle(wl, mode=1), mode=1)


@pytest.mark.parametrize("b", [1e-6, 1e-4, 1e-2, 1e-1])
def test_delay_rate_sweep(ctx, b):
    say("affine b sweep", b)
    wl = W.random_affine(30, n_models=2, queue_lens=[40, 25], batch_sizes=(1, 2, 4, 8, 16, 32),
                         n_bins=512, b_expo=b, tau_range=(0.0, 700.0))
    _, got = run_gpu(wl, ctx)
    parity.compare(wl, got, run_oracle(wl))


@pytest.mark.parametrize("case", [CASES[i] for i in (0, 5, 14)], ids=lambda c: f"seed{c['seed']}")
def test_cost_weighted_scores(ctx, case):
    say("affine costs", case)
    wl = W.random_affine(**case)
    r = np.random.default_rng(200 + case["seed"])
    wl = dataclasses.replace(wl, cost=r.uniform(0.0, 4.0, size=wl.cls.size))
    _, got = run_gpu(wl, ctx)
    parity.compare(wl, got, run_oracle(wl))


def same_but_scores(tab, aff):
    # P comes from the same products: the same bits.  The affine path reads
    # its bins in narrower panels, so members are grouped into other panel
    # passes: the expected finish count adds the same fp64 terms in another
    # order (equal to rounding), and a priority's discounted prefix is summed
    # in another order (the scores agree to rounding).  E[L_B] adds its
    # per-panel sums of 1 - G, each rounded to fp32 (at most 2^-25 of the
    # panel's sum, all terms >= 0), over other panels: the two sums differ
    # by at most 2^-24 of the total, and each E[L_B] is then rounded to fp32
    # once more (2^-24 each way).
    assert np.array_equal(tab["finish_prob"].view(np.uint8), aff["finish_prob"].view(np.uint8))
    assert np.allclose(aff["expected_latency_ms"], tab["expected_latency_ms"], rtol=3 * 2.0**-24, atol=0)
    assert np.allclose(aff["expected_finish"], tab["expected_finish"], rtol=1e-13, atol=1e-15)
    assert np.allclose(aff["score"], tab["score"], rtol=2e-6, atol=1e-12)
    assert np.array_equal(aff["sel_n"], tab["sel_n"]) and np.array_equal(aff["sel_bs"], tab["sel_bs"])


def test_reduces_to_tabulated_path(ctx):
    # c0 = 0 and c1 s = 1 at every batch size: the affine path must give the
    # tabulated path's results on the same tables (one batch size, s = 1)
    base = W.random_case(50, n_models=2, queue_lens=[1, 1], batch_sizes=(1,), n_bins=700)
    tab = dataclasses.replace(base, counts=np.ascontiguousarray(base.counts[:, :1]))
    aff = dataclasses.replace(base, counts=np.ascontiguousarray(base.counts[:, 0]),
                              c0_ms=np.zeros(2), c1=np.ones(2))
    _, g_tab = run_gpu(tab, ctx)
    _, g_aff = run_gpu(aff, ctx)
    same_but_scores(g_tab, g_aff)
    # and with s = 4, c1 = 1/4 the bin width c1 s w equals w exactly; at 256
    # bins or fewer both paths read 4 bins per lane: every bit agrees
    base = W.random_case(51, n_models=1, queue_lens=[4], batch_sizes=(4,), n_bins=250)
    tab = dataclasses.replace(base, counts=np.ascontiguousarray(base.counts[:, :1]))
    aff = dataclasses.replace(base, counts=np.ascontiguousarray(base.counts[:, 0]),
                              c0_ms=np.zeros(1), c1=np.full(1, 0.25))
    _, g_tab = run_gpu(tab, ctx)
    _, g_aff = run_gpu(aff, ctx)
    assert_same_bits(g_tab, g_aff)
    # rows of several panels (members homed in different panels; E[max] of
    # the affine path comes from per-panel sums formed once per prefix
    # length): c1 s = 1 exactly at s = 8 and s = 2
    for seed, K, s, c1 in [(52, 2500, 8, 0.125), (53, 2048, 2, 0.5), (54, 5000, 4, 0.25)]:
        base = W.random_case(seed, n_models=2, queue_lens=[s, s - 1], batch_sizes=(s,),
                             n_bins=K, tau_range=(-10.0, 1.1 * K))
        tab = dataclasses.replace(base, counts=np.ascontiguousarray(base.counts[:, :1]))
        aff = dataclasses.replace(base, counts=np.ascontiguousarray(base.counts[:, 0]),
                                  c0_ms=np.zeros(2), c1=np.full(2, c1))
        _, g_tab = run_gpu(tab, ctx)
        _, g_aff = run_gpu(aff, ctx)
        same_but_scores(g_tab, g_aff)


def test_scratch_grows_and_is_reused(ctx):
    # the context's scratch for the per-panel sums grows for a larger call
    # and still serves a smaller one after it, with the same bits as before
    small = W.random_affine(70, n_models=1, queue_lens=[5], n_bins=100)
    large = W.random_affine(71, n_models=6, queue_lens=[64, 30, 64, 1, 0, 50], n_bins=5000,
                            batch_sizes=(1, 8, 64))
    runs = []
    for wl in (small, large, small):
        _, got = run_gpu(wl, ctx)
        parity.compare(wl, got, run_oracle(wl))
        runs.append(got)
    assert_same_bits(runs[0], runs[2])


def test_stream_switch_keeps_results():
    c = O.Context()
    wl = W.random_affine(73, n_models=3, queue_lens=[9, 40, 17], n_bins=3000)
    _, first = run_gpu(wl, c)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        c.set_stream(s)
        _, second = run_gpu(wl, c)
        torch.cuda.synchronize()
    c.set_stream(torch.cuda.current_stream())
    assert_same_bits(first, second)


@pytest.mark.parametrize("cid,scale", [(1, 1.0), (1, 4.0), (2, 1.0), (2, 3.0), (3, 1.0),
                                       (3, 3.0), (3, 5.0), (4, 1.0), (4, 3.0)])
def test_config_full_size(ctx, cid, scale):
    say(f"affine config {cid} slo x{scale}")
    wl = W.affine(parity.make_cached(cid, scale))
    _, got = run_gpu(wl, ctx)
    err = parity.compare(wl, got, run_oracle(wl))
    say("  max errors", err, "P > 0:", float((got["finish_prob"] > 0).mean()))
    if scale > 1.0:     # relaxed SLOs: the comparison is not a trivial one
        P = got["finish_prob"]
        assert int((P > 0).sum()) >= min(1000, P.size // 2) and np.all(got["sel_n"] > 0)


@pytest.mark.parametrize("scale", [1.0, 4.0])
def test_config5_full_launch_all_models(ctx, scale):
    say(f"affine config 5 full launch, slo x{scale}, all models")
    wl = W.affine(parity.make_cached(5, scale))
    sc, got = run_gpu(wl, ctx)
    err = parity.compare(wl, got, run_oracle(wl, threads=ORACLE_THREADS))
    say("  max errors", err)
    P = got["finish_prob"]
    assert np.all((P >= 0) & (P <= 1))
    # the state is not a trivial one: members can finish, models pick batches
    assert (P > 0).mean() > 0.1 and (got["sel_n"] > 0).mean() > 0.9
    # E[L_B] >= c0 + c1 s w / 2 for every candidate
    for q in range(wl.n_models):
        a, b = sc.h_cand_off[q], sc.h_cand_off[q + 1]
        s = np.concatenate([np.full(min(int(x), wl.queue_len(q)), int(x)) for x in wl.batch_sizes])
        lo = wl.c0_ms[q] + wl.c1[q] * s * wl.bin_width_ms[q] * 0.5
        assert np.all(got["expected_latency_ms"][a:b] >= lo * (1 - 1e-6))


def test_invalid_constants_are_a_data_error(ctx):
    wl = W.random_affine(60, n_models=2, queue_lens=[5, 5])
    for c0, c1 in [((-1.0, 1.0), (0.5, 0.5)), ((1.0, 1.0), (0.0, 0.5)),
                   ((np.inf, 1.0), (0.5, 0.5)), ((1.0, 1.0), (np.nan, 0.5))]:
        w2 = dataclasses.replace(wl, c0_ms=np.asarray(c0), c1=np.asarray(c1))
        sc = O.Scorer(w2, ctx)
        sc.build()
        sc.score()
        with pytest.raises(O.OrlojError) as ei:
            ctx.sync()
        assert ei.value.code == O.ORLOJ_E_DATA
        assert "affine" in str(ei.value)
        # the bad model's requests score as dead
        P = sc.finish_prob[sc.h_prob_off[0]:sc.h_prob_off[1]].cpu().numpy()
        assert np.all(P == 0.0)
    ctx.sync()


def test_null_constants_are_rejected(ctx):
    wl = W.random_affine(61, n_models=1, queue_lens=[3])
    sc = O.Scorer(wl, ctx)
    sc.build()
    rc = ctx.L.orloj_score_candidates_affine(
        ctx.ctx, ctypes.byref(sc.grid), O._ptr(sc.ccdf), None, None, None,
        ctypes.byref(sc.queues), 1e-4, 0, O._ptr(sc.d_cand_off), O._ptr(sc.d_prob_off),
        O._ptr(sc.finish_prob), O._ptr(sc.expected_finish), O._ptr(sc.expected_latency),
        O._ptr(sc.score_out))
    assert rc == O.ORLOJ_E_INVALID
    torch.cuda.synchronize()
