"""Chunked scoring: a (model, batch size) pair's prefix lengths split over
several workgroups, each rebuilding the batch CDF of the prefixes before its
chunk with warm-up steps.  Every chunk size must give the bits of the
unsplit launch (the same fma sequence per bin), in both batch laws and both
prefix modes; the automatic choice is checked against the oracle as well.
Tabulated rows of more than two panels take every panel's E sums from the
emax_kernel pre-pass when the launch is chunked (the chunks then repeat only
the member panels): those cases must give the unsplit bits too."""
import dataclasses
import sys

import numpy as np
import pytest

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
    c = O.Context()
    yield c
    c.set_score_chunk(-1)


def run(wl, ctx, chunk, mode=0, trim=True):
    ctx.set_score_chunk(chunk)
    try:
        return O.Scorer(wl, ctx, prefix_mode=mode, trim=trim).run(build=True)
    finally:
        ctx.set_score_chunk(-1)


def same_bits(a, b):
    for k in a:
        assert np.array_equal(np.asarray(a[k]).view(np.uint8), np.asarray(b[k]).view(np.uint8)), k


CASES = [
    dict(seed=0),
    dict(seed=1, n_models=3, queue_lens=[0, 7, 13], batch_sizes=(1, 4, 16)),
    dict(seed=2, n_bins=2500, n_classes=4, queue_lens=[64, 40], batch_sizes=(1, 8, 33, 64),
         tau_range=(-20.0, 3000.0)),
    dict(seed=3, n_bins=4096, n_classes=6, queue_lens=[70, 64], batch_sizes=(16, 64),
         tau_range=(-5.0, 6000.0)),
    dict(seed=4, n_bins=300, sparsity=0.9, total=3, queue_lens=[50, 20]),
    dict(seed=5, n_bins=64, tau_range=(-50.0, -1.0), queue_lens=[30, 30]),     # all dead
    dict(seed=6, n_bins=64, tau_range=(500.0, 900.0), queue_lens=[30, 30]),    # beyond the grid
    dict(seed=7, n_models=1, n_bins=100, queue_lens=[200], batch_sizes=(128, 200)),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"seed{c['seed']}")
@pytest.mark.parametrize("law", ["tabulated", "affine"])
def test_every_chunk_size_gives_the_same_bits(ctx, case, law):
    say("chunks", law, case)
    wl = W.random_case(**case) if law == "tabulated" else W.random_affine(**case)
    ref = run(wl, ctx, 0)
    for ch in (1, 3, 8, 16, 32, -1):
        same_bits(run(wl, ctx, ch), ref)


@pytest.mark.parametrize("seed", [20, 21])
def test_rect_mode_chunks(ctx, seed):
    wl = W.random_case(seed, n_models=2, queue_lens=[90, 33], batch_sizes=(1, 8, 40),
                       n_bins=1500, tau_range=(-10.0, 1800.0))
    ref = run(wl, ctx, 0, mode=1)
    for ch in (7, 16, 64):
        same_bits(run(wl, ctx, ch, mode=1), ref)


def test_trimming_off_chunks(ctx):
    wl = W.random_case(30, n_models=2, queue_lens=[64, 50], batch_sizes=(2, 32, 64),
                       n_bins=3000, tau_range=(-10.0, 4000.0))
    ref = run(wl, ctx, 0, trim=False)
    same_bits(run(wl, ctx, 8, trim=False), ref)
    same_bits(run(wl, ctx, 8, trim=True), ref)


def test_chunked_against_the_oracle(ctx):
    wl = W.make(2, slo_scale=3.0)
    got = run(wl, ctx, 8)
    err = parity.compare(wl, got, oracle.score_workload(wl))
    say("  cfg2 x3, chunks of 8: max errors", err)


def test_config5_models_chunked(ctx):
    # eight models of the saturated state (four 1024-bin panels, 64 batch sizes)
    wl = W.make(5, models=[0, 17, 33, 50, 71, 90, 111, 127], workers=8)
    ref = run(wl, ctx, 0)
    for ch in (8, 16, 32, -1):
        same_bits(run(wl, ctx, ch), ref)
    aw = W.affine(wl)
    ref = run(aw, ctx, 0)
    same_bits(run(aw, ctx, 16), ref)


def test_small_config5_launch_against_the_oracle(ctx):
    # the scheduling loop's shape: a few idle models, every batch size; the
    # automatic choice chunks it and takes the E sums from the pre-pass
    wl = W.make(5, models=[5, 64], workers=8, slo_scale=2.0)
    got = run(wl, ctx, -1)
    err = parity.compare(wl, got, oracle.score_workload(wl))
    say("  cfg5, 2 models, automatic chunks: max errors", err)
    same_bits(got, run(wl, ctx, 0))


def test_bad_chunk_is_rejected(ctx):
    with pytest.raises(O.OrlojError) as ei:
        ctx.set_score_chunk(-2)
    assert ei.value.code == O.ORLOJ_E_INVALID
