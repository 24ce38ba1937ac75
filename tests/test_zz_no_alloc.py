"""The allocation-free affine scorer (orloj_score_candidates_affine_noalloc)
against the allocating one (orloj_score_candidates_affine), through the C
ABI: two calls in a row on one context, the second with a smaller input,
each giving the allocating entry point's outputs bit for bit (the same
kernels; the panel sums only live in another buffer), and the first also
checked against the oracle.  A call whose panel sums exceed the fixed
scratch is refused before any launch."""
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


def outputs(sc, noalloc):
    sc.score(noalloc=noalloc)
    sc.select()
    sc.ctx.sync()
    return sc.fetch()


def same_bits(a, b):
    for k in a:
        assert np.array_equal(np.asarray(a[k]).view(np.uint8), np.asarray(b[k]).view(np.uint8)), k


def test_noalloc_matches_the_allocating_entry_point():
    ctx = O.Context()
    large = W.random_affine(80, n_models=7, queue_lens=[64, 30, 64, 1, 0, 50, 9], n_bins=5000,
                            batch_sizes=(1, 8, 33, 64))
    small = W.random_affine(81, n_models=2, queue_lens=[5, 12], n_bins=300,
                            batch_sizes=(1, 2, 4, 16))
    for name, wl in (("large", large), ("small", small)):
        say(f"noalloc: {name} ({wl.n_models} models, {wl.n_bins} bins)")
        sc = O.Scorer(wl, ctx)
        sc.build()
        ctx.sync()
        got = outputs(sc, noalloc=True)
        ref = outputs(sc, noalloc=False)
        same_bits(got, ref)
        if name == "large":
            parity.compare(wl, got, oracle.score_workload_affine(wl, wl.c0_ms, wl.c1))
    # and again in the other order on the same context: the scratch keeps the
    # last call's contents, which no call reads before writing
    sc = O.Scorer(large, ctx)
    sc.build()
    ref = outputs(sc, noalloc=False)
    same_bits(outputs(sc, noalloc=True), ref)


def test_noalloc_refuses_calls_beyond_its_scratch():
    ctx = O.Context()
    # 513 models x 32 panels (8192 bins) x 256-member prefixes > 2^20 floats
    wl = W.random_affine(82, n_models=513, queue_lens=[256] * 513, n_bins=8192, n_classes=2,
                         batch_sizes=(1, 256))
    sc = O.Scorer(wl, ctx)
    sc.build()
    ctx.sync()
    with pytest.raises(O.OrlojError) as ei:
        sc.score(noalloc=True)
    assert ei.value.code == O.ORLOJ_E_UNSUPPORTED
    assert "scratch" in str(ei.value)
    ctx.sync()
