"""Deterministic edge cases of Eq. (2) and of the selection, through the C ABI
against the oracle.

- Deadlines exactly on the grid's milestones (§4.1 Eq. (2): the integral
  splits at the bin edges l_1, l_2): time left 0 (dead), exactly k w for
  k = 1, 2, the last and first bins of each panel the kernels sweep (bins
  1024 apart in the tabulated mode, 256 apart in the affine mode's score
  waves), the grid's end K w (beyond the grid), and one ulp below each of
  them; runs of equal deadlines.  Tabulated and affine batch laws, both
  prefix modes, every step-chunk setting giving the unsplit bits.
- The selection's tie rules (§3.2 Algorithm 1 pops one batch; equal scores
  go to the larger prefix, then to the smaller batch size): exact ties are
  built on purpose and the GPU's pick is asserted, not merely checked to
  score within the bar.
- Coherent rounding of the expected finish count: 256 members of one class
  whose deadlines share one bin, with the batch CDF near 1/e there, where
  every member reads the same two values of G.
"""
import dataclasses
import sys

import numpy as np
import pytest

import oracle
import parity
from paper_2209_00159_amd import workloads as W

TOTAL = 1_000_003          # histogram samples: not a power of two, so 1 - F rounds


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def decaying_counts(rng, B, C, K, total=TOTAL):
    """[B, C, K] counts: class c at batch size b has an exponential profile
    of scale L (log-uniform in [0.5, K] bins), all of it on the grid.  Short
    scales leave most bins empty, so the support trimming is exercised."""
    k = np.arange(K + 1, dtype=np.float64)
    out = np.zeros((B, C, K), np.uint32)
    for b in range(B):
        for c in range(C):
            L = float(np.exp(rng.uniform(np.log(0.5), np.log(K))))
            cdf = -np.expm1(-k / L)
            cdf /= cdf[-1]
            cum = np.rint(cdf * total)
            cum[0], cum[-1] = 0.0, float(total)
            out[b, c] = np.diff(np.maximum.accumulate(cum)).astype(np.uint32)
    return out


def milestone_deadlines(now, width, ks, repeats=(), below=True):
    """now + k width for every k (exact in binary when now and width are),
    one ulp below each milestone k >= 1, and `repeats` extra copies of the
    listed k (equal deadlines keep the caller's order)."""
    d = [now + k * width for k in ks]
    if below:
        d += [np.nextafter(now + k * width, -np.inf) for k in ks if k >= 1]
    for k, r in repeats:
        d += [now + k * width] * r
    return np.sort(np.asarray(d, np.float64), kind="stable")


def explicit_workload(name, counts, batch_sizes, width, queues, nows, cost=None,
                      b_expo=W.DEFAULT_B_EXPO):
    """counts [M, B, C, K]; queues[q] = (cls, deadline_ms), deadlines sorted."""
    M, B, C, K = counts.shape
    offs = np.zeros(M + 1, np.int64)
    for q, (c, _) in enumerate(queues):
        offs[q + 1] = offs[q] + len(c)
    return W.Workload(
        name, 0, M, C, K, np.asarray(batch_sizes, np.int32),
        np.asarray(width, np.float64).reshape(M), np.ascontiguousarray(counts), offs,
        np.concatenate([np.asarray(c, np.int32) for c, _ in queues]),
        np.concatenate([np.asarray(d, np.float64) for _, d in queues]),
        np.asarray(nows, np.float64), b_expo=b_expo,
        cost=None if cost is None else np.asarray(cost, np.float64))


# Tabulated milestone cases: (K, milestones).  The tabulated kernel sweeps
# 16 bins per lane at K >= 1024 (panels of 1024 bins), 4 bins per lane at
# K = 256 (one panel), and a ragged last panel at K = 3000.
TAB_CASES = [
    (4096, [0, 1, 2, 3, 1022, 1023, 1024, 1025, 1026, 2046, 2047, 2048, 2049, 3071, 3072,
            3073, 4094, 4095, 4096, 5000], [(0, 3), (1024, 3), (2048, 2), (4096, 2)]),
    (3000, [0, 1, 2, 1023, 1024, 1025, 2047, 2048, 2049, 2998, 2999, 3000, 3001], [(1025, 4)]),
    (256, [0, 1, 2, 3, 4, 5, 127, 128, 254, 255, 256, 300], [(2, 5)]),
    (8192, [0, 1, 1023, 1024, 1025, 4095, 4096, 4097, 7167, 7168, 7169, 8191, 8192],
     [(7168, 40), (8192, 20)]),
]


def tab_case(i, seed=0, mode=0):
    K, ks, reps = TAB_CASES[i]
    rng = np.random.default_rng([seed, i, K])
    now, w = 1000.0, 0.25
    d = milestone_deadlines(now, w, ks, reps)
    C = 4
    bs = (1, 2, 16, int(d.size)) if mode == 0 else (1, 5, 16)
    counts = decaying_counts(rng, len(bs), C, K)[None]
    cls = rng.integers(0, C, size=d.size)
    return explicit_workload(f"milestones-K{K}", counts, bs, [w], [(cls, d)], [now])


def affine_case(seed=0, below=True, K=4096):
    """Milestones on every batch size's own grid: bins c1 s w wide, time left
    tau - c0 (the affine score waves sweep 4 bins per lane: panels of 256)."""
    rng = np.random.default_rng([seed, 77])
    now, w, c0, c1 = 1000.0, 0.25, 0.5, 0.125
    bs = (1, 8, 64)
    ks = [0, 1, 2, 255, 256, 257, 511, 512, 1023, 1024, 1025, 4095, 4096]
    d = np.sort(np.concatenate([milestone_deadlines(now + c0, c1 * s * w, ks, below=below)
                                for s in bs]), kind="stable")
    C = 3
    counts = decaying_counts(rng, 1, C, K)[None]
    cls = rng.integers(0, C, size=d.size)
    wl = explicit_workload("milestones-affine", counts, bs + (max(65, int(d.size)),), [w],
                           [(cls, d)], [now])
    return dataclasses.replace(wl, counts=np.ascontiguousarray(counts[:, 0]),
                               c0_ms=np.array([c0]), c1=np.array([c1]))


def test_milestone_cases_sit_on_the_milestones():
    """The case builders put time-to-deadline / bin width exactly on the
    integers they name (fp64, as both sides compute it)."""
    for i in range(len(TAB_CASES)):
        wl = tab_case(i)
        K, ks, _ = TAB_CASES[i]
        u = (wl.deadline_ms - wl.now_ms[0]) / wl.bin_width_ms[0]
        for k in ks:
            assert np.any(u == k), (K, k)
            if k >= 1:
                assert np.any((u < k) & (u > k - 1e-9)), (K, k)
    aw = affine_case()
    tau = aw.deadline_ms - aw.now_ms[0] - aw.c0_ms[0]
    for s in (1, 8, 64):
        u = tau / (aw.c1[0] * s * aw.bin_width_ms[0])
        for k in (0, 1, 256, 1024, 4096):
            assert np.any(u == k), (s, k)


def test_tie_cases_tie_on_the_oracle():
    """The oracle side of the tie cases below: the scores tie exactly and the
    oracle's own pick follows the rule."""
    wl, n_star, s_star = prefix_tie_case(0)
    o = oracle.score_workload(wl)
    S = o["score"]
    cands = parity.candidates(wl, 0, 0)
    i = cands.index((n_star, s_star))
    assert S[i + 1] == S[i] and cands[i + 1] == (n_star + 1, s_star)
    assert (int(o["sel_n"][0]), int(o["sel_bs"][0])) == (n_star + 1, s_star)
    wl = batch_size_tie_case(0)
    o = oracle.score_workload(wl)
    S = o["score"].reshape(3, -1)
    assert np.array_equal(S[0], S[1]) and np.array_equal(S[0], S[2])
    assert int(o["sel_bs"][0]) == 4


# ---------------------------------------------------------------- ties
def batch_size_tie_case(seed):
    """Batch sizes 4, 8, 16 with the same table and a queue of 4: every
    prefix scores the same at every batch size."""
    rng = np.random.default_rng([seed, 5])
    K, C = 300, 3
    one = decaying_counts(rng, 1, C, K)[0]
    counts = np.repeat(one[None, None], 3, axis=1)
    now, w = 500.0, 0.5
    d = np.sort(now + rng.uniform(20.0, 140.0, size=4))
    cls = rng.integers(0, C, size=4)
    return explicit_workload("bs-tie", counts, (4, 8, 16), [w], [(cls, d)], [now])


def prefix_tie_case(seed):
    """A random queue, then one more member right after the oracle's best
    prefix n*: the same deadline as member n*, cost 0, and a class whose
    latency always falls in bin 0.  The batch CDF is unchanged at every grid
    point (F = 1 from x_1 on) and the new member adds priority 0, so prefix
    n* + 1 scores exactly as n* does.  Returns (workload, n*, s*) for a seed
    whose n* < s* (the longer prefix is a candidate at the same size)."""
    for t in range(64):
        rng = np.random.default_rng([seed, 9, t])
        K, C = 400, 4
        bs = (2, 6, 12)
        counts = decaying_counts(rng, len(bs), C + 1, K)
        counts[:, C] = 0
        counts[:, C, 0] = 17                       # class C: all mass in bin 0
        now, w = 200.0, 0.5
        N = 10
        d = np.sort(now + rng.uniform(5.0, 180.0, size=N))
        cls = rng.integers(0, C, size=N)
        wl = explicit_workload("n-tie", counts[None], bs, [w], [(cls, d)], [now],
                               cost=np.ones(N))
        o = oracle.score_workload(wl)
        n_star, s_star = int(o["sel_n"][0]), int(o["sel_bs"][0])
        if n_star == 0 or n_star >= s_star:
            continue
        S = sorted(o["score"], reverse=True)
        if S[0] - S[1] < 1e-4:                     # a clear best before the insertion
            continue
        cls2 = np.insert(cls, n_star, C)
        d2 = np.insert(d, n_star, d[n_star - 1])
        cost2 = np.insert(np.ones(N), n_star, 0.0)
        return (explicit_workload("n-tie", counts[None], bs, [w], [(cls2, d2)], [now],
                                  cost=cost2), n_star, s_star)
    raise AssertionError("no seed gives n* < s*")


# ---------------------------------------------------------------- coherent E
def coherent_case(n=256, theta=0.5, batch_sizes=(64, 256)):
    """n requests of one class, all with the same deadline inside bin k0,
    and F at the bin's edges near exp(-1/n), so that G = F^n is near 1/e
    there.  The counts around the edges are chosen so that 1 - F rounds to
    float32 with an error close to half an ulp (the worst case for the
    table's single rounding), with the same sign at both edges."""
    K, k0 = 64, 40
    T = TOTAL
    target = np.exp(-1.0 / n)

    def worst_cum(f):
        c0 = int(round(f * T))
        best, cbest = -1.0, c0
        for c in range(c0 - 15, c0 + 16):
            t = (T - c) / T
            t32 = float(np.float32(t))
            ulp = float(np.spacing(np.float32(t)))
            e = (t32 - t) / ulp            # the same sign at both edges
            if e > best:
                best, cbest = e, c
        return cbest

    cum = np.zeros(K + 1, np.int64)
    lo_c = worst_cum(target - 4e-5)
    hi_c = worst_cum(target + 4e-5)
    cum[1:k0 + 1] = np.rint(np.linspace(0, lo_c, k0 + 1)[1:]).astype(np.int64)
    cum[k0] = lo_c
    cum[k0 + 1] = hi_c
    cum[k0 + 2:] = np.rint(np.linspace(hi_c, T, K - k0)[1:]).astype(np.int64)
    cum[K] = T
    row = np.diff(cum).astype(np.uint32)
    counts = np.repeat(row[None, None, None], len(batch_sizes), axis=1)   # [1, B, 1, K]
    now, w = 100.0, 0.5
    d = np.full(n, now + (k0 + theta) * w)
    return explicit_workload(f"coherent-n{n}", counts, batch_sizes, [w],
                             [(np.zeros(n, np.int32), d)], [now])


# ---------------------------------------------------------------- GPU tests
gpu = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    from paper_2209_00159_amd import orloj as O
    return O.Context()


def run_gpu(wl, ctx, mode=0, trim=True, chunk=-1):
    from paper_2209_00159_amd import orloj as O
    ctx.set_score_chunk(chunk)
    try:
        sc = O.Scorer(wl, ctx, prefix_mode=mode, trim=trim)
        return sc, sc.run(build=True)
    finally:
        ctx.set_score_chunk(-1)


def same_bits(a, b):
    for k in a:
        assert np.array_equal(a[k].view(np.uint8), b[k].view(np.uint8)), k


@gpu
@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("i", range(len(TAB_CASES)))
def test_tabulated_milestones(ctx, i, mode):
    wl = tab_case(i, mode=mode)
    say(f"milestones K={wl.n_bins} mode={mode} members={wl.cls.size} bs={wl.batch_sizes.tolist()}")
    _, got = run_gpu(wl, ctx, mode=mode)
    err = parity.compare(wl, got, oracle.score_workload(wl, prefix_mode=mode), mode=mode)
    say("  max errors", err)
    for ch in (0, 3, 8):
        _, g2 = run_gpu(wl, ctx, mode=mode, chunk=ch)
        same_bits(got, g2)
    _, g3 = run_gpu(wl, ctx, mode=mode, trim=False)
    same_bits(got, g3)


@gpu
@pytest.mark.parametrize("below", [True, False])
@pytest.mark.parametrize("mode", [0, 1])
def test_affine_milestones(ctx, below, mode):
    aw = affine_case(below=below)
    say(f"affine milestones below={below} mode={mode} members={aw.cls.size}")
    _, got = run_gpu(aw, ctx, mode=mode)
    ora = oracle.score_workload_affine(aw, aw.c0_ms, aw.c1, prefix_mode=mode)
    err = parity.compare(aw, got, ora, mode=mode)
    say("  max errors", err)
    for ch in (0, 8):
        _, g2 = run_gpu(aw, ctx, mode=mode, chunk=ch)
        same_bits(got, g2)


@gpu
@pytest.mark.parametrize("seed", range(4))
def test_batch_size_tie_goes_to_the_smaller_size(ctx, seed):
    wl = batch_size_tie_case(seed)
    _, got = run_gpu(wl, ctx)
    ora = oracle.score_workload(wl)
    parity.compare(wl, got, ora)
    S = got["score"].reshape(3, -1)
    assert np.array_equal(S[0].view(np.uint32), S[1].view(np.uint32))
    assert np.array_equal(S[0].view(np.uint32), S[2].view(np.uint32))
    n_o = int(ora["sel_n"][0])
    assert n_o > 0 and int(ora["sel_bs"][0]) == 4
    assert (int(got["sel_n"][0]), int(got["sel_bs"][0])) == (n_o, 4)


@gpu
@pytest.mark.parametrize("seed", range(4))
def test_prefix_tie_goes_to_the_longer_prefix(ctx, seed):
    wl, n_star, s_star = prefix_tie_case(seed)
    _, got = run_gpu(wl, ctx)
    ora = oracle.score_workload(wl)
    parity.compare(wl, got, ora)
    cands = parity.candidates(wl, 0, 0)
    i = cands.index((n_star, s_star))
    assert got["score"][i] == got["score"][i + 1] > 0
    assert (int(got["sel_n"][0]), int(got["sel_bs"][0])) == (n_star + 1, s_star)


@gpu
@pytest.mark.parametrize("n,theta,bs", [(256, 0.5, (64, 256)), (256, 0.0, (256,)),
                                        (64, 0.5, (64,)), (200, 0.25, (1, 200))])
def test_coherent_expected_finish(ctx, n, theta, bs):
    wl = coherent_case(n, theta, bs)
    _, got = run_gpu(wl, ctx)
    ora = oracle.score_workload(wl)
    dE = np.abs(got["expected_finish"] - ora["expected_finish"])
    G = ora["finish_prob"][-n:]
    say(f"coherent n={n} theta={theta}: P of the longest prefix {G[0]:.6f}, "
        f"max |dE| {dE.max():.3e} at candidate {int(dE.argmax())}")
    parity.compare(wl, got, ora)


# ---------------------------------------------------------------------------
# The E-only loop's register copies of its most frequent classes' slices.
# Queues dominated by a few classes (so the cached classes repeat), rows whose
# mass sits in a window (so whole panels lie before a row's first bin with
# mass, where G becomes 0, or after its last, where the row is 0): a cached
# class's first member then falls on skipped steps, and its later members
# must still see this pass's slice.  Ragged and exact grids, chunked launches
# whose warm-up steps take the cached path too.
# ---------------------------------------------------------------------------
def window_counts(rng, B, C, K, total=TOTAL):
    """[B, C, K] counts: each row's mass spread over a window of random start
    and width (some near the grid's start, some near its end)."""
    out = np.zeros((B, C, K), np.uint32)
    for b in range(B):
        for c in range(C):
            w = int(rng.integers(1, K // 2))
            a = int(rng.integers(0, K - w))
            m = rng.random(w) + 0.05
            cum = np.rint(np.cumsum(m) / m.sum() * total)
            out[b, c, a:a + w] = np.diff(np.concatenate([[0.0], cum])).astype(np.uint32)
    return out


def repeated_class_case(seed, K):
    rng = np.random.default_rng(9100 + seed)
    M, C, bs = 2, 12, (8, 33, 64)
    counts = np.stack([window_counts(rng, len(bs), C, K) for _ in range(M)])
    # Zipf-like class draws: three or four classes take most members
    p = 1.0 / np.arange(1, C + 1) ** 1.6
    p /= p.sum()
    queues, nows = [], []
    for q in range(M):
        n = 64 + 7 * q
        cls = rng.permutation(C)[rng.choice(C, size=n, p=p)]
        d = np.sort(rng.uniform(1.0, 200.0, n))           # in the first panel
        queues.append((cls, d))
        nows.append(0.0)
    return explicit_workload(f"repeat-{seed}-K{K}", counts, bs, [1.0] * M, queues, nows)


def mixed_panel_case(seed, K):
    """Repeated classes with deadlines over the first three panels: the
    launch's short prefixes end in panel 0 (the kernel body for one member
    panel) and its long ones in later panels (the general body), and its
    largest prefix (57 members) leaves LDS for two cached slices, not three."""
    rng = np.random.default_rng(9200 + seed)
    M, C, bs = 3, 12, (8, 16, 33, 57)
    counts = np.stack([window_counts(rng, len(bs), C, K) for _ in range(M)])
    p = 1.0 / np.arange(1, C + 1) ** 1.2
    p /= p.sum()
    queues, nows = [], []
    for q in range(M):
        n = 57 + 5 * q
        cls = rng.permutation(C)[rng.choice(C, size=n, p=p)]
        d = np.sort(rng.uniform(1.0, 0.7 * K, n))          # panels 0 .. 2 (1-ms bins)
        queues.append((cls, d))
        nows.append(0.0)
    return explicit_workload(f"mixed-{seed}-K{K}", counts, bs, [1.0] * M, queues, nows)


@gpu
@pytest.mark.parametrize("K", [4096, 3000])
@pytest.mark.parametrize("seed", range(3))
def test_mixed_member_panels_cached_slices(ctx, seed, K):
    wl = mixed_panel_case(seed, K)
    say(f"[mixed-panel case] seed={seed} K={K}")
    ora = oracle.score_workload(wl)
    _, got = run_gpu(wl, ctx)
    err = parity.compare(wl, got, ora)
    say(f"  max errors {err}")
    _, untrimmed = run_gpu(wl, ctx, trim=False)
    same_bits(got, untrimmed)
    for chunk in (0, 8):
        _, split = run_gpu(wl, ctx, chunk=chunk)
        same_bits(got, split)


@gpu
@pytest.mark.parametrize("K", [4096, 3000, 2048])
@pytest.mark.parametrize("seed", range(3))
def test_repeated_classes_cached_slices(ctx, seed, K):
    wl = repeated_class_case(seed, K)
    say(f"[repeated-class case] seed={seed} K={K}")
    ora = oracle.score_workload(wl)
    _, got = run_gpu(wl, ctx)
    err = parity.compare(wl, got, ora)
    say(f"  max errors {err}")
    _, untrimmed = run_gpu(wl, ctx, trim=False)
    same_bits(got, untrimmed)
    for chunk in (0, 8):
        _, split = run_gpu(wl, ctx, chunk=chunk)
        same_bits(got, split)
