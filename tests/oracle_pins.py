"""Pins for the CPU oracle.

Each pin checks the oracle against something other than its own code: exact
rational brute force, closed forms, numerical quadrature of the priority's
definition, Monte Carlo of the batch maximum, the paper's Eq. (8), and
invariants the mathematics fixes.  Every pin takes a loaded oracle library
handle, so planted-mistake builds of the oracle source run through the very
same checks (tests/test_oracle_mutants.py); a pin raises AssertionError
when the oracle is wrong.
"""
from __future__ import annotations

import itertools
import math
from fractions import Fraction

import numpy as np
from scipy import integrate, special

import oracle
from paper_2209_00159_amd import workloads as W


def rng(seed):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([2209_00159, 7, seed])))


def run_model(L, class_rows, queue_cls, taus, w, b=1e-4, batch_sizes=None, now=1000.0,
              prefix_mode=0, per_bs_rows=None):
    """One model through the oracle.  ``class_rows`` [C, K] are used for
    every batch size unless ``per_bs_rows`` [B, C, K] is given.  Returns the
    oracle dict plus the effective time-to-deadline the oracle sees."""
    queue_cls = np.asarray(queue_cls, np.int32)
    if batch_sizes is None:
        batch_sizes = [max(1, len(queue_cls))]
    if per_bs_rows is None:
        counts = np.repeat(np.asarray(class_rows, np.uint32)[None], len(batch_sizes), axis=0)
    else:
        counts = np.asarray(per_bs_rows, np.uint32)
    dl = now + np.asarray(taus, np.float64)
    out = oracle.score_model(counts, batch_sizes, w, queue_cls, dl, now, b, prefix_mode,
                             want_priority=True, L=L)
    out["tau"] = dl - now
    return out


def slot(n, m):
    """Position of member m (1-based) of prefix n inside one batch size's
    block of per-member outputs."""
    return (n - 1) * n // 2 + (m - 1)


# ---------------------------------------------------------------- exact helpers
def enumerate_max_masses(rows):
    """Exact probability that the slowest member lands in bin j, by brute
    force over every tuple of member bins (members independent)."""
    rows = np.asarray(rows)
    n, K = rows.shape
    tots = [int(r.sum()) for r in rows]
    mass = [Fraction(0)] * K
    for tup in itertools.product(range(K), repeat=n):
        wgt = Fraction(1)
        for i, k in enumerate(tup):
            c = int(rows[i, k])
            if c == 0:
                wgt = Fraction(0)
                break
            wgt *= Fraction(c, tots[i])
        if wgt:
            mass[max(tup)] += wgt
    return mass


def exact_cdf_product(rows):
    """prod_i F_i(x_k) with exact rationals (the law of the max of
    independent variables), k = 0..K."""
    rows = np.asarray(rows)
    K = rows.shape[1]
    G = [Fraction(1)] * (K + 1)
    for r in rows:
        tot = int(r.sum())
        run = 0
        Fi = [Fraction(0)]
        for k in range(K):
            run += int(r[k])
            Fi.append(Fraction(run, tot))
        G = [g * f for g, f in zip(G, Fi)]
    return G


def histogram_prob_below(mass, w, tau):
    """P(L <= tau) for a histogram with uniform mass inside each bin."""
    if tau <= 0:
        return Fraction(0)
    u = Fraction(tau) / Fraction(w)
    K = len(mass)
    if u >= K:
        return sum(mass, Fraction(0))
    k = math.floor(u)
    return sum(mass[:k], Fraction(0)) + (u - k) * mass[k]


def histogram_mean(mass, w):
    return sum(((j + Fraction(1, 2)) * Fraction(w) * m for j, m in enumerate(mass)),
               Fraction(0))


def delay_gain_quadrature(mass, w, tau, b):
    """P(L <= tau < L + delay), delay ~ Exp(b), for L with density
    mass_j / w on bin j: the integral over l < tau of the density times
    P(delay > tau - l) = exp(-b (tau - l)), by adaptive quadrature."""
    total = 0.0
    for j, m in enumerate(mass):
        lo, hi = j * w, min((j + 1) * w, tau)
        if hi <= lo or m == 0:
            continue
        val, _ = integrate.quad(lambda l: math.exp(-b * (tau - l)), lo, hi,
                                epsabs=0.0, epsrel=1e-13, limit=200)
        total += float(m) / w * val
    return total


# ---------------------------------------------------------------- pins
def pin_enumeration(L):
    """Batch CDF, bin masses, E[L_B], finish probabilities and priorities of
    tiny batches against exact rational brute force over member bins and
    quadrature of the priority's definition."""
    for seed in range(6):
        r = rng(seed)
        K = int(r.integers(2, 7))
        C = int(r.integers(1, 4))
        n = int(r.integers(1, 5))
        rows = r.integers(0, 9, size=(C, K))
        rows[rows.sum(axis=1) == 0, -1] = 1
        cls = r.integers(0, C, size=n)
        w = float(r.uniform(0.5, 3.0))
        taus = np.sort(r.uniform(-0.5 * w, (K + 1.5) * w, size=n))
        b = float(r.choice([1e-4, 0.05, 0.7]))
        out = run_model(L, rows, cls, taus, w, b=b)
        for nn in range(1, n + 1):
            mass = enumerate_max_masses(rows[cls[:nn]])
            G = np.array([float(sum(mass[:k], Fraction(0))) for k in range(K + 1)])
            Gor = oracle.batch_cdf(rows[cls[:nn]], L=L)
            assert np.allclose(Gor, G, rtol=0, atol=1e-14), (seed, nn, Gor, G)
            E = float(histogram_mean(mass, w))
            assert abs(out["expected_latency_ms"][nn - 1] - E) <= 1e-12 * E, (seed, nn)
            ef = 0.0
            sc = 0.0
            for m in range(1, nn + 1):
                tau = float(out["tau"][m - 1])
                P = float(histogram_prob_below(mass, w, tau))
                ef += P
                got = out["finish_prob"][slot(nn, m)]
                assert abs(got - P) <= 1e-13, (seed, nn, m, got, P)
                pr = delay_gain_quadrature(mass, w, tau, b) / E
                sc += pr
                gp = out["priority"][slot(nn, m)]
                assert abs(gp - pr) <= 1e-11 * max(1.0, abs(pr)) + 1e-15, (seed, nn, m, gp, pr)
            assert abs(out["expected_finish"][nn - 1] - ef) <= 1e-12
            assert abs(out["score"][nn - 1] - sc) <= 1e-10 * max(1.0, sc)


def pin_iid_power(L):
    """Identical members: the batch CDF is F^n (§4.2.1)."""
    r = rng(11)
    K = 17
    row = r.integers(0, 50, size=K)
    row[-1] += 1
    tot = int(row.sum())
    cum = np.concatenate([[0], np.cumsum(row)])
    for n in (1, 2, 3, 7, 12):
        G = oracle.batch_cdf(np.repeat(row[None], n, axis=0), L=L)
        ref = np.array([float(Fraction(int(c), tot) ** n) for c in cum])
        assert np.allclose(G, ref, rtol=1e-14, atol=1e-300), n


def pin_point_mass(L):
    """Static models (all of a class's mass in one bin): the batch runs as
    long as its slowest member's bin, deterministically (§4.2 static case):
    P is a ramp across that bin, E[L_B] is the bin's midpoint, and as the
    delay rate b -> 0 the priority equals P / E[L_B]."""
    K, w = 12, 2.0
    C = 4
    pos = [1, 4, 4, 9]
    rows = np.zeros((C, K), np.int64)
    for c, j in enumerate(pos):
        rows[c, j] = 7 + c
    cls = np.array([0, 2, 1, 3, 0])
    taus = np.array([1.0, 2.5, 9.0, 10.0, 30.0])
    out = run_model(L, rows, cls, taus, w, b=1e-9)
    for nn in range(1, len(cls) + 1):
        jstar = max(pos[c] for c in cls[:nn])
        E = (jstar + 0.5) * w
        assert abs(out["expected_latency_ms"][nn - 1] - E) <= 1e-12 * E
        for m in range(1, nn + 1):
            tau = out["tau"][m - 1]
            P = min(1.0, max(0.0, tau / w - jstar))
            got = out["finish_prob"][slot(nn, m)]
            assert abs(got - P) <= 1e-12, (nn, m, got, P)
            pr = out["priority"][slot(nn, m)]
            assert abs(pr * E - P) <= 1e-7, (nn, m, pr * E, P)


def pin_quadrature_medium(L):
    """Medium batches (beyond brute force): priorities against quadrature of
    their definition on the exact-rational product of the member CDFs."""
    r = rng(21)
    K, C, n = 40, 5, 6
    rows = r.integers(0, 30, size=(C, K))
    rows[:, :3] = 0
    rows[rows.sum(axis=1) == 0, -1] = 1
    cls = r.integers(0, C, size=n)
    w = 0.8
    taus = np.sort(r.uniform(1.0, 45.0, size=n))
    for b in (1e-4, 0.02, 0.3):
        out = run_model(L, rows, cls, taus, w, b=b)
        G = exact_cdf_product(rows[cls])
        mass = [G[k + 1] - G[k] for k in range(K)]
        E = float(histogram_mean(mass, w))
        assert abs(out["expected_latency_ms"][n - 1] - E) <= 1e-12 * E
        for m in range(1, n + 1):
            tau = float(out["tau"][m - 1])
            pr = delay_gain_quadrature(mass, w, tau, b) / E
            got = out["priority"][slot(n, m)]
            assert abs(got - pr) <= 1e-11 * max(1.0, pr) + 1e-16, (b, m, got, pr)


def pin_b_to_zero(L):
    """As the anticipated delay rate b -> 0 a member's priority times
    E[L_B] tends to its finish probability (each bin's delay factor -> 1)."""
    r = rng(31)
    K, C, n = 30, 3, 5
    rows = r.integers(0, 20, size=(C, K))
    rows[rows.sum(axis=1) == 0, -1] = 1
    cls = r.integers(0, C, size=n)
    taus = np.sort(r.uniform(-2.0, 40.0, size=n))
    out = run_model(L, rows, cls, taus, 1.1, b=1e-10)
    for nn in range(1, n + 1):
        E = out["expected_latency_ms"][nn - 1]
        for m in range(1, nn + 1):
            P = out["finish_prob"][slot(nn, m)]
            pr = out["priority"][slot(nn, m)]
            assert abs(pr * E - P) <= 1e-7, (nn, m, pr * E, P)


def pin_monte_carlo_max(L):
    """Monte Carlo of the slowest member: sample each member's latency from
    its histogram (bin by count, uniform inside), take the max; at grid
    deadlines the oracle's finish probability must lie within 4 sigma of
    the empirical frequency."""
    r = rng(41)
    K, C, n = 24, 4, 5
    rows = r.integers(0, 40, size=(C, K))
    rows[rows.sum(axis=1) == 0, -1] = 1
    cls = r.integers(0, C, size=n)
    w = 1.0
    now = 0.0
    taus = np.arange(3, 3 + n, dtype=np.float64) * 4.0     # grid points
    out = run_model(L, rows, cls, taus, w, b=1e-4, now=now)
    S = 400_000
    lat = np.zeros(S)
    for c in cls:
        p = rows[c] / rows[c].sum()
        bins = r.choice(K, size=S, p=p)
        lat = np.maximum(lat, (bins + r.random(S)) * w)
    for m in range(1, n + 1):
        tau = taus[m - 1]
        emp = (lat <= tau).mean()
        P = out["finish_prob"][slot(n, m)]
        sig = math.sqrt(max(P * (1 - P), 1e-12) / S)
        assert abs(emp - P) <= 4 * sig + 1e-9, (m, emp, P, sig)


def pin_monte_carlo_priority(L):
    """Monte Carlo of the priority's definition (Eq. (1)): with L drawn from
    the batch histogram and the anticipated delay ~ Exp(b), the expected
    cost saved by running now is P(L <= tau < L + delay); dividing by
    E[L_B] must give the oracle's priority within 4 sigma."""
    r = rng(51)
    K, C, n = 20, 3, 4
    rows = r.integers(0, 25, size=(C, K))
    rows[rows.sum(axis=1) == 0, -1] = 1
    cls = r.integers(0, C, size=n)
    w, b = 1.5, 0.08
    taus = np.sort(r.uniform(5.0, 35.0, size=n))
    out = run_model(L, rows, cls, taus, w, b=b)
    G = exact_cdf_product(rows[cls])
    mass = np.array([float(G[k + 1] - G[k]) for k in range(K)])
    S = 1_000_000
    bins = r.choice(K, size=S, p=mass / mass.sum())
    lat = (bins + r.random(S)) * w
    delay = r.exponential(1.0 / b, size=S)
    E = out["expected_latency_ms"][n - 1]
    for m in range(1, n + 1):
        tau = out["tau"][m - 1]
        ev = ((lat <= tau) & (tau < lat + delay)).mean()
        pr = out["priority"][slot(n, m)] * E
        sig = math.sqrt(max(pr * (1 - pr), 1e-12) / S)
        assert abs(ev - pr) <= 4 * sig + 1e-9, (m, ev, pr, sig)
    assert abs(E - float(lat.mean())) <= 4 * float(lat.std()) / math.sqrt(S)


def ozbey_density(Fs, fs):
    """Density of the max of independent, non-identical variables by the
    inclusion-exclusion formula the paper cites (§4.2.2, Eq. (8)): a sum
    over subset sizes kappa of (-1)^(k-kappa) kappa^k / k! times, over the
    subsets s of that size, k [F^s]^(k-1) f^s with F^s, f^s the subset
    averages."""
    k = len(Fs)
    tot = 0.0
    for kappa in range(1, k + 1):
        coef = (-1) ** (k - kappa) * kappa ** k / math.factorial(k)
        inner = 0.0
        for s in itertools.combinations(range(k), kappa):
            Fs_avg = sum(Fs[i] for i in s) / kappa
            fs_avg = sum(fs[i] for i in s) / kappa
            inner += k * Fs_avg ** (k - 1) * fs_avg
        tot += coef * inner
    return tot


def pin_ozbey_eq8(L):
    """The product of the member CDFs is the CDF of the batch maximum: its
    change over each bin equals the integral of the paper's Eq. (8) density
    (Özbey et al.) for analytic lognormal members, up to the quantisation of
    the histograms (2^31 samples each)."""
    params = [(30.0, 0.3), (45.0, 0.5), (25.0, 0.2), (60.0, 0.4)]
    K, w = 64, 2.5
    x = np.arange(K + 1) * w
    rows = []
    for med, s in params:
        cdf = np.where(x > 0, special.ndtr((np.log(np.maximum(x, 1e-300)) - math.log(med)) / s),
                       0.0)
        rows.append(W.quantise_counts(cdf, total=1 << 31))
    rows = np.array(rows)
    G = oracle.batch_cdf(rows, L=L)
    mass = np.diff(G)

    def cdf_pdf(l):
        Fs, fs = [], []
        for med, s in params:
            z = (math.log(l) - math.log(med)) / s
            Fs.append(special.ndtr(z))
            fs.append(math.exp(-0.5 * z * z) / (l * s * math.sqrt(2 * math.pi)))
        return Fs, fs

    for j in range(8, K - 1):
        val, _ = integrate.quad(lambda l: ozbey_density(*cdf_pdf(l)), x[j], x[j + 1],
                                epsabs=1e-13, epsrel=1e-10)
        assert abs(val - mass[j]) <= 2e-8, (j, val, mass[j])


def pin_invariants(L):
    """G in [0, 1], non-decreasing along the grid, non-increasing as members
    join; E[L_B] non-decreasing as members join (adding a member never makes
    the batch faster); P non-decreasing in the time left; priorities and P
    unchanged when every histogram is scaled by an integer."""
    r = rng(61)
    K, C, n = 33, 4, 9
    rows = r.integers(0, 15, size=(C, K))
    rows[r.random(rows.shape) < 0.4] = 0
    rows[rows.sum(axis=1) == 0, -1] = 1
    cls = r.integers(0, C, size=n)
    prev = None
    for nn in range(1, n + 1):
        G = oracle.batch_cdf(rows[cls[:nn]], L=L)
        assert G[0] == 0.0 and G[-1] == 1.0
        assert np.all(np.diff(G) >= 0) and np.all((G >= 0) & (G <= 1))
        if prev is not None:
            assert np.all(G <= prev + 1e-15)
        prev = G
    taus = np.sort(r.uniform(-3.0, 45.0, size=n))
    out = run_model(L, rows, cls, taus, 1.3, b=0.01)
    EL = out["expected_latency_ms"]
    assert np.all(np.diff(EL) >= -1e-12)
    for nn in range(1, n + 1):
        P = out["finish_prob"][slot(nn, 1):slot(nn, nn) + 1]
        assert np.all(np.diff(P) >= -1e-15), nn
    out3 = run_model(L, rows * 3, cls, taus, 1.3, b=0.01)
    for k in ("finish_prob", "priority", "expected_latency_ms", "score"):
        assert np.allclose(out[k], out3[k], rtol=1e-13, atol=1e-15), k


def pin_continuity(L):
    """Eq. (2) is continuous in t: at the milestones where a bin edge meets
    the deadline (t = D - l) the priority and P have no jump."""
    r = rng(71)
    K, C = 16, 2
    rows = r.integers(1, 20, size=(C, K))
    w = 1.25
    for edge in (3, 7, 12):
        for b in (1e-4, 0.2):
            vals = []
            for eps in (-1e-9, 1e-9):
                out = run_model(L, rows, [0, 1], [edge * w + eps, 30.0], w, b=b, now=0.0)
                vals.append((out["priority"][slot(2, 1)], out["finish_prob"][slot(2, 1)]))
            assert abs(vals[0][0] - vals[1][0]) <= 1e-7, (edge, b, vals)
            assert abs(vals[0][1] - vals[1][1]) <= 1e-7, (edge, b, vals)


def pin_edge_cases(L):
    """Dead requests finish with probability 0 and add no priority; deadlines
    beyond the grid finish with probability 1; a batch always takes at least
    half a bin on average."""
    K, w = 10, 1.0
    rows = np.zeros((1, K), np.int64)
    rows[0, 0] = 5
    out = run_model(L, rows, [0, 0, 0], [-5.0, 0.0, 25.0], w, b=1e-3)
    n = 3
    assert out["finish_prob"][slot(n, 1)] == 0.0 and out["priority"][slot(n, 1)] == 0.0
    assert out["finish_prob"][slot(n, 2)] == 0.0 and out["priority"][slot(n, 2)] == 0.0
    assert out["finish_prob"][slot(n, 3)] == 1.0
    assert abs(out["expected_latency_ms"][n - 1] - 0.5 * w) <= 1e-15


def _brute_select(wl_model_out, batch_sizes, caps):
    best = None
    i = 0
    for bi, b in enumerate(batch_sizes):
        for n in range(1, caps[bi] + 1):
            s = wl_model_out["score"][i]
            i += 1
            if n > b:
                continue
            key = (s, n, -b)
            if best is None or key > best[0]:
                best = (key, n, b, s)
    if best is None or best[3] <= 0:
        return 0, 0
    return best[1], best[2]


def pin_selection(L):
    """Selection is the largest score over candidates n <= batch size; exact
    ties go to the larger prefix, then the smaller batch size; no batch when
    every score is <= 0."""
    r = rng(81)
    for seed in range(5):
        wl = W.random_case(seed, n_models=1, queue_lens=[int(r.integers(1, 12))])
        m = wl.model(0)
        out = oracle.score_model(m["counts"], wl.batch_sizes, m["bin_width_ms"], m["cls"],
                                 m["deadline_ms"], m["now_ms"], wl.b_expo, L=L)
        caps = np.minimum(wl.batch_sizes, wl.queue_len(0))
        assert (out["sel_n"], out["sel_bs"]) == _brute_select(out, wl.batch_sizes, caps)
    # identical tables for every batch size and one member: equal scores,
    # the smaller batch size wins.
    rows = np.array([[0, 3, 5, 1, 0, 0]])
    out = run_model(L, rows, [0], [4.0], 1.0, batch_sizes=[1, 2, 4])
    assert out["score"][0] == out["score"][1] == out["score"][2] > 0
    assert (out["sel_n"], out["sel_bs"]) == (1, 1)
    # two identical members: prefix 2 ties prefix 1 only if scores equal;
    # a dead queue selects nothing.
    out = run_model(L, rows, [0, 0], [-1.0, -0.5], 1.0, batch_sizes=[1, 2])
    assert out["sel_n"] == 0 and out["sel_bs"] == 0


def pin_rect_mode(L):
    """prefix_mode 1 scores prefixes up to the queue length at every batch
    size; prefixes within the batch size match prefix_mode 0 and longer ones
    are never selected."""
    wl = W.random_case(3, n_models=1, queue_lens=[9], batch_sizes=(1, 2, 4))
    m = wl.model(0)
    args = (m["counts"], wl.batch_sizes, m["bin_width_ms"], m["cls"], m["deadline_ms"],
            m["now_ms"], wl.b_expo)
    tri = oracle.score_model(*args, prefix_mode=0, L=L)
    rect = oracle.score_model(*args, prefix_mode=1, L=L)
    ti = ri = 0
    for b in wl.batch_sizes:
        for n in range(1, 10):
            if n <= b:
                assert rect["score"][ri] == tri["score"][ti]
                assert rect["expected_finish"][ri] == tri["expected_finish"][ti]
                ti += 1
            ri += 1
    assert rect["sel_n"] <= rect["sel_bs"]
    assert (rect["sel_n"], rect["sel_bs"]) == (tri["sel_n"], tri["sel_bs"])


def pin_toy_example(L):
    """The paper's toy example (§4.2.2): two distributions with the same
    mean, one concentrated and one early-or-late, batch of two.  The batch
    histogram is skewed to the right of both members (it dominates each
    member's CDF), and a member's priority rises as its deadline nears and
    falls to zero once even the fastest batch outcome can no longer make
    it."""
    K, w = 20, 1.0
    concentrated = np.zeros(K, np.int64)
    concentrated[9:11] = 50
    early_late = np.zeros(K, np.int64)
    early_late[2] = 50
    early_late[17] = 50
    rows = np.stack([concentrated, early_late])
    G = oracle.batch_cdf(rows, L=L)
    for row in rows:
        F = oracle.cdf(row, L=L)
        assert np.all(G <= F + 1e-15)
    assert np.all(np.diff(G)[:9] == 0.0)          # no batch outcome below bin 9
    # priority of a member vs time left (decreasing time left = time passes)
    pri = []
    taus = np.linspace(30.0, 0.5, 60)
    for tau in taus:
        out = run_model(L, rows, [0, 1], [tau, 40.0], w, b=0.05, now=0.0)
        pri.append(out["priority"][slot(2, 1)])
    pri = np.array(pri)
    peak = int(np.argmax(pri))
    assert 0 < peak < len(taus) - 1
    assert np.all(np.diff(pri[:peak + 1]) >= -1e-12)       # rises
    assert np.all(pri[taus <= 9.0] == 0.0)                 # then 0


# ---------------------------------------------------------------- Algorithm 1 iteration
def iterate(L, counts_bcK, batch_sizes, cls, taus, w, b=1e-4, now=500.0, weights=None):
    dl = now + np.asarray(taus, np.float64)
    out = oracle.iterate_model(counts_bcK, batch_sizes, w, np.asarray(cls, np.int32), dl, now, b,
                               weights=weights, L=L)
    out["tau"] = dl - now
    return out


def pin_iterate_one_class(L):
    """With a single class the law of a request's batch at batch size s is
    that of s identical members, F^s: its priority must equal the
    candidate-scoring priority of a member of the s-member batch of that
    class (a product of s CDFs there, a power of the mix here), for every
    request in Q_s, and the model-wide E[L] must be that batch's E[L_B]."""
    r = rng(61)
    K = 40
    row = r.integers(0, 30, size=K)
    row[:3] = 0
    row[-1] += 1
    w, b = 2.0, 0.01
    for s in (1, 3, 6):
        N = s + 3
        taus = np.sort(r.uniform(8.0, 90.0, size=N))
        it = iterate(L, row[None, None, :], [s], np.zeros(N), taus, w, b)
        assert it["cand_bs"] == s
        sc = run_model(L, row[None], np.zeros(s), taus[:s], w, b, batch_sizes=[s])
        E = sc["expected_latency_ms"][s - 1]
        for m in range(1, s + 1):
            pr = sc["priority"][slot(s, m)]
            assert abs(it["score"][m - 1] - pr) <= 1e-12 + 1e-10 * abs(pr), (s, m, it["score"][m - 1], pr)
        # E[L] enters as the normaliser: score * E[L_B] is the bare Eq. (2) sum
        for m in range(1, s + 1):
            assert abs(it["score"][m - 1] * E - sc["priority"][slot(s, m)] * E) <= 1e-10


def pin_iterate_point_mix(L):
    """A class mix concentrated on one class m0 makes the batch of a request
    of class c at batch size s the batch {c, m0 x (s-1)}: its priority must
    equal the candidate-scoring priority of that request as the first member
    of the prefix [c, m0, ..., m0], divided by the mix's own E[L] instead of
    that batch's."""
    r = rng(62)
    K, C = 30, 3
    rows = r.integers(0, 20, size=(C, K))
    rows[rows.sum(axis=1) == 0, -1] = 1
    w, b, s, m0 = 1.5, 0.02, 4, 2
    weights = np.zeros(C)
    weights[m0] = 1.0
    checked = 0
    for c in range(C):
        taus = np.array([25.0, 26.0, 27.0, 28.0, 29.0])
        cls = [c, m0, m0, m0, m0]
        it = iterate(L, rows[None], [s], cls, taus, w, b, weights=weights)
        if it["cand_bs"] != s or it["score"][0] == 0.0:
            continue
        sc = run_model(L, rows, cls[:s], [taus[0]] * s, w, b, batch_sizes=[s])
        E_batch = sc["expected_latency_ms"][s - 1]
        pr_times_E = sc["priority"][slot(s, 1)] * E_batch
        mixonly = run_model(L, rows, [m0] * s, [taus[0]] * s, w, b, batch_sizes=[s])
        E_mix = mixonly["expected_latency_ms"][s - 1]
        got = it["score"][0]
        assert abs(got - pr_times_E / E_mix) <= 1e-12 + 1e-9 * abs(got), (c, got, pr_times_E / E_mix)
        checked += 1
    assert checked >= 2


def pin_iterate_monte_carlo_mix(L):
    """Monte Carlo of the mix law: a request of class c plus s-1 members
    whose classes are drawn from the weights; the Eq. (1) event under that
    latency, divided by the model-wide E[L] (Monte Carlo of s mix members),
    must match the oracle's priority within 4 sigma."""
    r = rng(63)
    K, C, s = 16, 3, 3
    rows = r.integers(0, 12, size=(C, K))
    rows[rows.sum(axis=1) == 0, -1] = 1
    weights = np.array([0.5, 0.3, 0.2])
    w, b = 1.0, 0.05
    taus = np.array([9.0, 11.5, 14.0])
    cls = np.array([1, 0, 2])
    it = iterate(L, rows[None], [s], cls, taus, w, b, weights=weights)
    assert it["cand_bs"] == s
    S = 600_000

    def draw(c, size):
        p = rows[c] / rows[c].sum()
        return (r.choice(K, size=size, p=p) + r.random(size)) * w

    def draw_mix(size):
        cc = r.choice(C, size=size, p=weights)
        out = np.empty(size)
        for c in range(C):
            sel = cc == c
            out[sel] = draw(c, int(sel.sum()))
        return out

    model_lat = np.max(np.stack([draw_mix(S) for _ in range(s)]), axis=0)
    E_mix = model_lat.mean()
    for i, (c, tau) in enumerate(zip(cls, taus)):
        lat = draw(c, S)
        for _ in range(s - 1):
            lat = np.maximum(lat, draw_mix(S))
        delay = r.exponential(1.0 / b, size=S)
        ev = ((lat <= tau) & (tau < lat + delay)).mean()
        got = it["score"][i] * E_mix
        sig = math.sqrt(max(ev * (1 - ev), 1e-12) / S) + abs(got) * float(model_lat.std()) / math.sqrt(S) / E_mix
        assert abs(ev - got) <= 4 * sig + 1e-9, (i, ev, got, sig)


def pin_iterate_feasibility_and_popbatch(L):
    """The drop phase against the counts themselves (a request can finish
    by tau at batch size s iff tau lies past the left edge of the first bin
    holding mass of its class's histogram), the candidate rule's defining
    property, and PopBatch by brute force over all subsets of Q_cand."""
    import itertools
    r = rng(64)
    for trial in range(40):
        K, C = 12, 3
        bsz = sorted(set(int(x) for x in r.integers(1, 5, size=3)))
        B = len(bsz)
        counts = r.integers(0, 6, size=(B, C, K))
        counts[..., : int(r.integers(0, 6))] = 0
        counts[counts.sum(axis=-1) == 0, -1] = 1
        N = int(r.integers(0, 8))
        w, b = 1.0, 0.05
        taus = np.sort(r.uniform(-2.0, 14.0, size=N))
        cls = r.integers(0, C, size=N)
        it = iterate(L, counts, bsz, cls, taus, w, b)
        first = np.argmax(counts > 0, axis=-1)                 # [B, C]
        feas = np.array([[taus[i] > first[j, cls[i]] * w for j in range(B)] for i in range(N)],
                        dtype=bool).reshape(N, B)
        assert np.array_equal(it["timed_out"], (~feas.any(axis=1)).astype(np.int32)), trial
        sizes = feas.sum(axis=0)
        ok = [j for j in range(B) if sizes[j] >= bsz[j]]
        if not ok:
            assert it["cand_bs"] == 0 and it["batch"].size == 0
            continue
        key = lambda j: (taus[np.argmax(feas[:, j])], bsz[j])
        jbest = max(ok, key=key)
        assert it["cand_bs"] == bsz[jbest], trial
        q = [i for i in range(N) if feas[i, jbest]]
        sc = it["score"]
        assert all(sc[i] == 0.0 for i in range(N) if i not in q)
        best = max(sum(sc[list(c)]) for c in itertools.combinations(q, bsz[jbest]))
        assert abs(sum(sc[it["batch"]]) - best) <= 1e-12 * max(1.0, best)
        assert set(it["batch"]).issubset(q) and len(set(it["batch"])) == bsz[jbest]
        assert all(sc[it["batch"][i]] >= sc[it["batch"][i + 1]] for i in range(len(it["batch"]) - 1))


# ---------------------------------------------------------------- costs and profiler feedback
def pin_cost_weights(L):
    """Per-request miss costs (§4.1's c): unit costs change nothing; scaling
    every cost by lam scales every score by lam and leaves the selection; a
    member with cost 0 adds nothing; and a Monte Carlo of Eq. (1) with the
    cost, c P(L <= tau < L + delay) summed over the batch, matches the score
    times E[L_B]."""
    r = rng(71)
    K, C, n = 20, 3, 4
    rows = r.integers(0, 25, size=(C, K))
    rows[rows.sum(axis=1) == 0, -1] = 1
    cls = r.integers(0, C, size=n)
    w, b = 1.5, 0.08
    taus = np.sort(r.uniform(5.0, 35.0, size=n))
    dl = 1000.0 + taus
    counts = rows[None].repeat(1, axis=0)
    base = oracle.score_model(counts, [n], w, cls, dl, 1000.0, b, want_priority=True, L=L)
    unit = oracle.score_model(counts, [n], w, cls, dl, 1000.0, b, L=L, cost=np.ones(n))
    assert np.array_equal(base["score"], unit["score"])
    cost = r.uniform(0.2, 3.0, size=n)
    wgt = oracle.score_model(counts, [n], w, cls, dl, 1000.0, b, L=L, cost=cost)
    sc2 = oracle.score_model(counts, [n], w, cls, dl, 1000.0, b, L=L, cost=2.5 * cost)
    assert np.allclose(sc2["score"], 2.5 * wgt["score"], rtol=1e-13, atol=0)
    assert (sc2["sel_n"], sc2["sel_bs"]) == (wgt["sel_n"], wgt["sel_bs"])
    zero = cost.copy()
    zero[1] = 0.0
    z = oracle.score_model(counts, [n], w, cls, dl, 1000.0, b, L=L, cost=zero)
    assert z["score"][0] == wgt["score"][0]                         # prefix 1 does not hold member 2
    # Monte Carlo of the weighted event for the full batch
    G = exact_cdf_product(rows[cls])
    mass = np.array([float(G[k + 1] - G[k]) for k in range(K)])
    S = 1_000_000
    lat = (r.choice(K, size=S, p=mass / mass.sum()) + r.random(S)) * w
    delay = r.exponential(1.0 / b, size=S)
    ev = sum(cost[m] * ((lat <= taus[m]) & (taus[m] < lat + delay)).mean() for m in range(n))
    got = wgt["score"][n - 1] * wgt["expected_latency_ms"][n - 1]
    sig = math.sqrt(sum(cost ** 2) * 0.25 / S)
    assert abs(ev - got) <= 4 * sig, (ev, got, sig)


def pin_step_costs(L):
    """App. B: a piecewise-step cost function is the sum of single steps.
    A request whose cost rises by c1 at d1 and to c2 at d2 must score
    c1 p(d1) + (c2 - c1) p(d2), p(d) the score of a single-step request of
    the same class with deadline d in the same queue; and a Monte Carlo of
    the cost function itself, E[cost(L + delay) - cost(L)] over the batch
    law F^s, must match that score times E[L]."""
    r = rng(72)
    K = 30
    row = r.integers(0, 20, size=K)
    row[:2] = 0
    row[-1] += 1
    w, b, s = 1.0, 0.04, 2
    now = 100.0
    d1, d2, c1, c2 = now + 12.0, now + 19.0, 0.7, 1.9
    # queue: the step request (deadline d1) and single-step twins at d1, d2
    cls = np.zeros(3, np.int32)
    dl = np.array([d1, d1, d2])
    steps = (np.array([0, 2, 3, 4]), np.array([d1, d2, d1, d2]), np.array([c1, c2, 1.0, 1.0]))
    it = oracle.iterate_model(row[None, None, :], [s], w, cls, dl, now, b, L=L, steps=steps)
    assert it["cand_bs"] == s
    p1, p2 = it["score"][1], it["score"][2]
    assert p1 > 0 and p2 > 0
    assert abs(it["score"][0] - (c1 * p1 + (c2 - c1) * p2)) <= 1e-12 * it["score"][0]
    # Monte Carlo of the step cost function under the batch law F^s
    F = np.concatenate([[0.0], np.cumsum(row) / row.sum()])
    G = F ** s
    mass = np.diff(G)
    S = 1_000_000
    lat = (r.choice(K, size=S, p=mass / mass.sum()) + r.random(S)) * w
    delay = r.exponential(1.0 / b, size=S)

    def cost(fin):
        return np.where(fin <= d1 - now, 0.0, np.where(fin <= d2 - now, c1, c2))
    saved = cost(lat + delay) - cost(lat)
    E = w * (0.5 + np.sum(1.0 - G[1:]))
    got = it["score"][0] * E
    sig = float(saved.std()) / math.sqrt(S)
    assert abs(saved.mean() - got) <= 4 * sig + 1e-9, (saved.mean(), got, sig)
    # the drop phase looks at the last step: past d1 but before d2 a step
    # request is still kept, a single-step one is not
    later = oracle.iterate_model(row[None, None, :], [1], w, np.zeros(2, np.int32),
                                 np.array([d1, d1]), d1 + 1.0, b, L=L,
                                 steps=(np.array([0, 2, 3]), np.array([d1, d2, d1]),
                                        np.array([c1, c2, 1.0])))
    assert list(later["timed_out"]) == [0, 1]


def pin_accumulate(L):
    """Profiler feedback against numpy.histogram per (model, batch size,
    class) group, on latencies away from bin edges, with out-of-range,
    negative and non-finite samples rejected and beyond-grid ones in the
    last bin."""
    r = rng(73)
    M, B, C, K = 3, 2, 4, 16
    widths = np.array([0.5, 1.25, 2.0])
    counts = r.integers(0, 5, size=(M, B, C, K)).astype(np.uint32)
    before = counts.copy()
    n = 5000
    mo = r.integers(0, M, size=n)
    bi = r.integers(0, B, size=n)
    cl = r.integers(0, C, size=n)
    lat = (r.integers(0, K + 6, size=n) + r.uniform(0.01, 0.99, size=n)) * widths[mo]
    bad = r.random(n) < 0.05
    lat[bad & (r.random(n) < 0.5)] = -1.0
    lat[bad & (lat >= 0)] = np.nan
    mo[r.random(n) < 0.01] = M
    cl[r.random(n) < 0.01] = -1
    rej = oracle.accumulate(counts, widths, mo, bi, cl, lat, L=L)
    ok = (mo >= 0) & (mo < M) & (cl >= 0) & (cl < C) & np.isfinite(lat) & (lat >= 0)
    assert rej == int((~ok).sum())
    for q in range(M):
        edges = np.concatenate([np.arange(K) * widths[q], [np.inf]])
        for b_ in range(B):
            for c in range(C):
                sel = ok & (mo == q) & (bi == b_) & (cl == c)
                h, _ = np.histogram(lat[sel], bins=edges)
                assert np.array_equal(counts[q, b_, c].astype(np.int64) - before[q, b_, c], h), (q, b_, c)


# ------------------------------------------------------------- affine mode
def _affine(L, rows, bs, w, c0, c1, cls, taus, b=0.05, now=1000.0, cost=None):
    return oracle.score_model_affine(rows, bs, w, c0, c1, cls, now + np.asarray(taus, np.float64),
                                     now, b, want_priority=True, L=L, cost=cost)


def pin_affine_reduces(L):
    """Eq. (3) with c0 = 0 and c1 k = 1 is the tabulated mode on the same
    table, bit for bit (the setting of the toy example in §4.2.2); and for
    a single member at batch size s with c0 = 0, c1 = 1, L_B = s l has the
    table of l stretched s times: each bin split into s equal sub-bins of
    the base width (a brute-force restatement of Eq. (9) for one member)."""
    r = rng(81)
    K, C, n = 24, 3, 5
    rows = r.integers(0, 30, size=(C, K))
    rows[rows.sum(axis=1) == 0, -1] = 1
    cls = r.integers(0, C, size=n)
    taus = np.sort(r.uniform(0.5, 40.0, size=n))
    w = 1.25
    for bs, c1 in (([1], 1.0), ([2], 0.5), ([4], 0.25)):
        aff = _affine(L, rows, bs, w, 0.0, c1, cls, taus)
        tab = run_model(L, rows, cls, taus, w, b=0.05, batch_sizes=bs)
        for k in ("finish_prob", "priority", "expected_finish", "expected_latency_ms", "score"):
            assert np.array_equal(aff[k], tab[k]), (bs, k)
        assert (aff["sel_n"], aff["sel_bs"]) == (tab["sel_n"], tab["sel_bs"])
    bs = [1, 2, 3]
    aff = _affine(L, rows, bs, w, 0.0, 1.0, cls, taus)
    Kf = K * bs[-1]
    per = np.zeros((len(bs), C, Kf), np.int64)
    for bi, s in enumerate(bs):
        per[bi, :, :s * K] = np.repeat(rows, s, axis=1)     # sub-bin j of bin j // s
    tab = run_model(L, None, cls, taus, w, b=0.05, batch_sizes=bs, per_bs_rows=per)
    ai = ti = 0
    for s in bs:                                             # n = 1 of every batch size
        for k in ("expected_latency_ms", "score"):
            assert math.isclose(aff[k][ai], tab[k][ai], rel_tol=1e-12, abs_tol=1e-15), (s, k)
        assert math.isclose(aff["finish_prob"][ti], tab["finish_prob"][ti], rel_tol=1e-12,
                            abs_tol=1e-15), s
        ai += s
        ti += s * (s + 1) // 2


def pin_affine_shift(L):
    """Eq. (3)'s overhead c0 delays the whole batch: raising c0 and every
    deadline by the same amount leaves each finish probability and each
    E[L_B] p_m (the priority before its 1/E[L_B] factor) unchanged and adds
    the amount to E[L_B] (Eq. (5)); a request whose time left is positive
    but at most c0 cannot finish and has priority 0."""
    r = rng(82)
    K, C, n = 30, 4, 6
    rows = r.integers(0, 20, size=(C, K))
    rows[rows.sum(axis=1) == 0, -1] = 1
    cls = r.integers(0, C, size=n)
    taus = np.sort(r.uniform(1.0, 60.0, size=n))
    bs, w, c1 = [1, 3, 6], 0.9, 0.4
    a = _affine(L, rows, bs, w, 0.0, c1, cls, taus)
    sh = 7.3
    z = _affine(L, rows, bs, w, sh, c1, cls, taus + sh)
    assert np.allclose(z["finish_prob"], a["finish_prob"], rtol=1e-12, atol=1e-14)
    assert np.allclose(z["expected_latency_ms"], a["expected_latency_ms"] + sh, rtol=1e-12, atol=0)
    assert np.allclose(z["score"] * z["expected_latency_ms"], a["score"] * a["expected_latency_ms"],
                       rtol=1e-10, atol=1e-14)
    early = _affine(L, rows, [2], w, 5.0, c1, cls[:2], [2.0, 5.0])
    assert np.array_equal(early["finish_prob"], np.zeros(3))
    assert np.array_equal(early["priority"], np.zeros(3))


def pin_affine_nodes(L):
    """At a time left tau = c0 + c1 s w i (a node of the L_B grid) the
    finish probability of a batch of any size is the exact product of its
    members' CDFs at bin edge i (max of independent latencies, §4.2.2, with
    Eq. (3)); beyond the grid it is 1."""
    r = rng(83)
    K, C = 16, 3
    rows = r.integers(0, 12, size=(C, K))
    rows[rows.sum(axis=1) == 0, 0] = 1
    w, c0, c1, bs = 2.0, 3.5, 0.75, [4]
    cls = r.integers(0, C, size=4)
    edges = np.sort(r.integers(1, K, size=3))
    taus = [c0 + c1 * 4 * w * float(i) for i in edges] + [c0 + c1 * 4 * w * (K + 2.5)]
    out = _affine(L, rows, bs, w, c0, c1, cls, taus)
    for nn in range(1, 5):
        G = exact_cdf_product(rows[cls[:nn]])
        for m in range(1, nn + 1):
            want = 1.0 if m == 4 else float(G[int(edges[m - 1])])
            got = out["finish_prob"][slot(nn, m)]
            assert math.isclose(got, want, rel_tol=1e-12, abs_tol=1e-15), (nn, m, got, want)


def pin_affine_monte_carlo(L):
    """Eq. (1) by simulation with L_B = c0 + c1 s max_i l_i (Eq. (3)): draw
    each member's latency from its histogram (uniform inside a bin), an
    anticipated delay ~ Exp(b), and count the members that finish in time
    but not after the delay; its mean matches the score times E[L_B].  The
    sample mean of L_B matches E[L_B] within the half-bin spread of the
    uniform-in-bin model."""
    r = rng(84)
    K, C, n = 20, 3, 3
    rows = r.integers(0, 25, size=(C, K))
    rows[rows.sum(axis=1) == 0, -1] = 1
    cls = r.integers(0, C, size=n)
    w, c0, c1, s, b = 1.0, 4.0, 0.3, 5, 0.06
    taus = np.sort(r.uniform(8.0, 30.0, size=n))
    out = _affine(L, rows, [s], w, c0, c1, cls, taus, b=b)
    G = exact_cdf_product(rows[cls])
    mass = np.array([float(G[k + 1] - G[k]) for k in range(K)])
    S = 1_000_000
    lat = c0 + c1 * s * (r.choice(K, size=S, p=mass / mass.sum()) + r.random(S)) * w
    delay = r.exponential(1.0 / b, size=S)
    ev = sum(((lat <= taus[m]) & (taus[m] < lat + delay)).mean() for m in range(n))
    got = out["score"][n - 1] * out["expected_latency_ms"][n - 1]
    sig = math.sqrt(n * 0.25 / S)
    assert abs(ev - got) <= 4 * sig, (ev, got, sig)
    assert abs(lat.mean() - out["expected_latency_ms"][n - 1]) <= 4 * lat.std() / math.sqrt(S)


PINS = [pin_enumeration, pin_iid_power, pin_point_mass, pin_quadrature_medium, pin_b_to_zero,
        pin_monte_carlo_max, pin_monte_carlo_priority, pin_ozbey_eq8, pin_invariants,
        pin_continuity, pin_edge_cases, pin_selection, pin_rect_mode, pin_toy_example,
        pin_iterate_one_class, pin_iterate_point_mix, pin_iterate_monte_carlo_mix,
        pin_iterate_feasibility_and_popbatch, pin_cost_weights, pin_step_costs, pin_accumulate,
        pin_affine_reduces, pin_affine_shift, pin_affine_nodes, pin_affine_monte_carlo]
