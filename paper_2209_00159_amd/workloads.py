"""Seeded synthetic workloads for the candidate-batch scorer.

Input construction only.  Each request class gets an analytic execution-time
law shaped like the dynamic-DNN workloads the paper profiles: multi-modal
layer-skipping vision models, text models whose run time grows with a
geometric number of decoding steps, and mixtures of both (Background §2.2,
Evaluation §5 Table 1).  The law is scaled per batch size, discretised into
integer histogram counts on the model's shared bin grid (what the paper's
profiler accumulates, §3.2 "Long-Term Feedback Loop"), and paired with
deadline-ordered request queues (release time plus SLO, Problem Statement
§3.1).

None of the scoring arithmetic (CDFs of the counts, products, priorities)
lives here: the HIP path and the CPU oracle both receive these counts and
queues as plain inputs.  The paper's datasets and the Azure trace it replays
are not available; these seeded generators stand in for them.

Every random draw comes from numpy's PCG64 seeded with
``SeedSequence([2209_00159, config_id])`` and spawned per model, so one
model's inputs can be regenerated alone.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Callable, List, Optional, Sequence

import numpy as np
from scipy import optimize, special

SEED_ROOT = 2209_00159
COUNT_TOTAL = 1 << 20          # histogram samples per (model, batch size, class)
DEFAULT_B_EXPO = 1e-4          # anticipated-delay rate per ms (paper §4.4)


# --------------------------------------------------------------------------
# Execution-time laws (milliseconds).  cdf(x) is P(latency <= x) of the law
# at batch size 1; the batch-size scaling multiplies the latency.
# --------------------------------------------------------------------------
@dataclasses.dataclass
class LogNormalMix:
    """Mixture of lognormals given by (median_ms, sigma_log, weight)."""
    medians: np.ndarray
    sigmas: np.ndarray
    weights: np.ndarray

    def cdf(self, x: np.ndarray) -> np.ndarray:
        x = np.asarray(x, dtype=np.float64)
        out = np.zeros_like(x)
        pos = x > 0
        lx = np.log(x[pos])
        acc = np.zeros_like(lx)
        for m, s, w in zip(self.medians, self.sigmas, self.weights):
            acc += w * special.ndtr((lx - math.log(m)) / s)
        out[pos] = acc
        return out


@dataclasses.dataclass
class NormalMix:
    """Mixture of normal modes (mean_ms, sd_ms, weight); mass below 0 is
    folded into the first bin by the count quantiser."""
    means: np.ndarray
    sds: np.ndarray
    weights: np.ndarray

    def cdf(self, x: np.ndarray) -> np.ndarray:
        x = np.asarray(x, dtype=np.float64)
        acc = np.zeros_like(x)
        for m, s, w in zip(self.means, self.sds, self.weights):
            acc += w * special.ndtr((x - m) / s)
        return acc


@dataclasses.dataclass
class GeometricSteps:
    """base + step * N with N ~ Geometric(p) on {1, 2, ...}: a decoder whose
    number of generated tokens is geometric."""
    base: float
    step: float
    p: float

    def cdf(self, x: np.ndarray) -> np.ndarray:
        x = np.asarray(x, dtype=np.float64)
        j = np.floor((x - self.base) / self.step)
        j = np.maximum(j, 0.0)
        return np.where(j >= 1.0, -np.expm1(j * math.log1p(-self.p)), 0.0)

    def median(self) -> float:
        j = math.ceil(math.log(0.5) / math.log1p(-self.p))
        return self.base + self.step * j

    def min_latency(self) -> float:
        return self.base + self.step


def law_median(law) -> float:
    """p50 of a law at batch size 1 (analytic where closed, else bisection
    on the analytic CDF)."""
    if isinstance(law, GeometricSteps):
        return law.median()
    if isinstance(law, LogNormalMix) and len(law.medians) == 1:
        return float(law.medians[0])
    hi = 1.0
    while law.cdf(np.array([hi]))[0] < 0.5:
        hi *= 2.0
    return float(optimize.brentq(lambda v: law.cdf(np.array([v]))[0] - 0.5,
                                 1e-9, hi, xtol=1e-12))


def quantise_counts(cdf_at_grid: np.ndarray, total: int = COUNT_TOTAL) -> np.ndarray:
    """Integer histogram counts from an analytic CDF sampled at the K+1 grid
    points (last axis).  Cumulative rounding keeps the total exactly equal
    to ``total``; mass below the first grid point goes to bin 0 and mass
    beyond the last grid point to bin K-1 (the shared grid clips)."""
    cum = np.rint(cdf_at_grid * float(total))
    cum[..., 0] = 0.0
    cum[..., -1] = float(total)
    cum = np.maximum.accumulate(cum, axis=-1)
    counts = np.diff(cum, axis=-1)
    if total < (1 << 32):
        return counts.astype(np.uint32)
    raise ValueError("total must fit uint32 bins")


# --------------------------------------------------------------------------
# Workload container
# --------------------------------------------------------------------------
@dataclasses.dataclass
class Workload:
    name: str
    config_id: int
    n_models: int
    n_classes: int
    n_bins: int
    batch_sizes: np.ndarray        # int32 [B], strictly increasing
    bin_width_ms: np.ndarray       # float64 [M]
    counts: np.ndarray             # uint32 [M, B, C, K]
    queue_off: np.ndarray          # int64 [M+1]
    cls: np.ndarray                # int32 [N_total]
    deadline_ms: np.ndarray        # float64 [N_total], sorted within a model
    now_ms: np.ndarray             # float64 [M]
    b_expo: float = DEFAULT_B_EXPO
    description: str = ""
    cost: Optional[np.ndarray] = None  # float64 [N_total] miss cost per request (None: 1)
    class_p50_ms: Optional[np.ndarray] = None  # float64 [M, C] analytic class medians at batch size 1
    bs_scale: Optional[np.ndarray] = None      # float64 [B] latency scale of each batch size
    # Affine batch-latency mode (a batch of size s whose slowest member takes
    # l runs c0 + c1 s l): counts is then [M, C, K], one solo-latency
    # histogram per class, and these hold the per-model constants.
    c0_ms: Optional[np.ndarray] = None  # float64 [M]
    c1: Optional[np.ndarray] = None     # float64 [M]

    @property
    def affine(self) -> bool:
        return self.c1 is not None

    @property
    def n_bs(self) -> int:
        return int(self.batch_sizes.shape[0])

    def queue_len(self, q: int) -> int:
        return int(self.queue_off[q + 1] - self.queue_off[q])

    def model(self, q: int) -> dict:
        a, b = int(self.queue_off[q]), int(self.queue_off[q + 1])
        return dict(counts=self.counts[q], cls=self.cls[a:b],
                    deadline_ms=self.deadline_ms[a:b], now_ms=float(self.now_ms[q]),
                    bin_width_ms=float(self.bin_width_ms[q]),
                    cost=None if self.cost is None else self.cost[a:b])

    def subset(self, models: Sequence[int]) -> "Workload":
        """A workload made of the listed models only (same grid shapes)."""
        models = list(models)
        offs = [0]
        cls, dl, co = [], [], []
        for q in models:
            a, b = int(self.queue_off[q]), int(self.queue_off[q + 1])
            cls.append(self.cls[a:b])
            dl.append(self.deadline_ms[a:b])
            if self.cost is not None:
                co.append(self.cost[a:b])
            offs.append(offs[-1] + (b - a))
        return Workload(
            name=f"{self.name}[{len(models)} models]", config_id=self.config_id,
            n_models=len(models), n_classes=self.n_classes, n_bins=self.n_bins,
            batch_sizes=self.batch_sizes.copy(),
            bin_width_ms=self.bin_width_ms[models].copy(),
            counts=np.ascontiguousarray(self.counts[models]),
            queue_off=np.asarray(offs, dtype=np.int64),
            cls=np.concatenate(cls).astype(np.int32) if cls else np.zeros(0, np.int32),
            deadline_ms=np.concatenate(dl) if dl else np.zeros(0),
            now_ms=self.now_ms[models].copy(), b_expo=self.b_expo,
            description=self.description,
            cost=(np.concatenate(co) if co else np.zeros(0)) if self.cost is not None else None,
            class_p50_ms=None if self.class_p50_ms is None else self.class_p50_ms[models].copy(),
            bs_scale=self.bs_scale,
            c0_ms=None if self.c0_ms is None else self.c0_ms[models].copy(),
            c1=None if self.c1 is None else self.c1[models].copy())

    def with_queues(self, queues: List[tuple], now_ms: np.ndarray) -> "Workload":
        """Same histograms, new queues: ``queues[q] = (cls, deadline_ms)``."""
        offs = np.zeros(self.n_models + 1, dtype=np.int64)
        for q, (c, _) in enumerate(queues):
            offs[q + 1] = offs[q] + len(c)
        cls = np.concatenate([np.asarray(c, np.int32) for c, _ in queues]) \
            if queues else np.zeros(0, np.int32)
        dl = np.concatenate([np.asarray(d, np.float64) for _, d in queues]) \
            if queues else np.zeros(0)
        return dataclasses.replace(self, queue_off=offs, cls=cls.astype(np.int32),
                                   deadline_ms=dl, now_ms=np.asarray(now_ms, np.float64),
                                   cost=None)


def _sorted_queue(cls: np.ndarray, deadline: np.ndarray):
    order = np.argsort(deadline, kind="stable")
    return cls[order].astype(np.int32), deadline[order].astype(np.float64)


def _aged_backlog(rng, n, n_classes, slo_of_class: Callable, now):
    """n pending requests with uniform class; each was released an age
    ~ U[0, SLO/2) ago, so its deadline = now - age + SLO."""
    cls = rng.integers(0, n_classes, size=n)
    slo = slo_of_class(rng, cls)
    age = rng.uniform(0.0, 0.5, size=n) * slo
    return _sorted_queue(cls, now - age + slo)


def _poisson_backlog(rng, n_arrivals, rate_per_ms, n_classes, slo_of_class: Callable, now,
                     min_latency=None):
    """n_arrivals Poisson arrivals ending at ``now``.  Requests the
    scheduler has already timed out are gone from the queue (Algorithm 1's
    drop phase, read with a point estimate of a request's latency run
    alone): the deadline has passed, or the time left is at most
    ``min_latency[c]`` of the request's class (its analytic median at
    batch size 1)."""
    gaps = rng.exponential(1.0 / rate_per_ms, size=n_arrivals)
    release = now - np.cumsum(gaps)
    cls = rng.integers(0, n_classes, size=n_arrivals)
    deadline = release + slo_of_class(rng, cls)
    alive = deadline > now
    if min_latency is not None:
        alive &= (deadline - now) > np.asarray(min_latency)[cls]
    return _sorted_queue(cls[alive], deadline[alive])


def _grid_counts(laws, scales, n_bins, width, total=COUNT_TOTAL):
    """counts[B, C, K] of latency scale_b * l for each class law."""
    x = np.arange(n_bins + 1, dtype=np.float64) * width
    out = np.empty((len(scales), len(laws), n_bins), dtype=np.uint32)
    for bi, s in enumerate(scales):
        xs = x / s
        for c, law in enumerate(laws):
            out[bi, c] = quantise_counts(law.cdf(xs), total)
    return out


def _lognormal_mix_grid_counts(medians, sigmas, weights, scales, n_bins, width,
                               total=COUNT_TOTAL):
    """Vectorised counts[B, C, K] for lognormal-mixture classes
    (medians/sigmas/weights shaped [C, J])."""
    x = np.arange(1, n_bins + 1, dtype=np.float64) * width
    lx = np.log(x)[None, None, :]                       # [1,1,K]
    ls = np.log(np.asarray(scales, np.float64))
    out = np.empty((len(scales), medians.shape[0], n_bins), dtype=np.uint32)
    for bi in range(len(scales)):
        acc = np.zeros((medians.shape[0], n_bins))
        for j in range(medians.shape[1]):
            z = (lx[0] - ls[bi] - np.log(medians[:, j])[:, None]) / sigmas[:, j][:, None]
            acc += weights[:, j][:, None] * special.ndtr(z)
        grid = np.concatenate([np.zeros((acc.shape[0], 1)), acc], axis=1)
        out[bi] = quantise_counts(grid, total)
    return out


def linear_scale(b):
    return 1.0 + 0.08 * (np.asarray(b, np.float64) - 1.0)


def _model_streams(config_id: int, n_models: int):
    ss = np.random.SeedSequence([SEED_ROOT, config_id])
    return [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(n_models)]


# --------------------------------------------------------------------------
# The five configurations
# --------------------------------------------------------------------------
def config1(slo_scale: float = 1.0) -> Workload:
    """Tiny single model: 4 lognormal classes, 128 bins over 0-200 ms,
    batch sizes 1..16 with latency scale 1+0.08(b-1), 64 queued requests
    with SLO ~ U[50, 300] ms."""
    rng = _model_streams(1, 1)[0]
    C, K, span = 4, 128, 200.0
    bs = np.arange(1, 17, dtype=np.int32)
    w = span / K
    mu = rng.uniform(3.0, 4.5, size=C)
    sig = rng.uniform(0.2, 0.6, size=C)
    laws = [LogNormalMix(np.array([math.exp(m)]), np.array([s]), np.array([1.0]))
            for m, s in zip(mu, sig)]
    counts = _grid_counts(laws, linear_scale(bs), K, w)[None]
    now = 60_000.0
    cls, dl = _aged_backlog(rng, 64, C, lambda r, c: slo_scale * r.uniform(50.0, 300.0, size=c.size), now)
    return Workload("cfg1-tiny", 1, 1, C, K, bs, np.array([w]), counts,
                    np.array([0, cls.size], np.int64), cls, dl, np.array([now]),
                    description=config1.__doc__, class_p50_ms=np.exp(mu)[None],
                    bs_scale=linear_scale(bs))


def config2(slo_scale: float = 1.0) -> Workload:
    """Dynamic-NLP-like single model: 32 classes of base + step x Geom(0.02)
    steps, 1024 bins over 0-2 s, batch sizes 1..64, 1024 Poisson arrivals
    at 500 req/s with SLO U[2,5] x the class median (expired ones dropped)."""
    rng = _model_streams(2, 1)[0]
    C, K, span = 32, 1024, 2000.0
    bs = np.arange(1, 65, dtype=np.int32)
    w = span / K
    base = rng.uniform(10.0, 40.0, size=C)
    step = np.exp(rng.uniform(math.log(1.0), math.log(10.0), size=C))
    laws = [GeometricSteps(float(b0), float(k0), 0.02) for b0, k0 in zip(base, step)]
    med = np.array([law_median(l) for l in laws])
    counts = _grid_counts(laws, linear_scale(bs), K, w)[None]
    now = 60_000.0
    cls, dl = _poisson_backlog(rng, 1024, 0.5, C,
                               lambda r, c: slo_scale * r.uniform(2.0, 5.0, size=c.size) * med[c], now,
                               min_latency=med)
    return Workload("cfg2-nlp", 2, 1, C, K, bs, np.array([w]), counts,
                    np.array([0, cls.size], np.int64), cls, dl, np.array([now]),
                    description=config2.__doc__, class_p50_ms=med[None],
                    bs_scale=linear_scale(bs))


def config3(slo_scale: float = 1.0) -> Workload:
    """Layer-skipping-CV-like single model: 64 classes mixing normal modes
    at 5/12/25 ms (sd 10% of the mean, Dirichlet(1,1,1) weights), 2048 bins
    over 0-60 ms, batch sizes 1..128 with latency scale b^0.6, 4096 queued
    requests with SLO U[1.5,4] x the class p50."""
    rng = _model_streams(3, 1)[0]
    C, K, span = 64, 2048, 60.0
    bs = np.arange(1, 129, dtype=np.int32)
    w = span / K
    modes = np.array([5.0, 12.0, 25.0])
    wts = rng.dirichlet([1.0, 1.0, 1.0], size=C)
    laws = [NormalMix(modes, 0.1 * modes, wt) for wt in wts]
    p50 = np.array([law_median(l) for l in laws])
    counts = _grid_counts(laws, np.power(bs.astype(np.float64), 0.6), K, w)[None]
    now = 60_000.0
    cls, dl = _aged_backlog(rng, 4096, C,
                            lambda r, c: slo_scale * r.uniform(1.5, 4.0, size=c.size) * p50[c], now)
    return Workload("cfg3-cv", 3, 1, C, K, bs, np.array([w]), counts,
                    np.array([0, cls.size], np.int64), cls, dl, np.array([now]),
                    description=config3.__doc__, class_p50_ms=p50[None],
                    bs_scale=np.power(bs.astype(np.float64), 0.6))


def _mixture_models(config_id, M, C, K, span, bs, med_lo, med_hi, queue_fn,
                    models: Optional[Sequence[int]] = None, workers: int = 1):
    streams = _model_streams(config_id, M)
    models = list(range(M) if models is None else models)
    w = span / K
    scales = linear_scale(bs)
    counts = np.empty((len(models), len(bs), C, K), dtype=np.uint32)
    queues = [None] * len(models)
    nows = np.zeros(len(models))
    p50s = np.zeros((len(models), C))

    def one(i):
        rng = streams[models[i]]
        medians = rng.uniform(med_lo, med_hi, size=(C, 2))
        sigmas = rng.uniform(0.2, 0.6, size=(C, 2))
        w0 = rng.uniform(0.2, 0.8, size=C)
        weights = np.stack([w0, 1.0 - w0], axis=1)
        counts[i] = _lognormal_mix_grid_counts(medians, sigmas, weights, scales, K, w)
        p50 = np.array([law_median(LogNormalMix(medians[c], sigmas[c], weights[c]))
                        for c in range(C)])
        now = 60_000.0 + rng.uniform(0.0, 1.0)
        queues[i] = queue_fn(rng, C, p50, now)
        nows[i] = now
        p50s[i] = p50

    if workers > 1 and len(models) > 1:
        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(workers) as ex:
            list(ex.map(one, range(len(models))))
    else:
        for i in range(len(models)):
            one(i)
    return counts, queues, nows, w, p50s


def _assemble(name, cid, C, K, bs, counts, queues, nows, w, doc, p50s=None):
    M = counts.shape[0]
    offs = np.zeros(M + 1, dtype=np.int64)
    for q, (c, _) in enumerate(queues):
        offs[q + 1] = offs[q] + c.size
    cls = np.concatenate([c for c, _ in queues]).astype(np.int32)
    dl = np.concatenate([d for _, d in queues])
    return Workload(name, cid, M, C, K, bs, np.full(M, w), counts, offs, cls, dl,
                    nows, description=doc, class_p50_ms=p50s, bs_scale=linear_scale(bs))


def config4(models: Optional[Sequence[int]] = None, workers: int = 1,
            slo_scale: float = 1.0) -> Workload:
    """Multi-model, one launch: 64 models x 16 classes of two-component
    lognormal mixtures (medians U[20,200] ms, sigma U[0.2,0.6], weight
    U[0.2,0.8]), 1024 bins over 0-1000 ms, batch sizes 1..32; per model 2048
    Poisson arrivals at 500 req/s with SLO U[2,5] x the class median."""
    C, K, M = 16, 1024, 64
    bs = np.arange(1, 33, dtype=np.int32)

    def qfn(rng, C_, p50, now):
        return _poisson_backlog(rng, 2048, 0.5, C_,
                                lambda r, c: slo_scale * r.uniform(2.0, 5.0, size=c.size) * p50[c],
                                now, min_latency=p50)
    counts, queues, nows, w, p50s = _mixture_models(4, M, C, K, 1000.0, bs, 20.0, 200.0, qfn,
                                                    models, workers)
    return _assemble("cfg4-multi", 4, C, K, bs, counts, queues, nows, w, config4.__doc__, p50s)


CFG5_BACKLOG = 256

# models of the multi-model configurations
CONFIG_MODELS = {4: 64, 5: 128}


def config5(models: Optional[Sequence[int]] = None, workers: int = 1,
            slo_scale: float = 1.0) -> Workload:
    """Scheduling-loop stress, saturated decision state: 128 models x 32
    classes of two-component lognormal mixtures (medians U[5,40] ms), 4096
    bins over 0-1000 ms, batch sizes 1..64; every model holds a backlog of
    256 pending requests with SLO U[1.5,5] x the class p50, so each batch
    size's full triangle of prefix candidates is scored."""
    C, K, M = 32, 4096, 128
    bs = np.arange(1, 65, dtype=np.int32)

    def qfn(rng, C_, p50, now):
        return _aged_backlog(rng, CFG5_BACKLOG, C_,
                             lambda r, c: slo_scale * r.uniform(1.5, 5.0, size=c.size) * p50[c], now)
    counts, queues, nows, w, p50s = _mixture_models(5, M, C, K, 1000.0, bs, 5.0, 40.0, qfn,
                                                    models, workers)
    return _assemble("cfg5-stress", 5, C, K, bs, counts, queues, nows, w, config5.__doc__, p50s)


def config5_p50(models: Optional[Sequence[int]] = None) -> np.ndarray:
    """Class p50 (ms, batch size 1) of config 5's models: [M, C].  Used to
    draw SLOs for the arrival trace."""
    M, C = 128, 32
    streams = _model_streams(5, M)
    models = range(M) if models is None else models
    out = []
    for q in models:
        rng = streams[q]
        medians = rng.uniform(5.0, 40.0, size=(C, 2))
        sigmas = rng.uniform(0.2, 0.6, size=(C, 2))
        w0 = rng.uniform(0.2, 0.8, size=C)
        weights = np.stack([w0, 1.0 - w0], axis=1)
        out.append([law_median(LogNormalMix(medians[c], sigmas[c], weights[c]))
                    for c in range(C)])
    return np.asarray(out)


def trace5(p50: np.ndarray, n_arrivals: int = 1_000_000, rate_per_s: float = 20_000.0,
           seed_extra: int = 0):
    """Config 5's open-loop arrival trace: Poisson arrivals at ``rate_per_s``
    spread uniformly over models and classes, SLO U[1.5,5] x the class p50.
    Returns (release_ms, model, class, deadline_ms), sorted by release."""
    rng = np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([SEED_ROOT, 5, 1_000_003 + seed_extra])))
    M, C = p50.shape
    release = np.cumsum(rng.exponential(1000.0 / rate_per_s, size=n_arrivals))
    model = rng.integers(0, M, size=n_arrivals).astype(np.int32)
    cls = rng.integers(0, C, size=n_arrivals).astype(np.int32)
    slo = rng.uniform(1.5, 5.0, size=n_arrivals) * p50[model, cls]
    return release, model, cls, release + slo


CONFIGS = {1: config1, 2: config2, 3: config3, 4: config4, 5: config5}


def make(config_id: int, models: Optional[Sequence[int]] = None, workers: int = 1,
         slo_scale: float = 1.0) -> Workload:
    """Configuration ``config_id`` (1..5).  ``slo_scale`` multiplies every
    SLO draw (the paper sweeps SLO multiples; 1.0 is the configuration as
    specified)."""
    if config_id in (4, 5):
        wl = CONFIGS[config_id](models, workers, slo_scale)
    else:
        if models is not None and list(models) != [0]:
            raise ValueError("single-model configs have only model 0")
        wl = CONFIGS[config_id](slo_scale)
    if slo_scale != 1.0:
        wl.name = f"{wl.name}-slo{slo_scale:g}x"
    return wl


# --------------------------------------------------------------------------
# Affine batch-latency mode inputs
# --------------------------------------------------------------------------
def affine(wl: Workload) -> Workload:
    """The affine-mode counterpart of a configuration: each class keeps its
    batch-size-1 histogram as the solo-latency histogram (counts [M, C, K]),
    and the model's batch law c0 + c1 s l is the secant of the
    configuration's scaling law scale(s) l between the smallest and the
    largest batch size, at the model's fastest class median m:
        c1 = (scale(s_max) - scale(s_min)) / (s_max - s_min),
        c0 = (scale(s_min) - c1 s_min) m.
    (For 1 + 0.08 (s - 1): c1 = 0.08, c0 = 0.92 m.)  A fixed overhead above
    what the fastest class needs would leave the earliest deadlines no
    chance.  Queues, grid and batch sizes are unchanged."""
    if wl.class_p50_ms is None or wl.bs_scale is None:
        raise ValueError(f"{wl.name} records no class medians or scaling law")
    if wl.affine:
        return wl
    bs = np.asarray(wl.batch_sizes, np.float64)
    sc = np.asarray(wl.bs_scale, np.float64)
    c1 = (sc[-1] - sc[0]) / (bs[-1] - bs[0]) if bs.size > 1 else 0.0
    if not c1 > 0.0:
        raise ValueError("the scaling law must grow with the batch size")
    m = np.min(np.asarray(wl.class_p50_ms, np.float64), axis=1)
    return dataclasses.replace(
        wl, name=f"{wl.name}-affine", counts=np.ascontiguousarray(wl.counts[:, 0]),
        c0_ms=(sc[0] - c1 * bs[0]) * m, c1=np.full(wl.n_models, float(c1)))


def random_affine(seed: int, c0_range=(0.0, 3.0), c1_range=(0.05, 1.0), **kw) -> Workload:
    """random_case with one histogram per class (its batch-size-0 table) and
    per-model constants c0 ~ U[c0_range] ms, c1 ~ U[c1_range]."""
    wl = random_case(seed, **kw)
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_ROOT, 98, seed])))
    M = wl.n_models
    return dataclasses.replace(
        wl, name=f"{wl.name}-affine", counts=np.ascontiguousarray(wl.counts[:, 0]),
        c0_ms=rng.uniform(*c0_range, size=M), c1=rng.uniform(*c1_range, size=M))


# --------------------------------------------------------------------------
# Small random cases for tests (edge cases, ragged shapes)
# --------------------------------------------------------------------------
def random_case(seed: int, n_models=2, n_classes=3, n_bins=37, batch_sizes=(1, 2, 3, 5, 8),
                queue_lens=None, width_ms=None, total=1000, sparsity=0.3,
                tau_range=(-5.0, 60.0), b_expo=DEFAULT_B_EXPO, now_ms=1_000.0) -> Workload:
    """Random small workload: random integer histograms (some bins forced
    empty), random queues whose time-to-deadline spans dead, in-grid and
    beyond-grid requests."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_ROOT, 99, seed])))
    bs = np.asarray(batch_sizes, dtype=np.int32)
    M, C, K = n_models, n_classes, n_bins
    if queue_lens is None:
        queue_lens = rng.integers(0, 12, size=M)
    counts = rng.integers(0, total, size=(M, bs.size, C, K)).astype(np.uint32)
    counts[rng.random(counts.shape) < sparsity] = 0
    empty = counts.sum(axis=-1) == 0
    counts[..., -1][empty] = 1
    widths = np.asarray(width_ms if width_ms is not None else rng.uniform(0.5, 2.0, size=M),
                        dtype=np.float64).reshape(M)
    queues, nows = [], []
    for q in range(M):
        n = int(queue_lens[q])
        now = float(now_ms) + q * 3.25
        cls = rng.integers(0, C, size=n)
        tau = rng.uniform(tau_range[0], tau_range[1], size=n)
        queues.append(_sorted_queue(cls, now + tau))
        nows.append(now)
    offs = np.zeros(M + 1, dtype=np.int64)
    for q, (c, _) in enumerate(queues):
        offs[q + 1] = offs[q] + c.size
    cls = np.concatenate([c for c, _ in queues]).astype(np.int32) if M else np.zeros(0, np.int32)
    dl = np.concatenate([d for _, d in queues]) if M else np.zeros(0)
    return Workload(f"random{seed}", 0, M, C, K, bs, widths, counts, offs, cls, dl,
                    np.asarray(nows), b_expo=b_expo)
