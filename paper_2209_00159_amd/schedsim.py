"""Trace-driven scheduling loop around the scorer (configuration 5's
"re-score at every dispatch decision" stress test).

One worker per model runs one batch at a time (§3.1).  Every tick (0.5 ms
of simulated time) the loop:

  1. admits the trace's arrivals released by now into their model's queue,
     kept sorted by deadline;
  2. for every idle model, drops the requests that can no longer finish
     even if run alone: their time left is below the smallest latency their
     class's batch-size-1 histogram holds mass at (Algorithm 1's drop
     phase, §3.2);
  3. scores every idle model's queue (its first max-batch-size requests:
     no longer prefix is a candidate) and selects one batch per model, all
     in one orloj_score_candidates + orloj_select_batch launch (busy models
     get empty queues);
  4. dispatches each selected batch: its members leave the queue and the
     worker is busy for the batch's latency, sampled as the max of the
     members' latencies (each drawn from its class's batch-size-1
     histogram, scaled by the batch size's scaling factor).

All scoring runs in the HIP library.  TraceLoop keeps the queues and the
clock in Python; NativeTraceLoop runs the same loop in the library's native
runtime (orloj_sched_* and orloj_simulate_trace), with one pinned upload and
one download per round and no Python in the loop.  A decision is one model's
selection with a non-empty batch.  Each decision state (model, queue, time)
can be recorded so that it can be scored again elsewhere.
"""
from __future__ import annotations

import time
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np
import torch

from . import orloj as O
from . import workloads as W


@dataclass
class Decision:
    """One recorded decision state and the selection made in it."""
    model: int
    now_ms: float
    cls: np.ndarray
    deadline_ms: np.ndarray
    sel_n: int
    sel_bs: int


@dataclass
class LoopStats:
    ticks: int = 0
    launches: int = 0
    decisions: int = 0
    dispatched: int = 0
    dropped: int = 0
    on_time: int = 0
    late: int = 0
    wall_s: float = 0.0
    device_s: float = 0.0          # H2D of queues + score + select + D2H, per tick, summed
    sim_ms: float = 0.0
    recorded: List[Decision] = field(default_factory=list)

    def as_dict(self):
        d = {k: v for k, v in self.__dict__.items() if k != "recorded"}
        d["decisions_per_s"] = self.decisions / self.wall_s if self.wall_s else 0.0
        d["decisions_per_device_s"] = self.decisions / self.device_s if self.device_s else 0.0
        d["finish_rate"] = self.on_time / max(1, self.on_time + self.late + self.dropped)
        return d


class TraceLoop:
    def __init__(self, wl: W.Workload, trace, ctx: Optional[O.Context] = None,
                 tick_ms: float = 0.5, seed: int = 0, record_every: int = 0,
                 record_limit: int = 0, tables=None):
        """wl supplies the models' histograms, grids and batch sizes (its
        queues are ignored); trace = (release_ms, model, class, deadline_ms)
        sorted by release.  tables = (ccdf, support) already built on the
        device from wl.counts, or None to build them here."""
        self.ctx = ctx or O.Context()
        self.wl = wl
        self.tick = float(tick_ms)
        self.rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([W.SEED_ROOT, 77, seed])))
        self.record_every = int(record_every)
        self.record_limit = int(record_limit)
        dev = self.ctx.device
        M, B, C, K = wl.counts.shape
        self.M, self.K = M, K
        self.max_bs = int(wl.batch_sizes[-1])
        self.scale = W.linear_scale(wl.batch_sizes)
        self.width = np.asarray(wl.bin_width_ms, np.float64)
        # tables, once
        if tables is None:
            counts = torch.from_numpy(np.ascontiguousarray(wl.counts).view(np.int32)).to(dev)
            self.ccdf = torch.empty(counts.shape, dtype=torch.float32, device=dev)
            self.support = torch.empty(counts.shape[:-1] + (2,), dtype=torch.int32, device=dev)
            self.ctx.build_cdfs(counts, self.ccdf, self.support)
            del counts
        else:
            self.ccdf, self.support = tables
        self.d_width = torch.from_numpy(self.width.copy()).to(dev)
        self.grid = O.make_grid(M, C, K, wl.batch_sizes, self.d_width)
        # batch-size-1 sampling tables and the smallest latency of each class
        c1 = wl.counts[:, 0].astype(np.int64)                    # [M, C, K]
        self.cum1 = np.cumsum(c1, axis=-1)
        first = np.argmax(c1 > 0, axis=-1)                       # [M, C]
        self.min_latency = first * self.width[:, None]
        # device buffers sized for the fullest tick: every model holds max_bs requests
        cap_n = M * self.max_bs
        caps = np.minimum(wl.batch_sizes, self.max_bs).astype(np.int64)
        n_c = M * int(caps.sum())
        n_p = M * int((caps * (caps + 1) // 2).sum())
        pin = dict(pin_memory=True)
        self.h_off = torch.zeros(M + 1, dtype=torch.int64, **pin)
        self.h_cls = torch.zeros(cap_n, dtype=torch.int32, **pin)
        self.h_dl = torch.zeros(cap_n, dtype=torch.float64, **pin)
        self.h_now = torch.zeros(M, dtype=torch.float64, **pin)
        self.h_coff = torch.zeros(M + 1, dtype=torch.int64, **pin)
        self.h_poff = torch.zeros(M + 1, dtype=torch.int64, **pin)
        self.h_sel = torch.zeros(2 * M, dtype=torch.int32, **pin)
        self.d_off = torch.zeros(M + 1, dtype=torch.int64, device=dev)
        self.d_cls = torch.zeros(cap_n, dtype=torch.int32, device=dev)
        self.d_dl = torch.zeros(cap_n, dtype=torch.float64, device=dev)
        self.d_now = torch.zeros(M, dtype=torch.float64, device=dev)
        self.d_coff = torch.zeros(M + 1, dtype=torch.int64, device=dev)
        self.d_poff = torch.zeros(M + 1, dtype=torch.int64, device=dev)
        self.d_P = torch.empty(max(n_p, 1), dtype=torch.float32, device=dev)
        self.d_E = torch.empty(max(n_c, 1), dtype=torch.float64, device=dev)
        self.d_EL = torch.empty(max(n_c, 1), dtype=torch.float32, device=dev)
        self.d_S = torch.empty(max(n_c, 1), dtype=torch.float32, device=dev)
        self.d_sel = torch.zeros(3 * M, dtype=torch.int32, device=dev)
        # simulation state
        self.release, self.model, self.cls, self.deadline = trace
        self.i_next = 0
        empty = (np.zeros(0), np.zeros(0, np.int32))
        self.queues = [empty] * M                      # (deadlines, classes), sorted by deadline
        self.busy_until = np.zeros(M)
        self.now = float(self.release[0]) if len(self.release) else 0.0
        self.stats = LoopStats()

    # -- the host side ---------------------------------------------------------
    def _admit(self, t):
        j = self.i_next
        k = int(np.searchsorted(self.release, t, side="right"))
        if k > j:
            for i in range(j, k):
                q = int(self.model[i])
                dls, cls = self.queues[q]
                d = float(self.deadline[i])
                pos = int(np.searchsorted(dls, d, side="right"))   # equal deadlines keep arrival order
                self.queues[q] = (np.insert(dls, pos, d), np.insert(cls, pos, int(self.cls[i])))
        self.i_next = k

    def _drop(self, q, t):
        dls, cls = self.queues[q]
        if dls.size == 0:
            return
        keep = dls - t > self.min_latency[q][cls]
        if not keep.all():
            self.stats.dropped += int(dls.size - keep.sum())
            self.queues[q] = (dls[keep], cls[keep])

    def _sample_batch_latency(self, q, bi, classes):
        lat = 0.0
        w = self.width[q]
        for c in classes:
            row = self.cum1[q, c]
            u = self.rng.integers(0, row[-1])
            k = int(np.searchsorted(row, u, side="right"))
            lat = max(lat, (k + self.rng.random()) * w)
        return lat * self.scale[bi]

    # -- one tick --------------------------------------------------------------
    def step(self):
        t = self.now
        self._admit(t)
        M = self.M
        idle = self.busy_until <= t
        off = self.h_off.numpy()
        hcls = self.h_cls.numpy()
        hdl = self.h_dl.numpy()
        off[0] = 0
        n = 0
        any_q = False
        for q in range(M):
            if idle[q]:
                self._drop(q, t)
                dls, cls = self.queues[q]
                m = min(dls.size, self.max_bs)
                if m:
                    hdl[n:n + m] = dls[:m]
                    hcls[n:n + m] = cls[:m]
                    n += m
                    any_q = True
            off[q + 1] = n
        self.stats.ticks += 1
        if any_q:
            self._launch(t, n)
        self.now = t + self.tick
        self.stats.sim_ms += self.tick

    def _launch(self, t, n):
        M = self.M
        self.h_now.numpy()[:] = t
        qs = O.make_queues(self.h_off.numpy(), self.d_off, self.d_cls, self.d_dl, self.d_now)
        nc, npb, co, po = O.output_sizes(self.grid, qs, O.PREFIX_TRIANGLE)
        self.h_coff.numpy()[:] = co
        self.h_poff.numpy()[:] = po
        t0 = time.perf_counter()
        self.d_off.copy_(self.h_off, non_blocking=True)
        self.d_cls[:n].copy_(self.h_cls[:n], non_blocking=True)
        self.d_dl[:n].copy_(self.h_dl[:n], non_blocking=True)
        self.d_now.copy_(self.h_now, non_blocking=True)
        self.d_coff.copy_(self.h_coff, non_blocking=True)
        self.d_poff.copy_(self.h_poff, non_blocking=True)
        c = self.ctx
        c._check(c.L.orloj_score_candidates(
            c.ctx, O.ctypes.byref(self.grid), O._ptr(self.ccdf), O._ptr(self.support),
            O.ctypes.byref(qs), float(self.wl.b_expo), O.PREFIX_TRIANGLE,
            O._ptr(self.d_coff), O._ptr(self.d_poff), O._ptr(self.d_P), O._ptr(self.d_E),
            O._ptr(self.d_EL), O._ptr(self.d_S)))
        c._check(c.L.orloj_select_batch(
            c.ctx, O.ctypes.byref(self.grid), O.ctypes.byref(qs), O.PREFIX_TRIANGLE,
            O._ptr(self.d_coff), O._ptr(self.d_S), O._ptr(self.d_sel), O._ptr(self.d_sel[M:]),
            O._ptr(self.d_sel[2 * M:])))
        self.h_sel.copy_(self.d_sel[:2 * M], non_blocking=True)
        c.sync()
        self.stats.device_s += time.perf_counter() - t0
        self.stats.launches += 1
        sel = self.h_sel.numpy()
        off = self.h_off.numpy()
        for q in np.nonzero(sel[:M])[0]:
            q = int(q)
            sn, sb = int(sel[q]), int(sel[M + q])
            dls, cls = self.queues[q]
            st = self.stats
            if self.record_every and st.decisions % self.record_every == 0 and \
                    len(st.recorded) < self.record_limit:
                a, b = int(off[q]), int(off[q + 1])
                st.recorded.append(Decision(q, t, self.h_cls.numpy()[a:b].copy(),
                                            self.h_dl.numpy()[a:b].copy(), sn, sb))
            bi = int(np.searchsorted(self.wl.batch_sizes, sb))
            lat = self._sample_batch_latency(q, bi, cls[:sn])
            done = t + lat
            ok = int((dls[:sn] >= done).sum())
            st.on_time += ok
            st.late += sn - ok
            self.queues[q] = (dls[sn:], cls[sn:])
            self.busy_until[q] = done
            st.decisions += 1
            st.dispatched += sn

    def run(self, until_ms: Optional[float] = None, max_ticks: Optional[int] = None) -> LoopStats:
        """Run ticks until the trace is exhausted and every queue drained (or
        until the simulated clock passes until_ms / max_ticks ticks)."""
        t0 = time.perf_counter()
        ticks = 0
        while True:
            if until_ms is not None and self.now > until_ms:
                break
            if max_ticks is not None and ticks >= max_ticks:
                break
            if self.i_next >= len(self.release) and not any(d.size for d, _ in self.queues):
                break
            self.step()
            ticks += 1
        self.stats.wall_s += time.perf_counter() - t0
        return self.stats


class NativeTraceLoop:
    """The loop of TraceLoop run by the library's native runtime: the same
    tick, drop rule (time left at most the smallest latency the class's
    batch-size-1 histogram holds mass at), scored prefixes, latency model and
    on-time rule, with latencies drawn by the runtime's own generator."""

    def __init__(self, wl: W.Workload, trace, ctx: Optional[O.Context] = None,
                 tick_ms: float = 0.5, seed: int = 0, record_every: int = 0,
                 record_limit: int = 0, tables=None):
        self.ctx = ctx or O.Context()
        self.wl = wl
        self.trace = trace
        self.tick = float(tick_ms)
        self.seed = int(seed)
        self.record_every = int(record_every)
        self.record_limit = int(record_limit)
        dev = self.ctx.device
        M, B, C, K = wl.counts.shape
        if tables is None:
            counts = torch.from_numpy(np.ascontiguousarray(wl.counts).view(np.int32)).to(dev)
            self.ccdf = torch.empty(counts.shape, dtype=torch.float32, device=dev)
            self.support = torch.empty(counts.shape[:-1] + (2,), dtype=torch.int32, device=dev)
            self.ctx.build_cdfs(counts, self.ccdf, self.support)
            del counts
        else:
            self.ccdf, self.support = tables
        self.width = np.asarray(wl.bin_width_ms, np.float64)
        self.d_width = torch.from_numpy(self.width.copy()).to(dev)
        self.grid = O.make_grid(M, C, K, wl.batch_sizes, self.d_width)
        self.solo = np.ascontiguousarray(wl.counts[:, 0])             # [M, C, K]
        first = np.argmax(self.solo > 0, axis=-1)                      # [M, C]
        self.drop_ms = first * self.width[:, None]
        self.sched = O.Sched(self.ctx, self.grid, self.ccdf, self.support, self.drop_ms, wl.b_expo)

    def run(self, max_ticks: int = 0) -> LoopStats:
        st, states = self.sched.simulate(
            self.trace, self.tick, self.solo, self.width, W.linear_scale(self.wl.batch_sizes),
            seed=self.seed, max_ticks=max_ticks, record_every=self.record_every,
            record_limit=self.record_limit)
        self.ctx.sync()
        out = LoopStats(ticks=st["ticks"], launches=st["launches"], decisions=st["decisions"],
                        dispatched=st["dispatched"], dropped=st["dropped"], on_time=st["on_time"],
                        late=st["late"], wall_s=st["wall_s"], device_s=st["device_s"],
                        sim_ms=st["sim_ms"])
        out.recorded = [Decision(m, t, c, d, sn, sb) for m, t, c, d, sn, sb in states]
        self.arrivals = st["arrivals"]
        return out


def config5_trace(n_arrivals: int, models=None, rate_per_s: float = 20_000.0):
    """Configuration 5's Poisson trace (SLO U[1.5,5] x class p50).  With
    `models`, the trace of that subset, its rate scaled by the subset's
    share of the 128 models."""
    p50 = W.config5_p50(models)
    return W.trace5(p50, n_arrivals, rate_per_s * p50.shape[0] / 128.0)


def config5_loop(n_arrivals: int, ctx: Optional[O.Context] = None, models=None, workers: int = 16,
                 rate_per_s: float = 20_000.0, wl: Optional[W.Workload] = None,
                 native: bool = False, **kw):
    """Configuration 5's loop: its models' tables (wl, or generated here)
    and the Poisson trace of n_arrivals at rate_per_s; native=True runs it
    in the library's runtime."""
    if wl is None:
        wl = W.make(5, models=models, workers=workers)
    cls = NativeTraceLoop if native else TraceLoop
    return cls(wl, config5_trace(n_arrivals, models, rate_per_s), ctx=ctx, **kw)
