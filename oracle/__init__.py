"""CPU oracle for candidate-batch scoring (test infrastructure).

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The HIP library never loads it and
shares no code with it.  The arithmetic lives in ``orloj_oracle.c`` (plain
fp64 C, one step per quantity the paper defines); this module only
marshals numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

from . import build as _build

_LIB = None

_I32P = ctypes.POINTER(ctypes.c_int32)
_U32P = ctypes.POINTER(ctypes.c_uint32)
_F64P = ctypes.POINTER(ctypes.c_double)
_I64P = ctypes.POINTER(ctypes.c_int64)


def lib(path: Optional[str] = None):
    """Load the oracle library (built by ``oracle/build.py``).  ``path``
    loads another build of the oracle source (used by the mutation tests)."""
    global _LIB
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _LIB is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        _LIB = _bind(ctypes.CDLL(_build.LIB))
    return _LIB


def _bind(L):
    L.orloj_oracle_cdf.argtypes = [ctypes.c_int32, _U32P, _F64P]
    L.orloj_oracle_cdf.restype = ctypes.c_int
    L.orloj_oracle_batch_cdf.argtypes = [ctypes.c_int32, ctypes.c_int32, _U32P, _F64P]
    L.orloj_oracle_batch_cdf.restype = ctypes.c_int
    L.orloj_oracle_score_model.argtypes = [
        ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _I32P, ctypes.c_double,
        _U32P, ctypes.c_int64, _I32P, _F64P, _F64P, ctypes.c_double, ctypes.c_double,
        ctypes.c_int32, _F64P, _F64P, _F64P, _F64P, _F64P, _I32P, _I32P, _F64P]
    L.orloj_oracle_score_model.restype = ctypes.c_int
    L.orloj_oracle_iterate_model.argtypes = [
        ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _I32P, ctypes.c_double, _U32P, _F64P,
        ctypes.c_int64, _I32P, _F64P, _F64P, _I64P, _F64P, _F64P, ctypes.c_double,
        ctypes.c_double, _I32P, _F64P, _I32P, _I32P, _I32P]
    L.orloj_oracle_accumulate.argtypes = [
        ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _F64P, ctypes.c_int64,
        _I32P, _I32P, _I32P, _F64P, _U32P, _I64P]
    L.orloj_oracle_accumulate.restype = ctypes.c_int
    L.orloj_oracle_score_model_affine.argtypes = [
        ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _I32P, ctypes.c_double, _U32P,
        ctypes.c_double, ctypes.c_double, ctypes.c_int64, _I32P, _F64P, _F64P, ctypes.c_double,
        ctypes.c_double, ctypes.c_int32, _F64P, _F64P, _F64P, _F64P, _F64P, _I32P, _I32P, _F64P]
    L.orloj_oracle_score_model_affine.restype = ctypes.c_int
    L.orloj_oracle_iterate_model.restype = ctypes.c_int
    return L


def _p(a, t):
    return a.ctypes.data_as(t)


class OracleError(RuntimeError):
    pass


def cdf(counts_row, L=None) -> np.ndarray:
    L = L or lib()
    c = np.ascontiguousarray(counts_row, dtype=np.uint32)
    out = np.empty(c.size + 1, dtype=np.float64)
    rc = L.orloj_oracle_cdf(c.size, _p(c, _U32P), _p(out, _F64P))
    if rc:
        raise OracleError(f"orloj_oracle_cdf rc={rc}")
    return out


def batch_cdf(rows, L=None) -> np.ndarray:
    """CDF of the batch latency at the grid points for member count rows
    [n, K]."""
    L = L or lib()
    r = np.ascontiguousarray(rows, dtype=np.uint32)
    if r.ndim != 2:
        raise ValueError("rows must be [n_members, n_bins]")
    out = np.empty(r.shape[1] + 1, dtype=np.float64)
    rc = L.orloj_oracle_batch_cdf(r.shape[1], r.shape[0], _p(r, _U32P), _p(out, _F64P))
    if rc:
        raise OracleError(f"orloj_oracle_batch_cdf rc={rc}")
    return out


def ncap(batch_sizes, n_queue: int, prefix_mode: int = 0) -> np.ndarray:
    bs = np.asarray(batch_sizes, dtype=np.int64)
    return np.full(bs.size, n_queue, np.int64) if prefix_mode else np.minimum(bs, n_queue)


def output_sizes(queue_off, batch_sizes, prefix_mode: int = 0):
    """Candidate and member offsets per model: (cand_off[M+1], prob_off[M+1])."""
    qo = np.asarray(queue_off, dtype=np.int64)
    M = qo.size - 1
    cand_off = np.zeros(M + 1, np.int64)
    prob_off = np.zeros(M + 1, np.int64)
    for q in range(M):
        caps = ncap(batch_sizes, int(qo[q + 1] - qo[q]), prefix_mode)
        cand_off[q + 1] = cand_off[q] + caps.sum()
        prob_off[q + 1] = prob_off[q] + (caps * (caps + 1) // 2).sum()
    return cand_off, prob_off


def _opt64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float64)


def _map_models(fn, models, threads):
    """fn(q) over the models, in order; with threads > 1 on a pool of host
    threads (each call is one C function, which releases Python's lock)."""
    if threads is None or threads <= 1 or len(models) <= 1:
        return [fn(q) for q in models]
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(min(int(threads), len(models))) as ex:
        return list(ex.map(fn, models))


def score_model(counts, batch_sizes, bin_width_ms, cls, deadline_ms, now_ms, b_expo,
                prefix_mode: int = 0, want_priority: bool = False, L=None, cost=None) -> dict:
    """All candidates of one model (see orloj_oracle_score_model)."""
    L = L or lib()
    cnt = np.ascontiguousarray(counts, dtype=np.uint32)
    B, C, K = cnt.shape
    bs = np.ascontiguousarray(batch_sizes, dtype=np.int32)
    cl = np.ascontiguousarray(cls, dtype=np.int32)
    dl = np.ascontiguousarray(deadline_ms, dtype=np.float64)
    caps = ncap(bs, cl.size, prefix_mode)
    n_cand = int(caps.sum())
    n_prob = int((caps * (caps + 1) // 2).sum())
    P = np.empty(n_prob)
    pr = np.empty(n_prob) if want_priority else None
    E = np.empty(n_cand)
    EL = np.empty(n_cand)
    S = np.empty(n_cand)
    sn = np.zeros(1, np.int32)
    sb = np.zeros(1, np.int32)
    ss = np.zeros(1)
    co = _opt64(cost)
    rc = L.orloj_oracle_score_model(
        C, K, B, _p(bs, _I32P), float(bin_width_ms), _p(cnt, _U32P), cl.size,
        _p(cl, _I32P), _p(dl, _F64P), _p(co, _F64P) if co is not None else None,
        float(now_ms), float(b_expo), int(prefix_mode),
        _p(P, _F64P), _p(pr, _F64P) if pr is not None else None, _p(E, _F64P),
        _p(EL, _F64P), _p(S, _F64P), _p(sn, _I32P), _p(sb, _I32P), _p(ss, _F64P))
    if rc:
        raise OracleError(f"orloj_oracle_score_model rc={rc}")
    out = dict(finish_prob=P, expected_finish=E, expected_latency_ms=EL, score=S,
               sel_n=int(sn[0]), sel_bs=int(sb[0]), sel_score=float(ss[0]))
    if pr is not None:
        out["priority"] = pr
    return out


def score_workload(wl, prefix_mode: int = 0, models: Optional[Sequence[int]] = None,
                   want_priority: bool = False, L=None, threads: int = 1) -> dict:
    """Score every model of a workload (or the listed ones); outputs are
    concatenated in model order, as the HIP library lays them out.
    ``threads`` > 1 scores the models on that many host threads."""
    models = list(range(wl.n_models)) if models is None else list(models)

    def one(q):
        m = wl.model(q)
        return score_model(m["counts"], wl.batch_sizes, m["bin_width_ms"], m["cls"],
                           m["deadline_ms"], m["now_ms"], wl.b_expo, prefix_mode,
                           want_priority, L, cost=m["cost"])

    parts = _map_models(one, models, threads)
    cat = lambda k: (np.concatenate([p[k] for p in parts]) if parts else np.zeros(0))
    out = {k: cat(k) for k in ("finish_prob", "expected_finish", "expected_latency_ms", "score")}
    if want_priority:
        out["priority"] = cat("priority")
    out["sel_n"] = np.array([p["sel_n"] for p in parts], np.int32)
    out["sel_bs"] = np.array([p["sel_bs"] for p in parts], np.int32)
    out["sel_score"] = np.array([p["sel_score"] for p in parts])
    out["per_model"] = parts
    return out


def iterate_model(counts, batch_sizes, bin_width_ms, cls, deadline_ms, now_ms, b_expo,
                  weights=None, L=None, cost=None, steps=None) -> dict:
    """steps = (step_off [N+1], step_deadline_ms [S], step_cost [S]) or None."""
    """One Algorithm 1 iteration of one model (see orloj_oracle_iterate_model)."""
    L = L or lib()
    cnt = np.ascontiguousarray(counts, dtype=np.uint32)
    B, C, K = cnt.shape
    bs = np.ascontiguousarray(batch_sizes, dtype=np.int32)
    cl = np.ascontiguousarray(cls, dtype=np.int32)
    dl = np.ascontiguousarray(deadline_ms, dtype=np.float64)
    wt = None if weights is None else np.ascontiguousarray(weights, dtype=np.float64)
    N = cl.size
    timed_out = np.zeros(max(N, 1), np.int32)
    score = np.zeros(max(N, 1))
    batch = np.full(max(int(bs[-1]), 1), -1, np.int32)
    cand = np.zeros(1, np.int32)
    bn = np.zeros(1, np.int32)
    co = _opt64(cost)
    if steps is not None:
        so = np.ascontiguousarray(steps[0], dtype=np.int64)
        sd = np.ascontiguousarray(steps[1], dtype=np.float64)
        sc = np.ascontiguousarray(steps[2], dtype=np.float64)
    rc = L.orloj_oracle_iterate_model(
        C, K, B, _p(bs, _I32P), float(bin_width_ms), _p(cnt, _U32P),
        _p(wt, _F64P) if wt is not None else None, N, _p(cl, _I32P), _p(dl, _F64P),
        _p(co, _F64P) if co is not None else None,
        _p(so, _I64P) if steps is not None else None,
        _p(sd, _F64P) if steps is not None else None,
        _p(sc, _F64P) if steps is not None else None,
        float(now_ms), float(b_expo), _p(timed_out, _I32P), _p(score, _F64P), _p(cand, _I32P),
        _p(batch, _I32P), _p(bn, _I32P))
    if rc:
        raise OracleError(f"orloj_oracle_iterate_model rc={rc}")
    return dict(timed_out=timed_out[:N], score=score[:N], cand_bs=int(cand[0]),
                batch=batch[:int(bn[0])].copy())


def iterate_workload(wl, weights=None, models: Optional[Sequence[int]] = None, L=None,
                     steps=None, threads: int = 1) -> dict:
    """Algorithm 1 for every model of a workload (or the listed ones);
    per-request outputs concatenated in model order.  steps = (step_off over
    the whole queue array, step_deadline_ms, step_cost) or None.
    ``threads`` > 1 runs the models on that many host threads."""
    models = list(range(wl.n_models)) if models is None else list(models)

    def one(q):
        m = wl.model(q)
        st = None
        if steps is not None:
            a, b = int(wl.queue_off[q]), int(wl.queue_off[q + 1])
            off = np.asarray(steps[0], np.int64)
            lo, hi = int(off[a]), int(off[b])
            st = (off[a:b + 1] - lo, np.asarray(steps[1])[lo:hi], np.asarray(steps[2])[lo:hi])
        return iterate_model(m["counts"], wl.batch_sizes, m["bin_width_ms"], m["cls"],
                             m["deadline_ms"], m["now_ms"], wl.b_expo,
                             None if weights is None else weights[q], L, cost=m["cost"],
                             steps=st)

    parts = _map_models(one, models, threads)
    cat = lambda k: (np.concatenate([p[k] for p in parts]) if parts else np.zeros(0))
    return dict(timed_out=cat("timed_out").astype(np.int32), score=cat("score"),
                cand_bs=np.array([p["cand_bs"] for p in parts], np.int32),
                batch=[p["batch"] for p in parts], per_model=parts)


def accumulate(counts, bin_width_ms, model, bs_index, cls, latency_ms, L=None) -> int:
    """Add the samples to counts ([M][B][C][K] uint32, in place); returns the
    number of rejected samples (see orloj_oracle_accumulate)."""
    L = L or lib()
    if not (isinstance(counts, np.ndarray) and counts.dtype == np.uint32 and
            counts.flags.c_contiguous):
        raise TypeError("counts must be a C-contiguous uint32 array")
    M, B, C, K = counts.shape
    w = np.ascontiguousarray(bin_width_ms, dtype=np.float64)
    mo = np.ascontiguousarray(model, dtype=np.int32)
    bi = np.ascontiguousarray(bs_index, dtype=np.int32)
    cl = np.ascontiguousarray(cls, dtype=np.int32)
    la = np.ascontiguousarray(latency_ms, dtype=np.float64)
    rej = np.zeros(1, np.int64)
    rc = L.orloj_oracle_accumulate(M, B, C, K, _p(w, _F64P), la.size, _p(mo, _I32P), _p(bi, _I32P),
                                   _p(cl, _I32P), _p(la, _F64P), _p(counts, _U32P), _p(rej, _I64P))
    if rc:
        raise OracleError(f"orloj_oracle_accumulate rc={rc}")
    return int(rej[0])


def score_model_affine(counts_ck, batch_sizes, bin_width_ms, c0_ms, c1, cls, deadline_ms, now_ms,
                       b_expo, prefix_mode: int = 0, want_priority: bool = False, L=None,
                       cost=None) -> dict:
    """All candidates of one model in the affine batch-latency mode (see
    orloj_oracle_score_model_affine); counts_ck is [C][K]."""
    L = L or lib()
    cnt = np.ascontiguousarray(counts_ck, dtype=np.uint32)
    C, K = cnt.shape
    bs = np.ascontiguousarray(batch_sizes, dtype=np.int32)
    cl = np.ascontiguousarray(cls, dtype=np.int32)
    dl = np.ascontiguousarray(deadline_ms, dtype=np.float64)
    caps = ncap(bs, cl.size, prefix_mode)
    n_cand = int(caps.sum())
    n_prob = int((caps * (caps + 1) // 2).sum())
    P = np.empty(n_prob)
    pr = np.empty(n_prob) if want_priority else None
    E = np.empty(n_cand)
    EL = np.empty(n_cand)
    S = np.empty(n_cand)
    sn = np.zeros(1, np.int32)
    sb = np.zeros(1, np.int32)
    ss = np.zeros(1)
    co = _opt64(cost)
    rc = L.orloj_oracle_score_model_affine(
        C, K, bs.size, _p(bs, _I32P), float(bin_width_ms), _p(cnt, _U32P), float(c0_ms), float(c1),
        cl.size, _p(cl, _I32P), _p(dl, _F64P), _p(co, _F64P) if co is not None else None,
        float(now_ms), float(b_expo), int(prefix_mode), _p(P, _F64P),
        _p(pr, _F64P) if pr is not None else None, _p(E, _F64P), _p(EL, _F64P), _p(S, _F64P),
        _p(sn, _I32P), _p(sb, _I32P), _p(ss, _F64P))
    if rc:
        raise OracleError(f"orloj_oracle_score_model_affine rc={rc}")
    out = dict(finish_prob=P, expected_finish=E, expected_latency_ms=EL, score=S,
               sel_n=int(sn[0]), sel_bs=int(sb[0]), sel_score=float(ss[0]))
    if pr is not None:
        out["priority"] = pr
    return out


def score_workload_affine(wl, c0_ms, c1, prefix_mode: int = 0, models=None, L=None,
                          threads: int = 1) -> dict:
    """Affine mode over a workload whose counts are [M][C][K] (batch-size
    independent); outputs concatenated in model order.  ``threads`` > 1
    scores the models on that many host threads."""
    models = list(range(wl.n_models)) if models is None else list(models)

    def one(q):
        m = wl.model(q)
        return score_model_affine(m["counts"], wl.batch_sizes, m["bin_width_ms"], c0_ms[q],
                                  c1[q], m["cls"], m["deadline_ms"], m["now_ms"], wl.b_expo,
                                  prefix_mode, L=L, cost=m["cost"])

    parts = _map_models(one, models, threads)
    cat = lambda k: (np.concatenate([p[k] for p in parts]) if parts else np.zeros(0))
    out = {k: cat(k) for k in ("finish_prob", "expected_finish", "expected_latency_ms", "score")}
    out["sel_n"] = np.array([p["sel_n"] for p in parts], np.int32)
    out["sel_bs"] = np.array([p["sel_bs"] for p in parts], np.int32)
    out["sel_score"] = np.array([p["sel_score"] for p in parts])
    out["per_model"] = parts
    return out
