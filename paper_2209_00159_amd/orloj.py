"""Python binding of liborloj.so (include/orloj.h).

Argument marshalling only: every step of the scoring path runs in the HIP
kernels behind the C ABI.  PyTorch supplies device memory and the stream.
There is no fallback: if the library is not built, or no GPU is visible,
calls raise.
"""
from __future__ import annotations

import ctypes
import os
import sys
from typing import Optional

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liborloj.so")

ORLOJ_OK, ORLOJ_E_INVALID, ORLOJ_E_DATA, ORLOJ_E_HIP, ORLOJ_E_NOMEM, ORLOJ_E_UNSUPPORTED = range(6)
PREFIX_TRIANGLE, PREFIX_RECT = 0, 1
MAX_BINS, MAX_BATCH_SIZES, MAX_PREFIX = 8192, 256, 256

_STATUS = {0: "OK", 1: "E_INVALID", 2: "E_DATA", 3: "E_HIP", 4: "E_NOMEM", 5: "E_UNSUPPORTED"}


class OrlojError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"orloj {_STATUS.get(code, code)}: {msg}")
        self.code = code


class Grid(ctypes.Structure):
    _fields_ = [("n_models", ctypes.c_int32), ("n_classes", ctypes.c_int32),
                ("n_bins", ctypes.c_int32), ("n_bs", ctypes.c_int32),
                ("batch_sizes", ctypes.POINTER(ctypes.c_int32)),
                ("d_bin_width_ms", ctypes.c_void_p)]


class Queues(ctypes.Structure):
    _fields_ = [("h_queue_off", ctypes.POINTER(ctypes.c_int64)),
                ("d_queue_off", ctypes.c_void_p), ("d_class", ctypes.c_void_p),
                ("d_deadline_ms", ctypes.c_void_p), ("d_now_ms", ctypes.c_void_p),
                ("d_cost", ctypes.c_void_p)]


class Steps(ctypes.Structure):
    _fields_ = [("h_step_off", ctypes.POINTER(ctypes.c_int64)), ("d_step_off", ctypes.c_void_p),
                ("d_step_deadline_ms", ctypes.c_void_p), ("d_step_cost", ctypes.c_void_p)]


class Trace(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int64), ("h_release_ms", ctypes.c_void_p),
                ("h_model", ctypes.c_void_p), ("h_class", ctypes.c_void_p),
                ("h_deadline_ms", ctypes.c_void_p)]


class SimStats(ctypes.Structure):
    _fields_ = [(k, ctypes.c_int64) for k in ("ticks", "launches", "decisions", "dispatched",
                                             "dropped", "on_time", "late", "arrivals")] + \
               [(k, ctypes.c_double) for k in ("sim_ms", "wall_s", "device_s")]


class SimRecord(ctypes.Structure):
    _fields_ = [("every", ctypes.c_int32), ("limit", ctypes.c_int32), ("n", ctypes.c_int32),
                ("h_model", ctypes.c_void_p), ("h_now_ms", ctypes.c_void_p),
                ("h_sel_n", ctypes.c_void_p), ("h_sel_bs", ctypes.c_void_p),
                ("h_off", ctypes.c_void_p), ("h_class", ctypes.c_void_p),
                ("h_deadline_ms", ctypes.c_void_p)]


_LIB = None
_VP = ctypes.c_void_p
_GP = ctypes.POINTER(Grid)
_QP = ctypes.POINTER(Queues)
_SP = ctypes.POINTER(Steps)
_I64P = ctypes.POINTER(ctypes.c_int64)

EXPORTS = ("orloj_create", "orloj_destroy", "orloj_set_stream", "orloj_set_score_chunk",
           "orloj_last_error", "orloj_sync",
           "orloj_build_cdfs", "orloj_output_sizes", "orloj_score_candidates",
           "orloj_score_candidates_affine", "orloj_score_candidates_affine_noalloc",
           "orloj_select_batch", "orloj_build_model_laws",
           "orloj_iterate", "orloj_accumulate", "orloj_sched_create", "orloj_sched_destroy",
           "orloj_sched_admit", "orloj_sched_decide", "orloj_sched_queue_length",
           "orloj_simulate_trace")


def load(path: Optional[str] = None):
    """Load and bind liborloj.so (no GPU needed to load)."""
    global _LIB
    default = path is None or path == LIB_PATH
    path = LIB_PATH if path is None else path
    if _LIB is not None and default:
        return _LIB
    if not os.path.exists(path):
        raise OrlojError(ORLOJ_E_INVALID,
                         f"{path} is not built; run __graft_entry__.build() first")
    L = ctypes.CDLL(path)
    L.orloj_create.argtypes = [ctypes.POINTER(_VP), ctypes.c_int32, _VP]
    L.orloj_create.restype = ctypes.c_int
    L.orloj_destroy.argtypes = [_VP]
    L.orloj_destroy.restype = None
    L.orloj_set_stream.argtypes = [_VP, _VP]
    L.orloj_set_stream.restype = ctypes.c_int
    L.orloj_set_score_chunk.argtypes = [_VP, ctypes.c_int32]
    L.orloj_set_score_chunk.restype = ctypes.c_int
    L.orloj_last_error.argtypes = [_VP]
    L.orloj_last_error.restype = ctypes.c_char_p
    L.orloj_sync.argtypes = [_VP]
    L.orloj_sync.restype = ctypes.c_int
    L.orloj_build_cdfs.argtypes = [_VP, ctypes.c_int64, ctypes.c_int32, _VP, _VP, _VP]
    L.orloj_build_cdfs.restype = ctypes.c_int
    L.orloj_output_sizes.argtypes = [_GP, _QP, ctypes.c_int32, _I64P, _I64P, _I64P, _I64P]
    L.orloj_output_sizes.restype = ctypes.c_int
    L.orloj_score_candidates.argtypes = [_VP, _GP, _VP, _VP, _QP, ctypes.c_double, ctypes.c_int32,
                                         _VP, _VP, _VP, _VP, _VP, _VP]
    L.orloj_score_candidates.restype = ctypes.c_int
    L.orloj_score_candidates_affine.argtypes = [_VP, _GP, _VP, _VP, _VP, _VP, _QP, ctypes.c_double,
                                                ctypes.c_int32, _VP, _VP, _VP, _VP, _VP, _VP]
    L.orloj_score_candidates_affine.restype = ctypes.c_int
    L.orloj_score_candidates_affine_noalloc.argtypes = L.orloj_score_candidates_affine.argtypes
    L.orloj_score_candidates_affine_noalloc.restype = ctypes.c_int
    L.orloj_select_batch.argtypes = [_VP, _GP, _QP, ctypes.c_int32, _VP, _VP, _VP, _VP, _VP]
    L.orloj_select_batch.restype = ctypes.c_int
    L.orloj_build_model_laws.argtypes = [_VP, _GP, _VP, _VP, ctypes.c_double, _VP, _VP, _VP]
    L.orloj_build_model_laws.restype = ctypes.c_int
    L.orloj_iterate.argtypes = [_VP, _GP, _VP, _VP, _VP, _VP, _QP, _SP, ctypes.c_double, _VP,
                                _VP, _VP, _VP]
    L.orloj_iterate.restype = ctypes.c_int
    L.orloj_accumulate.argtypes = [_VP, _GP, ctypes.c_int64, _VP, _VP, _VP, _VP, _VP, _VP]
    L.orloj_accumulate.restype = ctypes.c_int
    L.orloj_sched_create.argtypes = [ctypes.POINTER(_VP), _VP, _GP, _VP, _VP, _VP, ctypes.c_double]
    L.orloj_sched_create.restype = ctypes.c_int
    L.orloj_sched_destroy.argtypes = [_VP]
    L.orloj_sched_destroy.restype = None
    L.orloj_sched_admit.argtypes = [_VP, ctypes.c_int64, _VP, _VP, _VP]
    L.orloj_sched_admit.restype = ctypes.c_int
    L.orloj_sched_decide.argtypes = [_VP, ctypes.c_double, _VP, _VP, _VP, _VP, _VP, _VP, _VP]
    L.orloj_sched_decide.restype = ctypes.c_int
    L.orloj_sched_queue_length.argtypes = [_VP, ctypes.c_int32]
    L.orloj_sched_queue_length.restype = ctypes.c_int64
    L.orloj_simulate_trace.argtypes = [_VP, ctypes.POINTER(Trace), ctypes.c_double, _VP, _VP, _VP,
                                       ctypes.c_uint64, ctypes.c_int64, ctypes.POINTER(SimRecord),
                                       ctypes.POINTER(SimStats)]
    L.orloj_simulate_trace.restype = ctypes.c_int
    if default:
        _LIB = L
    return L


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _need_cuda(t: torch.Tensor, name: str, dtypes, device):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.device != device:
        raise ValueError(f"{name} must live on {device}, not {t.device}")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


class Context:
    """An orloj_ctx bound to one device and (by default) torch's current
    stream on it."""

    def __init__(self, device=None, stream: Optional[torch.cuda.Stream] = None):
        if not torch.cuda.is_available():
            raise OrlojError(ORLOJ_E_INVALID, "no GPU visible")
        self.L = load()
        self.device = torch.device("cuda", torch.cuda.current_device() if device is None
                                   else torch.device(device).index or 0)
        st = stream if stream is not None else torch.cuda.current_stream(self.device)
        self.ctx = ctypes.c_void_p()
        rc = self.L.orloj_create(ctypes.byref(self.ctx), self.device.index,
                                 ctypes.c_void_p(st.cuda_stream))
        if rc:
            raise OrlojError(rc, "orloj_create failed")

    def __del__(self):
        finalizing = sys is None or sys.is_finalizing()
        if getattr(self, "ctx", None) and self.ctx.value and not finalizing:
            self.L.orloj_destroy(self.ctx)
            self.ctx = None

    def _check(self, rc: int):
        if rc:
            raise OrlojError(rc, self.L.orloj_last_error(self.ctx).decode())

    def set_stream(self, stream: torch.cuda.Stream):
        self._check(self.L.orloj_set_stream(self.ctx, ctypes.c_void_p(stream.cuda_stream)))

    def set_score_chunk(self, steps: int):
        """Prefix steps per score workgroup: -1 automatic, 0 never split."""
        self._check(self.L.orloj_set_score_chunk(self.ctx, int(steps)))

    def sync(self):
        self._check(self.L.orloj_sync(self.ctx))

    # -- orloj_build_cdfs ------------------------------------------------------
    def build_cdfs(self, counts: torch.Tensor, out: Optional[torch.Tensor] = None,
                   support: Optional[torch.Tensor] = None) -> torch.Tensor:
        """counts [..., K] (uint32 stored as int32 or uint32) -> 1 - CDF at
        each bin's right edge, float32.  If `support` (int32 [..., 2]) is
        given, each row's first and last bin holding mass are written to it."""
        _need_cuda(counts, "counts", (torch.int32, torch.uint32), self.device)
        K = counts.shape[-1]
        if out is None:
            out = torch.empty(counts.shape, dtype=torch.float32, device=self.device)
        _need_cuda(out, "out", (torch.float32,), self.device)
        if out.shape != counts.shape:
            raise ValueError("out must have the shape of counts")
        if support is not None:
            _need_cuda(support, "support", (torch.int32,), self.device)
            if support.shape != counts.shape[:-1] + (2,):
                raise ValueError("support must have shape counts.shape[:-1] + (2,)")
        rows = counts.numel() // K if K else 0
        self._check(self.L.orloj_build_cdfs(self.ctx, rows, K, _ptr(counts), _ptr(out),
                                            _ptr(support)))
        return out


def make_grid(n_models, n_classes, n_bins, batch_sizes: np.ndarray,
              d_bin_width_ms: Optional[torch.Tensor]):
    bs = np.ascontiguousarray(batch_sizes, dtype=np.int32)
    g = Grid(int(n_models), int(n_classes), int(n_bins), int(bs.size),
             bs.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), _ptr(d_bin_width_ms))
    g._keep = bs
    return g


def make_queues(h_queue_off: np.ndarray, d_queue_off, d_class, d_deadline_ms, d_now_ms,
                d_cost=None):
    ho = np.ascontiguousarray(h_queue_off, dtype=np.int64)
    qs = Queues(ho.ctypes.data_as(_I64P), _ptr(d_queue_off), _ptr(d_class), _ptr(d_deadline_ms),
                _ptr(d_now_ms), _ptr(d_cost))
    qs._keep = ho
    return qs


def output_sizes(grid: Grid, queues: Queues, prefix_mode: int = PREFIX_TRIANGLE):
    """(n_cands, n_probs, cand_off[M+1], prob_off[M+1]) computed by the
    library on the host."""
    L = load()
    M = grid.n_models
    nc = ctypes.c_int64()
    npb = ctypes.c_int64()
    co = np.zeros(M + 1, np.int64)
    po = np.zeros(M + 1, np.int64)
    rc = L.orloj_output_sizes(ctypes.byref(grid), ctypes.byref(queues), prefix_mode,
                              ctypes.byref(nc), ctypes.byref(npb), co.ctypes.data_as(_I64P),
                              po.ctypes.data_as(_I64P))
    if rc:
        raise OrlojError(rc, "orloj_output_sizes rejected its arguments")
    return nc.value, npb.value, co, po


class Scorer:
    """A workload resident in HBM plus its output buffers: uploads the
    histograms and queues once, then builds the CDF tables, scores all
    candidates and selects a batch per model through the C ABI.  An affine
    workload (``wl.affine``: counts [M][C][K] and per-model c0, c1) is
    scored with orloj_score_candidates_affine."""

    def __init__(self, wl, ctx: Optional[Context] = None, prefix_mode: int = PREFIX_TRIANGLE,
                 counts_device: Optional[torch.Tensor] = None, trim: bool = True):
        self.ctx = ctx or Context()
        self.wl = wl
        self.mode = prefix_mode
        self.trim = trim
        dev = self.ctx.device
        if counts_device is not None:
            self.counts = counts_device
        else:
            self.counts = torch.from_numpy(np.ascontiguousarray(wl.counts).view(np.int32)).to(dev)
        self.ccdf = torch.empty(self.counts.shape, dtype=torch.float32, device=dev)
        self.support = torch.empty(self.counts.shape[:-1] + (2,), dtype=torch.int32, device=dev)
        self.width = torch.from_numpy(np.ascontiguousarray(wl.bin_width_ms, np.float64)).to(dev)
        self.grid = make_grid(wl.n_models, wl.n_classes, wl.n_bins, wl.batch_sizes, self.width)
        self.affine = bool(getattr(wl, "affine", False))
        if self.affine:
            self.c0 = torch.from_numpy(np.ascontiguousarray(wl.c0_ms, np.float64)).to(dev)
            self.c1 = torch.from_numpy(np.ascontiguousarray(wl.c1, np.float64)).to(dev)
        self.set_queues(wl.queue_off, wl.cls, wl.deadline_ms, wl.now_ms)
        M = wl.n_models
        self.sel_n = torch.zeros(M, dtype=torch.int32, device=dev)
        self.sel_bs = torch.zeros(M, dtype=torch.int32, device=dev)
        self.sel_score = torch.zeros(M, dtype=torch.float32, device=dev)

    def set_queues(self, queue_off, cls, deadline_ms, now_ms, cost=None):
        dev = self.ctx.device
        self.h_queue_off = np.ascontiguousarray(queue_off, np.int64)
        self.d_queue_off = torch.from_numpy(self.h_queue_off).to(dev)
        self.d_class = torch.from_numpy(np.ascontiguousarray(cls, np.int32)).to(dev)
        self.d_deadline = torch.from_numpy(np.ascontiguousarray(deadline_ms, np.float64)).to(dev)
        self.d_now = torch.from_numpy(np.ascontiguousarray(now_ms, np.float64)).to(dev)
        c = getattr(self.wl, "cost", None) if cost is None else cost
        self.d_cost = None if c is None else torch.from_numpy(np.ascontiguousarray(c, np.float64)).to(dev)
        self.queues = make_queues(self.h_queue_off, self.d_queue_off, self.d_class,
                                  self.d_deadline, self.d_now, self.d_cost)
        self.n_cands, self.n_probs, self.h_cand_off, self.h_prob_off = output_sizes(
            self.grid, self.queues, self.mode)
        self.d_cand_off = torch.from_numpy(self.h_cand_off).to(dev)
        self.d_prob_off = torch.from_numpy(self.h_prob_off).to(dev)
        self.finish_prob = torch.empty(max(self.n_probs, 1), dtype=torch.float32, device=dev)
        self.expected_finish = torch.empty(max(self.n_cands, 1), dtype=torch.float64, device=dev)
        self.expected_latency = torch.empty(max(self.n_cands, 1), dtype=torch.float32, device=dev)
        self.score_out = torch.empty(max(self.n_cands, 1), dtype=torch.float32, device=dev)

    # -- the three entry points --------------------------------------------------
    def build(self):
        self.ctx.build_cdfs(self.counts, self.ccdf, self.support)

    def score(self, b_expo: Optional[float] = None, noalloc: bool = False):
        """Enqueue the scoring call; ``noalloc`` (affine workloads only) calls
        orloj_score_candidates_affine_noalloc, which allocates nothing."""
        b = self.wl.b_expo if b_expo is None else b_expo
        c = self.ctx
        sup = _ptr(self.support) if self.trim else None
        outs = (_ptr(self.d_cand_off), _ptr(self.d_prob_off), _ptr(self.finish_prob),
                _ptr(self.expected_finish), _ptr(self.expected_latency), _ptr(self.score_out))
        if noalloc and not self.affine:
            raise ValueError("the allocation-free entry point scores affine workloads")
        if self.affine:
            fn = (c.L.orloj_score_candidates_affine_noalloc if noalloc
                  else c.L.orloj_score_candidates_affine)
            c._check(fn(
                c.ctx, ctypes.byref(self.grid), _ptr(self.ccdf), sup, _ptr(self.c0), _ptr(self.c1),
                ctypes.byref(self.queues), float(b), self.mode, *outs))
        else:
            c._check(c.L.orloj_score_candidates(
                c.ctx, ctypes.byref(self.grid), _ptr(self.ccdf), sup, ctypes.byref(self.queues),
                float(b), self.mode, *outs))

    def select(self):
        c = self.ctx
        c._check(c.L.orloj_select_batch(
            c.ctx, ctypes.byref(self.grid), ctypes.byref(self.queues), self.mode,
            _ptr(self.d_cand_off), _ptr(self.score_out), _ptr(self.sel_n), _ptr(self.sel_bs),
            _ptr(self.sel_score)))

    def run(self, build: bool = True, b_expo: Optional[float] = None) -> dict:
        if build:
            self.build()
        self.score(b_expo)
        self.select()
        self.ctx.sync()
        return self.fetch()

    def fetch(self) -> dict:
        torch.cuda.synchronize(self.ctx.device)
        return dict(
            finish_prob=self.finish_prob[:self.n_probs].cpu().numpy(),
            expected_finish=self.expected_finish[:self.n_cands].cpu().numpy(),
            expected_latency_ms=self.expected_latency[:self.n_cands].cpu().numpy(),
            score=self.score_out[:self.n_cands].cpu().numpy(),
            sel_n=self.sel_n.cpu().numpy(), sel_bs=self.sel_bs.cpu().numpy(),
            sel_score=self.sel_score.cpu().numpy())


class Iterator:
    """The scheduler iteration (Algorithm 1 with the paper's own priority)
    over a workload resident in HBM: builds the CDF tables, their support and
    the model-wide batch laws once, then runs orloj_iterate on the queues."""

    def __init__(self, wl, ctx: Optional[Context] = None, class_weights=None,
                 counts_device: Optional[torch.Tensor] = None):
        self.ctx = ctx or Context()
        self.wl = wl
        dev = self.ctx.device
        self.counts = counts_device if counts_device is not None else \
            torch.from_numpy(np.ascontiguousarray(wl.counts).view(np.int32)).to(dev)
        shape = self.counts.shape
        self.ccdf = torch.empty(shape, dtype=torch.float32, device=dev)
        self.support = torch.empty(shape[:-1] + (2,), dtype=torch.int32, device=dev)
        self.law = torch.empty(shape, dtype=torch.float32, device=dev)
        self.disc = torch.empty(shape, dtype=torch.float32, device=dev)
        self.model_el = torch.empty(shape[:2], dtype=torch.float32, device=dev)
        self.weights = None if class_weights is None else \
            torch.from_numpy(np.ascontiguousarray(class_weights, np.float64)).to(dev)
        self.width = torch.from_numpy(np.ascontiguousarray(wl.bin_width_ms, np.float64)).to(dev)
        self.grid = make_grid(wl.n_models, wl.n_classes, wl.n_bins, wl.batch_sizes, self.width)
        self.bs_max = int(wl.batch_sizes[-1])
        self.cand_bs = torch.zeros(wl.n_models, dtype=torch.int32, device=dev)
        self.batch = torch.full((wl.n_models, self.bs_max), -1, dtype=torch.int32, device=dev)
        self.set_queues(wl.queue_off, wl.cls, wl.deadline_ms, wl.now_ms)

    def set_queues(self, queue_off, cls, deadline_ms, now_ms, cost=None, steps=None):
        """steps = (step_off [N+1] over the whole queue array, step_deadline_ms,
        step_cost) for piecewise-step cost functions, or None."""
        dev = self.ctx.device
        self.h_queue_off = np.ascontiguousarray(queue_off, np.int64)
        self.d_queue_off = torch.from_numpy(self.h_queue_off).to(dev)
        self.d_class = torch.from_numpy(np.ascontiguousarray(cls, np.int32)).to(dev)
        self.d_deadline = torch.from_numpy(np.ascontiguousarray(deadline_ms, np.float64)).to(dev)
        self.d_now = torch.from_numpy(np.ascontiguousarray(now_ms, np.float64)).to(dev)
        c = getattr(self.wl, "cost", None) if cost is None else cost
        self.d_cost = None if c is None else torch.from_numpy(np.ascontiguousarray(c, np.float64)).to(dev)
        self.queues = make_queues(self.h_queue_off, self.d_queue_off, self.d_class,
                                  self.d_deadline, self.d_now, self.d_cost)
        self.steps = None
        if steps is not None:
            self.h_step_off = np.ascontiguousarray(steps[0], np.int64)
            self.d_step_off = torch.from_numpy(self.h_step_off).to(dev)
            self.d_step_dl = torch.from_numpy(np.ascontiguousarray(steps[1], np.float64)).to(dev)
            self.d_step_cost = torch.from_numpy(np.ascontiguousarray(steps[2], np.float64)).to(dev)
            self.steps = Steps(self.h_step_off.ctypes.data_as(_I64P), _ptr(self.d_step_off),
                               _ptr(self.d_step_dl), _ptr(self.d_step_cost))
        n = int(self.h_queue_off[-1])
        self.timed_out = torch.zeros(max(n, 1), dtype=torch.int32, device=dev)
        self.score = torch.zeros(max(n, 1), dtype=torch.float32, device=dev)

    def build(self, b_expo: Optional[float] = None):
        b = self.wl.b_expo if b_expo is None else b_expo
        self.b = float(b)
        self.ctx.build_cdfs(self.counts, self.ccdf, self.support)
        c = self.ctx
        c._check(c.L.orloj_build_model_laws(
            c.ctx, ctypes.byref(self.grid), _ptr(self.ccdf), _ptr(self.weights), self.b,
            _ptr(self.law), _ptr(self.disc), _ptr(self.model_el)))

    def iterate(self):
        c = self.ctx
        c._check(c.L.orloj_iterate(
            c.ctx, ctypes.byref(self.grid), _ptr(self.support), _ptr(self.law), _ptr(self.disc),
            _ptr(self.model_el), ctypes.byref(self.queues),
            ctypes.byref(self.steps) if self.steps is not None else None, self.b,
            _ptr(self.timed_out),
            _ptr(self.score), _ptr(self.cand_bs), _ptr(self.batch)))

    def run(self, build: bool = True, b_expo: Optional[float] = None) -> dict:
        if build:
            self.build(b_expo)
        self.iterate()
        self.ctx.sync()
        return self.fetch()

    def fetch(self) -> dict:
        torch.cuda.synchronize(self.ctx.device)
        n = int(self.h_queue_off[-1])
        return dict(timed_out=self.timed_out[:n].cpu().numpy(), score=self.score[:n].cpu().numpy(),
                    cand_bs=self.cand_bs.cpu().numpy(), batch=self.batch.cpu().numpy(),
                    model_el=self.model_el.cpu().numpy())


def accumulate(ctx: Context, grid: Grid, counts: torch.Tensor, model, bs_index, cls,
               latency_ms) -> int:
    """Profiler feedback: add the samples (device tensors: int32 model,
    batch-size index, class; float64 latency) to counts (int32/uint32
    [M][B][C][K] on the device).  Returns the number of rejected samples
    (this synchronises)."""
    _need_cuda(counts, "counts", (torch.int32, torch.uint32), ctx.device)
    for t, name, dt in ((model, "model", torch.int32), (bs_index, "bs_index", torch.int32),
                        (cls, "cls", torch.int32), (latency_ms, "latency_ms", torch.float64)):
        _need_cuda(t, name, (dt,), ctx.device)
    n = int(latency_ms.numel())
    if not (model.numel() == bs_index.numel() == cls.numel() == n):
        raise ValueError("sample arrays differ in length")
    rej = torch.zeros(1, dtype=torch.int64, device=ctx.device)
    ctx._check(ctx.L.orloj_accumulate(ctx.ctx, ctypes.byref(grid), n, _ptr(model), _ptr(bs_index),
                                      _ptr(cls), _ptr(latency_ms), _ptr(counts), _ptr(rej)))
    ctx.sync()
    return int(rej.item())


def _host(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _vp(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


class Sched:
    """The host scheduling runtime (orloj_sched_*): per-model deadline queues,
    the drop phase and one score + select round per decide() call.  The
    tables (ccdf, support) and the grid's bin-width tensor must outlive it."""

    def __init__(self, ctx: Context, grid: Grid, ccdf: torch.Tensor,
                 support: Optional[torch.Tensor], drop_ms: np.ndarray, b_expo: float):
        self.ctx = ctx
        self.grid = grid
        self._keep = (ccdf, support, grid)
        self.M = grid.n_models
        self.smax = int(grid.batch_sizes[grid.n_bs - 1])
        d = _host(drop_ms, np.float64)
        if d.shape != (grid.n_models, grid.n_classes):
            raise ValueError("drop_ms must be [n_models, n_classes]")
        self.s = ctypes.c_void_p()
        ctx._check(ctx.L.orloj_sched_create(ctypes.byref(self.s), ctx.ctx, ctypes.byref(grid),
                                            _ptr(ccdf), _ptr(support), _vp(d), float(b_expo)))

    def __del__(self):
        finalizing = sys is None or sys.is_finalizing()
        if getattr(self, "s", None) and self.s.value and not finalizing:
            self.ctx.L.orloj_sched_destroy(self.s)
            self.s = None

    def admit(self, model, cls, deadline_ms):
        m, c, d = _host(model, np.int32), _host(cls, np.int32), _host(deadline_ms, np.float64)
        if not (m.size == c.size == d.size):
            raise ValueError("admit: arrays differ in length")
        self.ctx._check(self.ctx.L.orloj_sched_admit(self.s, m.size, _vp(m), _vp(c), _vp(d)))

    def queue_length(self, model: int) -> int:
        return int(self.ctx.L.orloj_sched_queue_length(self.s, int(model)))

    def decide(self, now_ms: float, idle=None) -> dict:
        M = self.M
        idle_a = None if idle is None else _host(idle, np.uint8)
        sn = np.zeros(M, np.int32)
        sb = np.zeros(M, np.int32)
        dropped = np.zeros(1, np.int64)
        boff = np.zeros(M + 1, np.int64)
        bcls = np.zeros(M * self.smax, np.int32)
        bdl = np.zeros(M * self.smax, np.float64)
        self.ctx._check(self.ctx.L.orloj_sched_decide(
            self.s, float(now_ms), None if idle_a is None else _vp(idle_a), _vp(sn), _vp(sb),
            _vp(dropped), _vp(boff), _vp(bcls), _vp(bdl)))
        n = int(boff[-1])
        return dict(sel_n=sn, sel_bs=sb, dropped=int(dropped[0]), batch_off=boff,
                    batch_class=bcls[:n], batch_deadline_ms=bdl[:n])

    def simulate(self, trace, tick_ms: float, solo_counts: np.ndarray, bin_width_ms, bs_scale,
                 seed: int = 0, max_ticks: int = 0, record_every: int = 0, record_limit: int = 0):
        """orloj_simulate_trace over trace = (release_ms, model, class,
        deadline_ms).  Returns (stats dict, recorded states as a list of
        (model, now_ms, class[], deadline_ms[], sel_n, sel_bs))."""
        rel, mod, cls, dl = (_host(trace[0], np.float64), _host(trace[1], np.int32),
                             _host(trace[2], np.int32), _host(trace[3], np.float64))
        tr = Trace(rel.size, _vp(rel), _vp(mod), _vp(cls), _vp(dl))
        counts = _host(solo_counts, np.uint32)
        if counts.shape != (self.M, self.grid.n_classes, self.grid.n_bins):
            raise ValueError("solo_counts must be [n_models, n_classes, n_bins]")
        w = _host(bin_width_ms, np.float64)
        sc = _host(bs_scale, np.float64)
        if w.size != self.M or sc.size != self.grid.n_bs:
            raise ValueError("bin_width_ms must be [n_models] and bs_scale [n_bs]")
        L = max(int(record_limit), 0) if record_every > 0 else 0
        bufs = dict(model=np.zeros(max(L, 1), np.int32), now=np.zeros(max(L, 1)),
                    sn=np.zeros(max(L, 1), np.int32), sb=np.zeros(max(L, 1), np.int32),
                    off=np.zeros(L + 1, np.int64),
                    cls=np.zeros(max(L, 1) * self.smax, np.int32),
                    dl=np.zeros(max(L, 1) * self.smax))
        rec = SimRecord(int(record_every), L, 0, _vp(bufs["model"]), _vp(bufs["now"]),
                        _vp(bufs["sn"]), _vp(bufs["sb"]), _vp(bufs["off"]), _vp(bufs["cls"]),
                        _vp(bufs["dl"]))
        st = SimStats()
        self.ctx._check(self.ctx.L.orloj_simulate_trace(
            self.s, ctypes.byref(tr), float(tick_ms), _vp(counts), _vp(w), _vp(sc), int(seed),
            int(max_ticks), ctypes.byref(rec) if L > 0 else None, ctypes.byref(st)))
        stats = {k: getattr(st, k) for k, _ in SimStats._fields_}
        states = []
        o = bufs["off"]
        for r in range(rec.n if L > 0 else 0):
            a, b = int(o[r]), int(o[r + 1])
            states.append((int(bufs["model"][r]), float(bufs["now"][r]), bufs["cls"][a:b].copy(),
                           bufs["dl"][a:b].copy(), int(bufs["sn"][r]), int(bufs["sb"][r])))
        return stats, states
