"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function include/orloj.h declares, sizes outputs exactly as the
oracle lays them out, and rejects bad arguments before any launch."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2209_00159_amd import orloj as O
from paper_2209_00159_amd import workloads as W

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "include", "orloj.h")


def declared_functions():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(orloj_[a-z_0-9]+)\s*\(", txt)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(O.LIB_PATH):
        from paper_2209_00159_amd import build
        build.build()
    return O.load()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert set(names) == set(O.EXPORTS), names
    for n in names:
        assert hasattr(lib, n), n


def _grid_queues(batch_sizes, qlens, n_bins=16, n_classes=3):
    offs = np.concatenate([[0], np.cumsum(qlens)]).astype(np.int64)
    g = O.make_grid(len(qlens), n_classes, n_bins, np.asarray(batch_sizes), None)
    g.d_bin_width_ms = ctypes.c_void_p(8)         # never dereferenced on the host
    qs = O.make_queues(offs, None, None, None, None)
    return g, qs, offs


@pytest.mark.parametrize("mode", [0, 1])
def test_output_sizes_match_oracle_layout(lib, mode):
    r = np.random.default_rng(5)
    for _ in range(20):
        bs = np.unique(r.integers(1, 40, size=r.integers(1, 8))).astype(np.int32)
        qlens = r.integers(0, 70, size=r.integers(1, 6))
        g, qs, offs = _grid_queues(bs, qlens)
        nc, npb, co, po = O.output_sizes(g, qs, mode)
        oc, op = oracle.output_sizes(offs, bs, mode)
        assert np.array_equal(co, oc) and np.array_equal(po, op)
        assert nc == oc[-1] and npb == op[-1]


def test_output_sizes_rejects_bad_arguments(lib):
    g, qs, _ = _grid_queues([1, 2, 2], [3])
    with pytest.raises(O.OrlojError):
        O.output_sizes(g, qs, 0)                     # batch sizes not increasing
    g, qs, _ = _grid_queues([1, 2], [3])
    with pytest.raises(O.OrlojError):
        O.output_sizes(g, qs, 2)                     # unknown prefix mode
    g, qs, _ = _grid_queues([1, 2], [3], n_bins=O.MAX_BINS + 1)
    with pytest.raises(O.OrlojError) as ei:
        O.output_sizes(g, qs, 0)
    assert ei.value.code == O.ORLOJ_E_UNSUPPORTED
    g, qs, _ = _grid_queues([0, 2], [3])
    with pytest.raises(O.OrlojError):
        O.output_sizes(g, qs, 0)                     # batch size < 1


def test_null_context_is_rejected_without_touching_the_gpu(lib):
    g, qs, _ = _grid_queues([1, 2], [3])
    rc = lib.orloj_score_candidates(None, ctypes.byref(g), None, None, ctypes.byref(qs), 1e-4, 0,
                                    None, None, None, None, None, None)
    assert rc == O.ORLOJ_E_INVALID
    rc = lib.orloj_select_batch(None, ctypes.byref(g), ctypes.byref(qs), 0, None, None, None,
                                None, None)
    assert rc == O.ORLOJ_E_INVALID
    rc = lib.orloj_score_candidates_affine(None, ctypes.byref(g), None, None, None, None,
                                           ctypes.byref(qs), 1e-4, 0, None, None, None, None,
                                           None, None)
    assert rc == O.ORLOJ_E_INVALID
    assert lib.orloj_build_cdfs(None, 1, 4, None, None, None) == O.ORLOJ_E_INVALID
    assert lib.orloj_sync(None) == O.ORLOJ_E_INVALID
    assert lib.orloj_set_score_chunk(None, 16) == O.ORLOJ_E_INVALID
    assert lib.orloj_last_error(None)
    lib.orloj_destroy(None)


def test_binding_fails_loudly_without_library(tmp_path):
    with pytest.raises(O.OrlojError):
        O.load(str(tmp_path / "missing.so"))


def test_workload_shapes():
    wl = W.make(1)
    assert wl.counts.shape == (1, 16, 4, 128) and wl.counts.dtype == np.uint32
    assert np.all(wl.counts.sum(axis=-1) == W.COUNT_TOTAL)
    assert np.all(np.diff(wl.deadline_ms) >= 0)
    wl = W.random_case(1, n_models=3, queue_lens=[0, 5, 2])
    assert wl.queue_len(0) == 0 and wl.queue_len(1) == 5


def test_affine_workloads():
    wl = W.make(2)
    aff = W.affine(wl)
    assert aff.affine and not wl.affine
    assert aff.counts.shape == (1, 32, 1024)
    assert np.array_equal(aff.counts[0], wl.counts[0, 0])
    # secant of 1 + 0.08 (s - 1) at the fastest class median
    assert np.isclose(aff.c1[0], 0.08)
    assert np.isclose(aff.c0_ms[0], 0.92 * np.min(wl.class_p50_ms[0]))
    a3 = W.affine(W.make(3))
    assert np.isclose(a3.c1[0], (128 ** 0.6 - 1) / 127)
    assert np.isclose(a3.c0_ms[0], (1 - a3.c1[0]) * np.min(a3.class_p50_ms[0]))
    assert np.array_equal(aff.deadline_ms, wl.deadline_ms)
    r = W.random_affine(3, n_models=4)
    base = W.random_case(3, n_models=4)
    assert np.array_equal(r.counts, base.counts[:, 0])
    assert np.all((r.c0_ms >= 0) & (r.c0_ms <= 3.0)) and np.all((r.c1 >= 0.05) & (r.c1 <= 1.0))
    sub = r.subset([2, 0])
    assert np.array_equal(sub.c0_ms, r.c0_ms[[2, 0]]) and np.array_equal(sub.c1, r.c1[[2, 0]])


def test_runtime_rejects_null_handles_without_touching_the_gpu(lib):
    g, qs, _ = _grid_queues([1, 4], [3, 2])
    out = ctypes.c_void_p(123)
    rc = lib.orloj_sched_create(ctypes.byref(out), None, ctypes.byref(g), None, None, None, 1e-4)
    assert rc == O.ORLOJ_E_INVALID and out.value is None
    assert lib.orloj_sched_create(None, None, ctypes.byref(g), None, None, None, 1e-4) == \
        O.ORLOJ_E_INVALID
    assert lib.orloj_sched_admit(None, 0, None, None, None) == O.ORLOJ_E_INVALID
    sel = (ctypes.c_int32 * 2)()
    assert lib.orloj_sched_decide(None, 0.0, None, sel, sel, None, None, None, None) == \
        O.ORLOJ_E_INVALID
    assert lib.orloj_sched_queue_length(None, 0) == -1
    lib.orloj_sched_destroy(None)
    st = O.SimStats()
    assert lib.orloj_simulate_trace(None, None, 0.5, None, None, None, 1, 0, None,
                                    ctypes.byref(st)) == O.ORLOJ_E_INVALID
