"""Host-side checks of the measurement helpers (no GPU)."""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2209_00159_amd import profsum  # noqa: E402
from paper_2209_00159_amd import workloads as W  # noqa: E402


def test_source_hash_ignores_comments_only(tmp_path):
    a = tmp_path / "a.hip"
    a.write_text("int f(int x) {\n  // add one\n  return x + 1; /* done */\n}\n")
    b = tmp_path / "b.hip"
    b.write_text("int f(int x) {\n    return x + 1;\n}  // reworded\n")
    c = tmp_path / "c.hip"
    c.write_text("int f(int x) {\n  return x + 2;\n}\n")
    assert profsum.source_sha(a) == profsum.source_sha(b)
    assert profsum.source_sha(a) != profsum.source_sha(c)


def test_traffic_summary_is_ignored_for_other_code(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("int k;\n")
    summ = tmp_path / "t.txt"
    summ.write_text(f"# comment: not a key\nsource_sha256: {profsum.source_sha(src)}\n"
                    "traffic_bytes_per_launch: 1234\n")
    monkeypatch.setattr(bench, "TRAFFIC_SUMMARY", {"tabulated": str(summ),
                                                   "affine": str(tmp_path / "missing.txt")})
    monkeypatch.setattr(bench, "KERNEL_SOURCE", str(src))
    assert bench.measured_traffic("tabulated") == 1234.0
    assert bench.measured_traffic("affine") is None
    src.write_text("int k2;\n")
    assert bench.measured_traffic("tabulated") is None


def test_affine_flops_by_hand():
    wl = W.random_affine(4, n_models=2, queue_lens=[5, 3], batch_sizes=(1, 4), n_bins=16)
    # per model: 2 K per prefix length up to the longest prefix, 2 K per candidate
    want = 0
    for N in (5, 3):
        caps = [min(1, N), min(4, N)]
        want += 2 * 16 * max(caps) + 2 * 16 * sum(caps)
    assert bench.affine_algorithmic_flops(wl) == want


def test_algorithmic_bytes_by_hand():
    wl = W.random_case(3, n_models=2, queue_lens=[5, 3], batch_sizes=(1, 4), n_bins=16)
    ab = bench.algorithmic_bytes(wl)
    rows = cands = probs = 0
    for q in range(2):
        cls = wl.cls[wl.queue_off[q]:wl.queue_off[q + 1]]
        for s in (1, 4):
            cap = min(s, len(cls))
            rows += len(set(cls[:cap].tolist()))
            cands += cap
            probs += cap * (cap + 1) // 2
    assert ab["table"] == rows * 16 * 4
    assert ab["outputs"] == probs * 4 + cands * 16
    sup = bench.support_table_bytes(wl)
    assert 0 < sup <= ab["table"]
    # a row's support is never empty, so one bin per distinct row is the floor
    assert sup >= rows * 4
    assert np.all(wl.counts.sum(axis=-1) > 0)
