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


def test_affine_work_by_hand():
    # dead, in-grid and beyond-the-grid members (tau / bin width from -5 to 75)
    wl = W.random_affine(4, n_models=2, queue_lens=[5, 3], batch_sizes=(1, 4), n_bins=16,
                         tau_range=(-20.0, 60.0))
    K = 16
    flops = 0
    rows = reqs = cands = probs = 0
    for q, N in enumerate((5, 3)):
        a = int(wl.queue_off[q])
        caps = [min(1, N), min(4, N)]
        longest = max(caps)
        # product update and E[X] sum once per prefix length, all bins
        flops += 3 * K * longest
        rows += len(set(wl.cls[a:a + longest].tolist()))
        reqs += longest
        for s, cap in zip((1, 4), caps):
            cands += cap
            probs += cap * (cap + 1) // 2
            ws = wl.c1[q] * s * wl.bin_width_ms[q]
            for n in range(1, cap + 1):
                last = -1               # largest bin a member's priority reads
                for m in range(n):
                    tau = wl.deadline_ms[a + m] - wl.now_ms[q] - wl.c0_ms[q]
                    if tau <= 0:
                        continue
                    k = int(np.floor(tau / ws))
                    kz = K - 2 if tau / ws >= K else k - 2
                    last = max(last, kz)
                flops += 2 * (last + 1) if last >= 0 else 0
    w = bench.affine_algorithmic(wl)
    assert w["flops"] == flops
    assert w["table"] == rows * K * 4
    assert w["outputs"] == probs * 4 + cands * 16
    assert w["queue"] == reqs * 12 + 2 * (8 * 4 + 8 + 8 * 4)


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


def test_traffic_sums_the_kernels_of_one_call(tmp_path):
    # two dispatches of each kernel (counter values summed over instances
    # within a dispatch), and a 1 GiB copy that reads as 512 MiB / 1 GiB
    def csv_for(counter, copy_kib):
        rows = ['"Dispatch_Id","Kernel_Name","Counter_Name","Counter_Value"']
        vals = {"emax_kernel<16>": [100.0, 300.0], "score_kernel<16>": [1000.0, 3000.0]}
        d = 0
        for k, v in vals.items():
            for x in v:
                d += 1
                rows += [f'{d},"{k}","{counter}",{x / 2}', f'{d},"{k}","{counter}",{x / 2}']
        rows.append(f'{d + 1},"__amd_rocclr_copyBuffer","{counter}",{copy_kib}')
        p = tmp_path / f"{counter}.csv"
        p.write_text("\n".join(rows) + "\n")
        return str(p)
    src = tmp_path / "k.hip"
    src.write_text("int k;\n")
    fetch = csv_for("FETCH_SIZE", 512 * 1024)
    write = csv_for("WRITE_SIZE", 1024 * 1024)
    d = {}
    for line in profsum.traffic(fetch, write, "emax_kernel,score_kernel", 1 << 30, str(src),
                                None).splitlines():
        k, v = line.split(": ", 1)
        d[k] = v
    assert float(d["fetch_scale"]) == 2.0 and float(d["write_scale"]) == 1.0
    # means per dispatch: 200 + 2000 KiB, scaled by 2 (fetch) and 1 (write)
    assert float(d["fetch_bytes_per_launch"]) == 2200 * 1024 * 2.0
    assert float(d["traffic_bytes_per_launch"]) == 2200 * 1024 * 3.0


def test_committed_traffic_summaries_match_the_kernel_source():
    """The benchmark's roofline.traffic comes from the committed FETCH/WRITE
    summaries only while they were taken on the kernel source as it stands
    (its hash without comments and whitespace); a kernel change without a
    fresh profile would leave the benchmark line without traffic."""
    import bench
    for mode in ("tabulated", "affine"):
        t = bench.measured_traffic(mode)
        assert t is not None, f"profiles/ {mode} traffic summary is stale or missing"
        assert t > 0
