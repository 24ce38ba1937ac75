"""Summaries of rocprofv3 CSV output for the scorer's kernels.

    python -m paper_2209_00159_amd.profsum stats  <run_kernel_stats.csv>
    python -m paper_2209_00159_amd.profsum trace  <run_kernel_trace.csv>
    python -m paper_2209_00159_amd.profsum pmc    <run_counter_collection.csv> [...]
    python -m paper_2209_00159_amd.profsum traffic --fetch <csv> --write <csv> \
            --kernel score_kernel --copy-bytes N --source <file> --out <summary.txt>

`traffic` turns FETCH_SIZE and WRITE_SIZE (KiB per dispatch) into HBM bytes
per launch of one kernel (or per call, summed over the comma-separated
kernels one call launches, e.g. --kernel emax_kernel,score_kernel), each
scaled by what the same counter reads for a
plain device copy of known size run in the same process (bench.py
--calibrate-copy copies N bytes once): scale = N / (counter KiB x 1024).  It
writes a `key: value` text summary that bench.py reads back while the
kernel's code is unchanged (the summary records a SHA-256 of the source
with comments and whitespace removed).
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import re
import statistics
import sys
from collections import defaultdict


def _short(name: str) -> str:
    name = name.replace("(anonymous namespace)::", "")
    return name if len(name) <= 80 else name[:77] + "..."


def _rows(path):
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def stats_table(path) -> str:
    rows = _rows(path)
    out = ["| kernel | calls | total ns | average ns | min ns | max ns | % |", "|---|---|---|---|---|---|---|"]
    for r in rows:
        out.append(f"| `{_short(r['Name'])}` | {r['Calls']} | {r['TotalDurationNs']} | "
                   f"{float(r['AverageNs']):.0f} | {r['MinNs']} | {r['MaxNs']} | "
                   f"{float(r['Percentage']):.2f} |")
    return "\n".join(out)


def trace_table(path) -> str:
    by = defaultdict(list)
    for r in _rows(path):
        by[r["Kernel_Name"]].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    out = ["| kernel | calls | mean us | median us | min us | max us |", "|---|---|---|---|---|---|"]
    for k, v in sorted(by.items(), key=lambda kv: -sum(kv[1])):
        out.append(f"| `{_short(k)}` | {len(v)} | {statistics.mean(v):.2f} | "
                   f"{statistics.median(v):.2f} | {min(v):.2f} | {max(v):.2f} |")
    return "\n".join(out)


def pmc_means(paths):
    """{kernel: {counter: [values per dispatch]}} (values summed over the
    counter's instances within one dispatch)."""
    per = defaultdict(float)
    names = {}
    for p in paths:
        for r in _rows(p):
            key = (p, r["Dispatch_Id"], r["Counter_Name"])
            per[key] += float(r["Counter_Value"])
            names[(p, r["Dispatch_Id"])] = r["Kernel_Name"]
    agg = defaultdict(lambda: defaultdict(list))
    for (p, d, c), v in per.items():
        agg[names[(p, d)]][c].append(v)
    return agg


def pmc_table(paths) -> str:
    agg = pmc_means(paths)
    out = ["| kernel | counter | dispatches | mean | min | max |", "|---|---|---|---|---|---|"]
    for k, d in agg.items():
        for c, v in sorted(d.items()):
            out.append(f"| `{_short(k)}` | {c} | {len(v)} | {statistics.mean(v):.6g} | "
                       f"{min(v):.6g} | {max(v):.6g} |")
    return "\n".join(out)


def _kernel_and_copy(path, counter, kernel):
    """Mean per-dispatch value of `counter`, summed over the comma-separated
    kernels (one call that launches several), and the copy's value."""
    agg = pmc_means([path])
    total = 0.0
    for name in kernel.split(","):
        ks = [v for k, d in agg.items() if name in k for c, v in d.items() if c == counter]
        if not ks:
            raise SystemExit(f"no {name} dispatch with {counter} in {path}")
        total += statistics.mean(ks[0])
    copies = [max(d[counter]) for k, d in agg.items() if "copy" in k.lower() and counter in d]
    if not copies:
        raise SystemExit(f"no copy kernel with {counter} in {path} (run with --calibrate-copy)")
    return total, max(copies)


def source_sha(path) -> str:
    """SHA-256 of the source with comments and whitespace removed, so that
    editing documentation does not invalidate a counter summary while any
    change to the code does."""
    with open(path) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    text = re.sub(r"\s+", "", text)
    return hashlib.sha256(text.encode()).hexdigest()


def traffic(fetch_csv, write_csv, kernel, copy_bytes, source, out):
    f_kib, f_copy = _kernel_and_copy(fetch_csv, "FETCH_SIZE", kernel)
    w_kib, w_copy = _kernel_and_copy(write_csv, "WRITE_SIZE", kernel)
    f_scale = copy_bytes / (f_copy * 1024.0)
    w_scale = copy_bytes / (w_copy * 1024.0)
    fetch_b = f_kib * 1024.0 * f_scale
    write_b = w_kib * 1024.0 * w_scale
    lines = [
        f"kernel: {kernel}",
        f"source: {source}",
        f"source_sha256: {source_sha(source)}",
        f"fetch_kib_per_dispatch: {f_kib:.1f}",
        f"write_kib_per_dispatch: {w_kib:.1f}",
        f"copy_bytes: {copy_bytes}",
        f"copy_fetch_kib: {f_copy:.1f}",
        f"copy_write_kib: {w_copy:.1f}",
        f"fetch_scale: {f_scale:.4f}",
        f"write_scale: {w_scale:.4f}",
        f"fetch_bytes_per_launch: {fetch_b:.0f}",
        f"write_bytes_per_launch: {write_b:.0f}",
        f"traffic_bytes_per_launch: {fetch_b + write_b:.0f}",
    ]
    text = "\n".join(lines) + "\n"
    if out:
        with open(out, "a") as f:
            f.write(text)
    return text


def read_summary(path) -> dict:
    d = {}
    with open(path) as f:
        for ln in f:
            if ":" in ln and not ln.lstrip().startswith(("#", "|", "`")):
                k, v = ln.split(":", 1)
                d[k.strip()] = v.strip()
    return d


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    sub.add_parser("stats").add_argument("csv")
    sub.add_parser("trace").add_argument("csv")
    p = sub.add_parser("pmc")
    p.add_argument("csv", nargs="+")
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--kernel", default="score_kernel",
                   help="kernel name, or comma-separated names summed per call")
    t.add_argument("--copy-bytes", type=int, default=1 << 30)
    t.add_argument("--source", required=True)
    t.add_argument("--out")
    a = ap.parse_args(argv)
    if a.cmd == "stats":
        print(stats_table(a.csv))
    elif a.cmd == "trace":
        print(trace_table(a.csv))
    elif a.cmd == "pmc":
        print(pmc_table(a.csv))
    else:
        print(traffic(a.fetch, a.write, a.kernel, a.copy_bytes, a.source, a.out), end="")


if __name__ == "__main__":
    sys.exit(main())
