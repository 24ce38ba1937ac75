"""Benchmark: candidate-batch x histogram-bin evaluations per second.

One step = one scheduling pass of the hot path over every model of the
workload: orloj_score_candidates (scan over queue position of the members'
CDF rows into the batch CDF, E[L_B], finish probabilities, priorities) and
orloj_select_batch (one batch per model).  The CDF tables are built once
before timing (orloj_build_cdfs refreshes profiles off the scheduling path)
and timed on their own.  Inputs are resident in HBM when the timed
region starts.

Default workload: configuration 5 in its saturated decision state (128
models x 64 batch sizes x 32 classes x 4096 bins, every model holding a
backlog deep enough for all 64-member prefixes).

Prints ONE JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("candidate-batch × histogram-bin evaluations/sec; "
          "scheduling decisions/sec")
HBM_PEAK_GBS = 8000.0
# fp64 vector peak: 256 CUs x 64 fp64 FMA lanes per clock x 2 flops x 2.4 GHz
FP64_VECTOR_PEAK_TFLOPS = 256 * 64 * 2 * 2.4e9 / 1e12


def algorithmic_bytes(wl, mode=0):
    """Bytes one score launch must move at least: each distinct CDF row
    a (model, batch size) workgroup reads, each queued request read once
    (class + deadline), the per-model scalars, and every output."""
    K = wl.n_bins
    rows = 0
    reqs = 0
    n_c = 0
    n_p = 0
    for q in range(wl.n_models):
        a, b = int(wl.queue_off[q]), int(wl.queue_off[q + 1])
        N = b - a
        cls = wl.cls[a:b]
        maxcap = 0
        for s in wl.batch_sizes:
            cap = N if mode else min(int(s), N)
            maxcap = max(maxcap, cap)
            rows += len(np.unique(cls[:cap]))
            n_c += cap
            n_p += cap * (cap + 1) // 2
        reqs += maxcap
    table = rows * K * 4
    queue = reqs * 12 + wl.n_models * (8 + 8 + 8 * 4)
    outputs = n_p * 4 + n_c * 16
    return dict(total=table + queue + outputs, table=table, queue=queue, outputs=outputs,
                distinct_rows=rows, n_cands=n_c, n_probs=n_p)


def support_table_bytes(wl, mode=0):
    """Table bytes of the same distinct rows counting only each row's
    support (first to last bin holding mass): the entries outside it are
    known to be exactly 1 or 0 once the table is built."""
    nz = wl.counts > 0
    K = wl.n_bins
    lo = np.argmax(nz, axis=-1)
    hi = K - 1 - np.argmax(nz[..., ::-1], axis=-1)
    width = hi - lo + 1
    total = 0
    for q in range(wl.n_models):
        a, b = int(wl.queue_off[q]), int(wl.queue_off[q + 1])
        N = b - a
        cls = wl.cls[a:b]
        for bi, s in enumerate(wl.batch_sizes):
            cap = N if mode else min(int(s), N)
            total += int(width[q, bi, np.unique(cls[:cap])].sum())
    return total * 4


TRAFFIC_SUMMARY = {
    "tabulated": os.path.join(ROOT, "profiles", "score_kernel_cfg5_traffic.txt"),
    "affine": os.path.join(ROOT, "profiles", "score_kernel_affine_cfg5_traffic.txt"),
}
KERNEL_SOURCE = os.path.join(ROOT, "paper_2209_00159_amd", "csrc", "orloj.hip")


def measured_traffic(mode="tabulated"):
    """HBM bytes per score launch from the committed rocprofv3 counter
    summary of that mode, or None when it is missing or was taken on
    another version of the kernel source."""
    from paper_2209_00159_amd import profsum
    path = TRAFFIC_SUMMARY[mode]
    if not os.path.exists(path):
        return None
    d = profsum.read_summary(path)
    if d.get("source_sha256") != profsum.source_sha(KERNEL_SOURCE):
        return None
    return float(d["traffic_bytes_per_launch"])


def affine_algorithmic(aw, mode=0):
    """Work one affine-mode score pass must do at least.  Under Eq. (3)
    every batch size of a model shares the members' product on the solo
    grid, so:
      bytes: each distinct solo-latency row among a model's longest prefix,
             read once per model; each queued request read once; the
             per-model scalars (now, width, c0, c1, offsets); every output;
      flops: per (model, prefix length n, bin) the product update (one fma)
             and the E[X] sum (one add), shared by every batch size; per
             candidate the discounted-prefix step (one fma per bin) over the
             bins its members' priorities read: up to bin k - 2 of its
             latest deadline on that batch size's grid, the whole grid when
             a member's deadline lies beyond it, none when all are dead."""
    K = aw.n_bins
    rows = reqs = n_c = n_p = 0
    product_flops = prefix_flops = 0
    for q in range(aw.n_models):
        a, b = int(aw.queue_off[q]), int(aw.queue_off[q + 1])
        N = b - a
        caps = [N if mode else min(int(s), N) for s in aw.batch_sizes]
        longest = max(caps, default=0)
        cls = aw.cls[a:b]
        rows += len(np.unique(cls[:longest]))
        reqs += longest
        product_flops += 3 * K * longest
        tau = aw.deadline_ms[a:a + longest] - aw.now_ms[q] - aw.c0_ms[q]
        for s, cap in zip(aw.batch_sizes, caps):
            n_c += cap
            n_p += cap * (cap + 1) // 2
            if cap == 0:
                continue
            u = tau[:cap] / (aw.c1[q] * int(s) * aw.bin_width_ms[q])
            kz = np.where(tau[:cap] <= 0.0, -1, np.where(u >= K, K - 2, np.floor(u) - 2))
            need = np.maximum.accumulate(kz) + 1          # bins 0 .. max kz of prefix n
            prefix_flops += 2 * int(np.clip(need, 0, None).sum())
    table = rows * K * 4
    queue = reqs * 12 + aw.n_models * (8 * 4 + 8 + 8 * 4)
    outputs = n_p * 4 + n_c * 16
    return dict(bytes=table + queue + outputs, table=table, queue=queue, outputs=outputs,
                flops=product_flops + prefix_flops, product_flops=product_flops,
                prefix_flops=prefix_flops)


def valid_candidates(wl):
    return sum(min(int(s), wl.queue_len(q)) for q in range(wl.n_models) for s in wl.batch_sizes)


def _oracle_leg(wl, affine, budget_s, threads):
    """One timed leg of the oracle on the workload's models: `threads` host
    threads at a time (the C oracle releases the GIL; threads = 1 runs in
    the calling thread), each taking the next model until about budget_s
    seconds have passed.  Returns (models, evals, seconds)."""
    import threading
    from concurrent.futures import ThreadPoolExecutor

    import oracle

    lock = threading.Lock()
    state = dict(next=0, done=0, evals=0)
    t0 = time.perf_counter()

    def worker():
        while True:
            with lock:
                if state["next"] >= wl.n_models or time.perf_counter() - t0 > budget_s:
                    return
                q = state["next"]
                state["next"] += 1
            sub = wl.subset([q])
            if affine:
                oracle.score_workload_affine(sub, sub.c0_ms, sub.c1)
            else:
                oracle.score_workload(sub)
            ev = sum(min(int(s), wl.queue_len(q)) for s in wl.batch_sizes) * wl.n_bins
            with lock:
                state["done"] += 1
                state["evals"] += ev

    if threads == 1:
        worker()
    else:
        with ThreadPoolExecutor(threads) as ex:
            for f in [ex.submit(worker) for _ in range(threads)]:
                f.result()
    return state["done"], state["evals"], time.perf_counter() - t0


def host_cores():
    """The host CPUs this process may run on (the GPU's CPU share)."""
    return len(os.sched_getaffinity(0))


def cpu_baseline(config_id, max_models, budget_s=10.0, affine=False, legs=3):
    """The oracle, as it stands, on the models of the same state, timed in
    `legs` legs of each kind, the median leg reported:
      - on every host core this process may use (one model per thread at a
        time); value = its evals/s, cores = that count;
      - on one core: the calling thread pinned to one CPU with
        os.sched_setaffinity for the leg, then restored.
    The whole run takes about 2 x budget_s seconds."""
    from paper_2209_00159_amd import workloads as W

    cores = host_cores()
    n_cfg = W.CONFIG_MODELS.get(config_id)
    wl = W.make(config_id, models=list(range(min(max_models, n_cfg))) if n_cfg else None,
                workers=cores)
    if affine:
        wl = W.affine(wl)
    per_leg = budget_s / legs

    def median_leg(runs):
        runs = sorted(runs, key=lambda r: r[1] / r[2])
        return runs[len(runs) // 2], [round(r[1] / r[2], 1) for r in runs]

    many, many_rates = median_leg([_oracle_leg(wl, affine, per_leg, cores) for _ in range(legs)])
    mask = os.sched_getaffinity(0)
    pin = min(mask)
    os.sched_setaffinity(0, {pin})
    try:
        one, one_rates = median_leg([_oracle_leg(wl, affine, per_leg, 1) for _ in range(legs)])
    finally:
        os.sched_setaffinity(0, mask)
    dn, en, tn = many
    d1, e1, t1 = one
    whole = dn == wl.n_models
    return dict(value=en / tn, unit="evals/s", cores=cores, kind="oracle",
                sample=(f"{wl.name}: {'all ' if whole else 'the first '}{dn} model(s) of the same "
                        f"state, full triangles, fp64 C oracle, median of {legs} legs on "
                        f"{cores} host threads (every core this process may use, one model per "
                        f"thread at a time), {tn:.2f} s for the median leg"),
                nproc=os.cpu_count(), legs=legs, seconds=round(tn, 2), decisions_per_s=dn / tn,
                leg_rates=many_rates,
                single_core=dict(value=e1 / t1, unit="evals/s", cores=1, pinned_cpu=pin,
                                 models=d1, seconds=round(t1, 2), decisions_per_s=d1 / t1,
                                 leg_rates=one_rates))


def oracle_on_states(wl, recorded, budget_s=10.0, threads=None):
    """The oracle on decision states recorded by the scheduling loop, on
    `threads` host threads, for about budget_s seconds: decisions/s, and how
    many of its selections equal the GPU's."""
    import threading
    from concurrent.futures import ThreadPoolExecutor

    import oracle

    threads = host_cores() if threads is None else threads
    lock = threading.Lock()
    state = dict(next=0, done=0, same=0)
    t0 = time.perf_counter()

    def worker():
        while True:
            with lock:
                if state["next"] >= len(recorded) or time.perf_counter() - t0 > budget_s:
                    return
                dec = recorded[state["next"]]
                state["next"] += 1
            sub = wl.subset([dec.model]).with_queues([(dec.cls, dec.deadline_ms)], [dec.now_ms])
            o = oracle.score_workload(sub)
            same = int((int(o["sel_n"][0]), int(o["sel_bs"][0])) == (dec.sel_n, dec.sel_bs))
            with lock:
                state["done"] += 1
                state["same"] += same

    with ThreadPoolExecutor(threads) as ex:
        for f in [ex.submit(worker) for _ in range(threads)]:
            f.result()
    dt = time.perf_counter() - t0
    return dict(decisions_per_s=state["done"] / dt, states=state["done"],
                same_selection=state["same"], seconds=round(dt, 2), cores=threads)


def tabulated_roofline(wl, ab, kms):
    achieved = ab["total"] / (kms * 1e-3) / 1e9
    traffic = measured_traffic("tabulated")
    sup_bytes = ab["total"] - ab["table"] + support_table_bytes(wl)
    roof = dict(bound="hbm", achieved=round(achieved, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                frac=round(achieved / HBM_PEAK_GBS, 4),
                traffic=None if traffic is None else round(traffic),
                traffic_unit="bytes/launch",
                kernel="score_kernel", kernel_ms=round(kms, 5),
                algorithmic_bytes=ab["total"],
                support_only_bytes=sup_bytes,
                support_only_frac=round(sup_bytes / (kms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4))
    if traffic is not None:
        roof["traffic_gbs"] = round(traffic / (kms * 1e-3) / 1e9, 1)
    return roof


def affine_roofline(aw, kms):
    """Roofline of one affine scoring call (emax_kernel + score_kernel):
    the bound is whichever of the algorithmic bytes at the HBM peak and the
    algorithmic flops at the fp64 vector peak takes longer."""
    w = affine_algorithmic(aw)
    t = kms * 1e-3
    gbs = w["bytes"] / t / 1e9
    tflops = w["flops"] / t / 1e12
    traffic = measured_traffic("affine")
    hbm_bound = w["bytes"] / (HBM_PEAK_GBS * 1e9) >= w["flops"] / (FP64_VECTOR_PEAK_TFLOPS * 1e12)
    if hbm_bound:
        head = dict(bound="hbm", achieved=round(gbs, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                    frac=round(gbs / HBM_PEAK_GBS, 4))
    else:
        head = dict(bound="alu", achieved=round(tflops, 2), peak=round(FP64_VECTOR_PEAK_TFLOPS, 1),
                    unit="TFLOP/s", frac=round(tflops / FP64_VECTOR_PEAK_TFLOPS, 4))
    return dict(head, traffic=None if traffic is None else round(traffic),
                traffic_unit="bytes/launch", kernel="emax_kernel + score_kernel (affine)",
                kernel_ms=round(kms, 5), algorithmic_bytes=w["bytes"],
                algorithmic_flops=w["flops"],
                alu_achieved_tflops=round(tflops, 3),
                alu_frac=round(tflops / FP64_VECTOR_PEAK_TFLOPS, 4))


def bench_affine(wl, ctx, args, torch, O, W):
    """Time orloj_score_candidates_affine (+ select) on the same queues with
    one solo-latency table per class and the batch law c0 + c1 s l."""
    aw = W.affine(wl)
    sc = O.Scorer(aw, ctx, trim=not args.no_trim)
    sc.build()
    ctx.sync()
    for _ in range(args.warmup):
        sc.score()
        sc.select()
    ctx.sync()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for e0, e1 in evs:
        e0.record()
        sc.score()
        e1.record()
        sc.select()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ctx.sync()
    times = [e0.elapsed_time(e1) for e0, e1 in evs]
    kms = float(np.mean(times))
    ms = wall * 1e3 / args.steps
    evals = valid_candidates(aw) * aw.n_bins
    print(f"[bench] affine: {ms:.4f} ms/step, score kernel {kms:.4f} ms", file=sys.stderr,
          flush=True)
    del sc
    return dict(
        what="orloj_score_candidates_affine + orloj_select_batch: batch latency c0 + c1 s l "
             "(one solo-latency table per class), same queues, grid and batch sizes",
        workload=aw.name, c1=float(aw.c1[0]), ms_per_step=round(ms, 5),
        evals_per_s=evals / (ms * 1e-3),
        saturated_pass_selections_per_s=aw.n_models / (ms * 1e-3),
        table_bytes=int(aw.counts.size * 4),
        roofline=dict(affine_roofline(aw, kms), kernel_ms_median=round(float(np.median(times)), 5)))


def copy_reference(torch, dev, nbytes=1 << 30, reps=10):
    """Measured HBM rate of a plain device copy (torch's copy kernel, 1 GiB
    read + 1 GiB written per launch), HIP events on the current stream: the
    attainable stream rate beside the 8 TB/s peak."""
    src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del src, dst
    return (round(2 * nbytes / (ms * 1e-3) / 1e9, 1),
            f"device copy of {nbytes >> 20} MiB (read + write), mean of {reps} launches")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    # The first launches of a fresh process run slow and the time per launch
    # settles over about 50 of them (score kernel at configuration 5: 0.37 ms
    # for the first, 0.33 by the tenth, 0.32 from about the fortieth), so the
    # untimed warm-up is long enough for that by default.
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--config", type=int, default=5)
    ap.add_argument("--cpu-models", type=int, default=128,
                    help="most models the CPU oracle sample may take (each leg stops after ~10 s)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--workers", type=int, default=None,
                    help="host threads for the workload generator (default: every host core)")
    ap.add_argument("--trace-arrivals", type=int, default=1_000_000,
                    help="arrivals of the configuration-5 trace replayed by the native "
                         "scheduling loop after the timed steps (0 = skip)")
    ap.add_argument("--no-iterate", action="store_true",
                    help="skip timing the Algorithm 1 iteration (orloj_iterate) on the same state")
    ap.add_argument("--no-trim", action="store_true",
                    help="score without the table support (every table entry is read)")
    ap.add_argument("--no-affine", action="store_true",
                    help="skip timing the affine batch-latency mode on the same state")
    ap.add_argument("--mode", choices=("tabulated", "affine"), default="tabulated",
                    help="batch-latency law of the timed step: per-batch-size tables "
                         "(default) or the affine law c0 + c1 s l (then the affine, iteration "
                         "and scheduling-loop legs are skipped)")
    ap.add_argument("--no-copy-ref", action="store_true",
                    help="skip timing the plain device copy reported as roofline.copy_gbs")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="after timing, copy a 1 GiB buffer once (a plain copy kernel of "
                         "known size, for scaling HBM traffic counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU: the scorer has no multi-GPU path "
              f"(--gpus {args.gpus} requested)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2209_00159_amd import orloj as O
    from paper_2209_00159_amd import workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)

    t0 = time.perf_counter()
    workers = args.workers or len(os.sched_getaffinity(0))
    wl = W.make(args.config, workers=workers)
    print(f"[bench] generated {wl.name} in {time.perf_counter() - t0:.1f} s", file=sys.stderr,
          flush=True)
    affine = args.mode == "affine"
    if affine:
        wl = W.affine(wl)
        args.no_affine = args.no_iterate = True
        args.trace_arrivals = 0
    ctx = O.Context(0)
    sc = O.Scorer(wl, ctx, trim=not args.no_trim)
    ab = None if affine else algorithmic_bytes(wl)
    K = wl.n_bins
    evals = valid_candidates(wl) * K

    # profile refresh (off the scheduling path): timed on its own
    sc.build()
    ctx.sync()
    b0, b1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    b0.record()
    sc.build()
    b1.record()
    ctx.sync()
    build_ms = b0.elapsed_time(b1)

    for _ in range(args.warmup):
        sc.score()
        sc.select()
    ctx.sync()
    print(f"[bench] warmup done", file=sys.stderr, flush=True)

    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for e0, e1 in evs:
        e0.record()
        sc.score()
        e1.record()
        sc.select()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ctx.sync()
    score_times = [e0.elapsed_time(e1) for e0, e1 in evs]
    score_ms = float(np.mean(score_times))
    ms_per_step = wall * 1e3 / args.steps
    print(f"[bench] timed {args.steps} steps: {ms_per_step:.4f} ms/step, score kernel "
          f"{score_ms:.4f} ms", file=sys.stderr, flush=True)

    if affine:
        roof = affine_roofline(wl, score_ms)
    else:
        roof = tabulated_roofline(wl, ab, score_ms)
    roof["kernel_ms_median"] = round(float(np.median(score_times)), 5)
    line = dict(
        metric=METRIC, value=evals / (ms_per_step * 1e-3), unit="evals/s", n_gpus=1,
        steps=args.steps, warmup=args.warmup, ms_per_step=round(ms_per_step, 5),
        higher_is_better=True, scaling="weak", vs_baseline=None, dtype="f64+f32",
        data="synthetic",
        config=dict(workload=wl.name, models=wl.n_models, classes=wl.n_classes, bins=K,
                    batch_sizes=f"{int(wl.batch_sizes[0])}..{int(wl.batch_sizes[-1])}",
                    candidates=valid_candidates(wl), evals_per_step=evals,
                    prefix_mode="triangle", b_expo_per_ms=wl.b_expo,
                    batch_law="affine c0 + c1 s l" if affine else "per-batch-size tables"),
        decisions_per_s=None,
        saturated_pass_selections_per_s=wl.n_models / (ms_per_step * 1e-3),
        saturated_pass_note=("one selection per model per timed step (every model scored at "
                             "once, all 64-deep prefixes present); configuration 5's scheduling "
                             "decisions/s, with the queue re-scored at every dispatch decision, "
                             "is decisions_per_s from the trace-driven loop"),
        build_cdfs_ms=round(build_ms, 4),
        build_cdfs_gbs=round(wl.counts.nbytes * 2 / (build_ms * 1e-3) / 1e9, 1),
        roofline=roof,
    )
    if args.calibrate_copy:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        line["calibration_copy_bytes"] = src.numel() * 4
        del src, dst
    if not args.no_copy_ref:
        roof["copy_gbs"], roof["copy_note"] = copy_reference(torch, dev)
    if not args.no_affine:
        line["affine"] = bench_affine(wl, ctx, args, torch, O, W)
    if not args.no_iterate:
        it = O.Iterator(wl, ctx, counts_device=sc.counts)
        torch.cuda.synchronize()
        l0, l1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        it.build()
        ctx.sync()
        l0.record()
        it.build()
        l1.record()
        ctx.sync()
        laws_ms = l0.elapsed_time(l1)
        for _ in range(args.warmup):
            it.iterate()
        ctx.sync()
        iev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
        for e0, e1 in iev:
            e0.record()
            it.iterate()
            e1.record()
        ctx.sync()
        it_ms = float(np.mean([e0.elapsed_time(e1) for e0, e1 in iev]))
        res = it.fetch()
        n_batches = int((res["cand_bs"] > 0).sum())
        line["iterate"] = dict(
            what="orloj_iterate: one Algorithm 1 iteration (drop phase, candidate batch size, "
                 "priority of every kept request, PopBatch) for every model, one launch "
                 "(two for long queues on few models)",
            ms_per_iteration=round(it_ms, 5), models_with_batch=n_batches,
            decisions_per_s=round(n_batches / (it_ms * 1e-3), 1),
            requests=int(wl.queue_off[-1]),
            build_tables_ms=round(laws_ms, 4),
            build_tables_note="orloj_build_cdfs + orloj_build_model_laws, off the scheduling path")
        print(f"[bench] iterate: {it_ms:.4f} ms per iteration, tables {laws_ms:.2f} ms",
              file=sys.stderr, flush=True)
        del it
    recorded = []
    if args.trace_arrivals and args.config == 5:
        from paper_2209_00159_amd import schedsim
        print(f"[bench] scheduling loop over {args.trace_arrivals} arrivals", file=sys.stderr,
              flush=True)
        loop = schedsim.NativeTraceLoop(wl, schedsim.config5_trace(args.trace_arrivals), ctx=ctx,
                                        record_every=45, record_limit=2000,
                                        tables=(sc.ccdf, sc.support if not args.no_trim else None))
        st = loop.run()
        recorded = st.recorded
        d = st.as_dict()
        line["trace"] = dict(
            arrivals=args.trace_arrivals, simulated_ms=round(d["sim_ms"], 1), ticks=d["ticks"],
            launches=d["launches"], decisions=d["decisions"], dispatched=d["dispatched"],
            dropped=d["dropped"], finish_rate=round(d["finish_rate"], 4),
            decisions_per_s=round(d["decisions_per_s"], 1),
            decisions_per_device_s=round(d["decisions_per_device_s"], 1),
            loop="native runtime (orloj_simulate_trace)",
            note="decisions_per_s: wall clock of the whole loop (queues, drop phase, "
                 "simulated workers and the rounds); decisions_per_device_s: queue upload + "
                 "score + select + selection download of the rounds only")
        line["decisions_per_s"] = line["trace"]["decisions_per_s"]
        print(f"[bench] loop: {d['decisions']} decisions in {d['wall_s']:.2f} s wall "
              f"({d['device_s']:.2f} s on device)", file=sys.stderr, flush=True)
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(args.config, args.cpu_models, affine=affine)
        if recorded:
            line["cpu_baseline"]["trace"] = oracle_on_states(wl, recorded, budget_s=10.0)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
