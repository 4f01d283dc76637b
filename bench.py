#!/usr/bin/env python
"""Benchmark of the per-iteration hot path on one MI355X.

A step is one boosting iteration (one tree) of the sampled-regression
workload: 10,000,000 rows x 50 uniform features with 20% missing values,
squared error, max_bin 256, depth 8, minimal variance sampling with f = 0.1
in front of the tree.  The quantized ELLPACK page, labels and margins are
resident in HBM before the timed region.  Each step runs gradients, MVS
sampling and compaction into one device page, the fixed-point conversion,
the level-wise tree (histograms with the sibling subtraction, split search,
partitions), the leaves and the margin update of all 10M rows.

Prints one JSON line: value = histogram row-feature updates performed per
second of step time (G/s); ms_per_step is seconds per tree x 1000 (the timed
trees carry no events); roofline is that of the histogram kernel
(algorithmic bytes / its HIP-event time: every histogram launch of as many
further timed trees fills two events with its own start and end);
cpu_baseline times the CPU oracle (its OpenMP build, on the threads the
process is given, and the first tree again in one thread) on the first trees
of the same workload on the host and reports the same unit.
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

HBM_PEAK_GBS = 8000.0
METRIC = "histogram row-feature updates/sec (G/s), sec/tree, achieved HBM GB/s on 1 MI355X"
# the dense histogram kernels, by the hist_kernel field of the tree stats
HIST_KERNELS = {1: "k_hist_dense", 2: "k_hist_rot"}
# sources of the histogram kernel: stored counter traffic is reported only
# while these are unchanged
HIST_SOURCES = ["hist.hip", "hist_impl.h", "common.h"]
# a plain device-to-device copy of this size after the timed region scales the
# HBM counters (FETCH_SIZE / WRITE_SIZE) to bytes
CALIB_BYTES = 1 << 30


def hist_source_hash():
    import hashlib
    h = hashlib.sha256()
    for name in HIST_SOURCES:
        with open(os.path.join(ROOT, "paper_2005_09148_amd", "csrc", name), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def traffic_file(workload_key, kernel):
    return os.path.join(ROOT, "profiles", f"{kernel}_traffic_{workload_key}.json")


def stored_traffic(workload_key, kernel):
    """HBM bytes per histogram launch from the stored counter runs, or None
    when there are none or the kernel's sources changed since."""
    path = traffic_file(workload_key, kernel)
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    if rec.get("source_sha256") != hist_source_hash():
        return None
    return rec["traffic_bytes_per_launch"]


def read_counters(path):
    """Per-dispatch counter values from one rocprofv3 --pmc run (csv output):
    {dispatch_id: (kernel_name, grid_size, value)}."""
    import csv
    import glob
    files = glob.glob(os.path.join(path, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {path}")
    out = {}
    for fn in files:
        with open(fn) as fh:
            for r in csv.DictReader(fh):
                key = (fn, r["Dispatch_Id"])
                prev = out.get(key, (r["Kernel_Name"], int(r["Grid_Size"]), 0.0))
                out[key] = (prev[0], prev[1], prev[2] + float(r["Counter_Value"]))
    return out


def pmc_summary(fetch_dir, write_dir, workload_key, commands, kernel):
    """Turns the FETCH_SIZE and WRITE_SIZE runs into HBM bytes per histogram
    launch, each counter scaled by what it reads for the calibration copy."""
    res = {}
    for name, path, calib_field in (("fetch", fetch_dir, "FETCH_SIZE"), ("write", write_dir, "WRITE_SIZE")):
        rows = read_counters(path)
        hist = [v for (k, g, v) in rows.values() if kernel + "<" in k]
        copies = [(g, v) for (k, g, v) in rows.values() if "copyBuffer" in k]
        if not hist or not copies:
            raise SystemExit(f"{calib_field}: no {kernel} or copy dispatches in {path}")
        grid, copy_kib = max(copies)
        factor = CALIB_BYTES / (copy_kib * 1024.0)
        res[name] = {"counter": calib_field, "dispatches": len(hist),
                     "kib_per_dispatch": sum(hist) / len(hist),
                     "calib_copy_kib": copy_kib, "calib_copy_grid": grid, "scale": factor}
    traffic = sum(r["kib_per_dispatch"] * 1024.0 * r["scale"] for r in res.values())
    rec = {"kernel": kernel, "workload": workload_key, "source_sha256": hist_source_hash(),
           "calib_copy_bytes": CALIB_BYTES, "commands": commands, "counters": res,
           "traffic_bytes_per_launch": round(traffic)}
    with open(traffic_file(workload_key, kernel), "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec, indent=1))


# the in-HBM workloads: name -> (config id, description)
INHBM = {
    "tiny": (1, "tiny dense {n:,} x 28, logistic, max_bin 256, depth 6, no sampling"),
    "higgs": (2, "Higgs-shaped dense {n:,} x 28, logistic, max_bin 256, depth 8, no sampling"),
    "regression": (3, "sampled regression {n:,} x 50, 20% missing, squared error, max_bin 256, depth 8, "
                      "MVS f={f}"),
    "sparse": (5, "wide sparse CSR {n:,} x 2000 (1% dense, Zipf features), logistic, max_bin 64, depth 10, "
                  "gamma 0.1, no sampling"),
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--rows", type=int, default=None, help="override the row count (testing)")
    ap.add_argument("--f", type=float, default=None, help="override the sampling fraction")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--hist-kernel", default="auto", choices=["auto", "plain", "rotated"],
                    help="dense histogram kernel (auto: the library's choice by pass size)")
    ap.add_argument("--cpu-trees", type=int, default=4)
    ap.add_argument("--sampler", default="mvs", choices=["mvs", "sgb", "goss"],
                    help="the sampler used when f < 1 (Sec. 2.3-2.4)")
    ap.add_argument("--compaction", choices=["auto", "stream", "gather"], default="auto",
                    help="outofcore: how the compaction reads the pinned pages (stream every page, or gather "
                         "only the kept rows through their device mapping)")
    ap.add_argument("--page-dir", default=None,
                    help="outofcore: keep the pages in (unlinked) files under this directory instead of "
                         "pinned host memory")
    ap.add_argument("--naive", action="store_true",
                    help="outofcore: Alg. 6, the naive construction (f = 1, every level streams every page)")
    ap.add_argument("--sketch-summary", type=int, default=65536,
                    help="outofcore: entries per feature of the merged quantile sketch (Alg. 3); 0 keeps the "
                         "whole strided sample on the device for the exact rule")
    ap.add_argument("--goss-a", type=float, default=0.05,
                    help="GOSS top fraction a (the rest fraction is f - a)")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarize two rocprofv3 --pmc runs of this script (no GPU work)")
    ap.add_argument("--pmc-commands", nargs="*", default=[], help="the commands of those runs")
    ap.add_argument("--pmc-kernel", default="k_hist_dense", choices=sorted(HIST_KERNELS.values()))
    ap.add_argument("--workload", default="regression", choices=sorted(INHBM) + ["outofcore"],
                    help="regression: 10M x 50 in HBM, MVS f = 0.1 (the default line); tiny: 10k x 28; "
                         "higgs: 1M x 28 Higgs-shaped; sparse: 2M x 2000 CSR; outofcore: 200M x 100 in "
                         "pinned host pages under an 8 GB device budget")
    return ap.parse_args()


def oracle_updates(b, res, depth):
    """Histogram updates the oracle performs for one tree: every evaluated node
    (depth < max_depth) sums every non-missing symbol of each of its rows."""
    from oracle import oracle as orc
    rows = res.sel
    nodes = res.nodes
    nonnull = (b.dense[rows] != orc.MISSING).sum(1).astype(np.int64)
    node = np.zeros(len(rows), np.int64)
    levels = np.zeros(len(rows), np.int64)
    active = np.ones(len(rows), bool)
    for d in range(depth):
        levels += active
        idx = np.nonzero(active)[0]
        nd = nodes[node[idx]]
        leaf = (nd["flags"] & orc.NODE_LEAF) != 0
        act_idx = idx[~leaf]
        feat = nd["feature"][~leaf]
        sb = nd["split_bin"][~leaf]
        dl = (nd["flags"][~leaf] & orc.NODE_DEFAULT_LEFT) != 0
        binv = b.dense[rows[act_idx], feat]
        miss = binv == orc.MISSING
        left = np.where(miss, dl, binv < sb)
        node[act_idx] = np.where(left, 2 * node[act_idx] + 1, 2 * node[act_idx] + 2)
        active[:] = False
        active[act_idx] = True
    return int((nonnull * levels).sum())


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(X, y, cfg, n_trees, gpu_trees, gpu_updates, sampler=(0, 0.0)):
    """Times the oracle on the first n_trees iterations of the same workload,
    in its OpenMP build on every thread OpenMP is given (OMP_NUM_THREADS, else
    the process's CPUs), and once more the first tree in one thread.
    Updates per tree: counted from the oracle's tree for dense data; for CSR
    data the GPU's count of the same (identical) tree."""
    from oracle import oracle as orc
    orc.select("omp")
    threads = orc.threads()
    print(f"[bench] cpu baseline: oracle cuts and bins ({threads} threads)", file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    if isinstance(X, dict):
        cuts = orc.sketch_cuts_csr(X["indptr"], X["indices"], X["values"], X["m"], cfg.max_bin)
        b = orc.bin_csr(X["indptr"], X["indices"], X["values"], X["m"], cuts)
    else:
        cuts = orc.sketch_cuts_dense(X, cfg.max_bin)
        b = orc.bin_dense(X, cuts)
    prep = time.perf_counter() - t0
    P = orc.Params(loss=cfg.loss, max_depth=cfg.max_depth, eta=cfg.eta, lambda_=cfg.lambda_,
                   gamma=cfg.gamma, min_child_weight=cfg.min_child_weight, f=cfg.f,
                   mvs_lambda=cfg.mvs_lambda, seed=cfg.seed, sampler=sampler[0], goss_a=sampler[1])
    if b.sparse:  # the update count comes from the GPU's identical trees
        n_trees = min(n_trees, len(gpu_updates))

    def run(trees):
        margin = np.full(len(y), cfg.base_margin, np.float32)
        secs, updates, out = 0.0, 0, []
        for t in range(trees):
            t1 = time.perf_counter()
            res = orc.train_tree(b, y, margin, P, iteration=t, want_detail=True)
            secs += time.perf_counter() - t1
            print(f"[bench] oracle tree {t} ({orc.threads()} threads): {time.perf_counter() - t1:.2f} s",
                  file=sys.stderr, flush=True)
            out.append(res.nodes.tobytes())
            updates += oracle_updates(b, res, cfg.max_depth) if not b.sparse else gpu_updates[t]
        return secs, updates, out

    secs, updates, trees = run(n_trees)
    same = all(t == g.tobytes() for t, g in zip(trees, gpu_trees)) if len(gpu_trees) else None
    orc.threads(1)
    secs1, updates1, trees1 = run(1)
    orc.threads(threads)
    return {
        "value": round(updates / secs / 1e9, 4),
        "unit": "G updates/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"first {n_trees} trees of the same {len(y):,}-row workload on {threads} OpenMP threads "
                  f"(oracle cuts and bins prepared untimed in {prep:.0f} s); {secs / n_trees:.3f} s/tree",
        "sec_per_tree": round(secs / n_trees, 4),
        "trees_identical_to_gpu": same,
        "omp_num_threads": os.environ.get("OMP_NUM_THREADS"),
        "affinity_cpus": len(os.sched_getaffinity(0)),
        "cpu_model": cpu_model(),
        "single_thread": {"value": round(updates1 / secs1 / 1e9, 4), "unit": "G updates/s", "cores": 1,
                          "sample": "first tree of the same workload in one OpenMP thread",
                          "sec_per_tree": round(secs1, 4),
                          "tree_identical_to_threaded": trees1[0] == trees[0]},
    }


def pinned_h2d_peak(torch, nbytes=1 << 30, reps=5):
    """Host-to-device GB/s of plain copies from pinned memory."""
    src = torch.empty(nbytes, dtype=torch.uint8).pin_memory()
    dst = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst.copy_(src, non_blocking=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        dst.copy_(src, non_blocking=True)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    del src, dst
    return nbytes * reps / dt / 1e9


def run_outofcore(args):
    """The 200M x 100 workload: twelve 2^24-row pages of binned rows in pinned
    host memory, an 8 GB cap on the library's device memory, MVS f = 0.1.
    Every tree streams the pages twice over the host link (compaction of the
    sampled rows, then the margin update of all rows)."""
    import torch

    from paper_2005_09148_amd import datagen, gbt

    cfg = datagen.CONFIGS[4]
    n = args.rows or datagen.FULL_ROWS[4]
    page_rows = datagen.C4_PAGE_ROWS
    sizes = datagen.config4_page_rows(n, page_rows)
    budget = 8 << 30
    ctx = gbt.Context(0, budget_bytes=budget)
    ctx.set_compaction({"auto": ctx.COMPACT_AUTO, "stream": ctx.COMPACT_STREAM,
                        "gather": ctx.COMPACT_GATHER}[args.compaction])
    sub = 1 << 21  # rows per host batch handed to the quantizer
    t = time.perf_counter()
    home = gbt.HOME_DISK if args.page_dir else gbt.HOME_PINNED_HOST
    # Alg. 3: each batch's sample is summarised and merged into running
    # summaries of sketch_summary entries per feature (0: the whole sample
    # is kept on the device for the exact rule)
    q = gbt.Quantizer(ctx, 100, n, max_bin=cfg.max_bin, page_rows=page_rows, page_home=home,
                      page_dir=args.page_dir, sketch_summary=args.sketch_summary)
    raw, labels = [], []
    for p, rows in enumerate(sizes):
        d = datagen.config4_page(p, rows=rows)
        for lo in range(0, rows, sub):
            q.sketch(d["X"][lo:lo + sub])
        raw.append(d["X"])
        labels.append(d["y"])
        print(f"[bench] page {p}: generated and sketched ({time.perf_counter() - t:.0f} s)", file=sys.stderr,
              flush=True)
    q.finalize()
    for p in range(len(sizes)):
        X = raw[p]
        for lo in range(0, len(X), sub):
            q.encode(X[lo:lo + sub])
        raw[p] = None
        print(f"[bench] page {p}: encoded ({time.perf_counter() - t:.0f} s)", file=sys.stderr, flush=True)
    mx = q.end()
    quant_secs = time.perf_counter() - t
    quant_peak = ctx.memory()[1]
    info = mx.info()
    y = np.concatenate(labels)
    del labels
    print(f"[bench] {info.n_pages} {'disk' if args.page_dir else 'pinned'} pages, row_words {info.row_words}, quantized in "
          f"{time.perf_counter() - t:.0f} s", file=sys.stderr, flush=True)
    label = torch.from_numpy(y).cuda()
    margin = torch.full((n,), cfg.base_margin, dtype=torch.float32, device="cuda")
    P = gbt.make_train_params(loss=cfg.loss, max_depth=cfg.max_depth, eta=cfg.eta, lambda_=cfg.lambda_,
                              gamma=cfg.gamma, min_child_weight=cfg.min_child_weight,
                              f=1.0 if args.naive else cfg.f, mvs_lambda=cfg.mvs_lambda, seed=cfg.seed)
    train = gbt.gbt_train_tree_naive if args.naive else gbt.gbt_train_tree
    ctx.set_timing(1)
    for w in range(args.warmup):
        P.iteration = w
        train(ctx, mx, label, margin, P)
        print(f"[bench] warm-up tree {w}", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    stats = []
    t0 = time.perf_counter()
    for k in range(args.steps):
        P.iteration = args.warmup + k
        stats.append(train(ctx, mx, label, margin, P).stats)
        print(f"[bench] tree {k}: {stats[-1].ms_total:.0f} ms", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ctx.set_timing(0)
    used, peak = ctx.memory()
    h2d = sum(s.h2d_bytes for s in stats)
    upd = sum(s.hist_updates for s in stats)
    hbytes = sum(s.hist_bytes for s in stats)
    hms = sum(s.ms_hist for s in stats)
    launches = sum(s.hist_launches for s in stats)
    achieved = hbytes / (hms * 1e-3) / 1e9 if hms > 0 else 0.0
    link_peak = pinned_h2d_peak(torch)
    kernels = {HIST_KERNELS.get(s.hist_kernel, "k_hist_sparse") for s in stats}
    line = {
        "metric": METRIC,
        "value": round(upd / dt / 1e9, 4),
        "unit": "G updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(dt * 1e3 / args.steps, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {"workload": f"out-of-core {n:,} x 100 in {info.n_pages} "
                               + ("disk" if args.page_dir else "pinned") + f" pages of {page_rows:,} rows, "
                               f"logistic, max_bin 256, depth 8, "
                               + ("Alg. 6 naive construction (f = 1, every level streams every page)"
                                  if args.naive else f"MVS f={cfg.f}") + ", 8 GB device budget",
                   "rows": n, "features": 100, "page_rows": page_rows, "f": 1.0 if args.naive else cfg.f,
                   "naive": bool(args.naive), "compaction": args.compaction,
                   "pages": "disk" if args.page_dir else "pinned host"},
        "sec_per_tree": round(dt / args.steps, 4),
        "rows_sampled_per_tree": round(sum(s.n_sampled for s in stats) / args.steps),
        "host_link": {"h2d_bytes_per_tree": round(h2d / args.steps), "achieved_gbs": round(h2d / dt / 1e9, 2),
                      "pinned_copy_peak_gbs": round(link_peak, 2),
                      "frac": round(h2d / dt / 1e9 / link_peak, 4)},
        "device_memory": {"budget_bytes": budget, "peak_bytes": peak, "quantize_peak_bytes": quant_peak},
        "quantize": {"secs": round(quant_secs, 1), "sketch": (f"merged summaries of {args.sketch_summary} "
                                                              "entries per feature, batches of 2^21 rows")
                     if args.sketch_summary else "exact rule on the whole strided sample"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": "+".join(sorted(kernels)), "launches": launches,
                     "avg_launch_us": round(hms * 1e3 / max(launches, 1), 2),
                     "algorithmic_bytes_per_launch": hbytes // max(launches, 1)},
        "cpu_baseline": None,
        "cpu_baseline_note": "not run at this size (the oracle needs minutes per tree on 200M rows); "
                             "tests/test_gpu_fullsize.py checks the same page shape against the oracle",
    }
    print(json.dumps(line), flush=True)


def workload_key(args):
    from paper_2005_09148_amd import datagen
    cfg_id = INHBM.get(args.workload, (3, ""))[0]
    n = args.rows or datagen.FULL_ROWS[cfg_id]
    f = args.f if args.f is not None else datagen.CONFIGS[cfg_id].f
    m = {1: 28, 2: 28, 3: 50, 5: 2000}[cfg_id]
    smp = "" if args.sampler == "mvs" or f >= 1 else f"_{args.sampler}"
    return f"{args.workload if args.workload in INHBM else 'regression'}_{n}x{m}_f{f:g}{smp}"


def main():
    args = parse()
    if args.pmc_summary:
        pmc_summary(*args.pmc_summary, workload_key(args), args.pmc_commands, args.pmc_kernel)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: the hot path here runs on a single MI355X "
              "(no multi-GPU path is built); run it with --gpus 1", file=sys.stderr)
        sys.exit(2)
    if args.workload == "outofcore":
        run_outofcore(args)
        return
    import torch

    from paper_2005_09148_amd import datagen, gbt

    cfg_id, desc = INHBM[args.workload]
    cfg = datagen.CONFIGS[cfg_id]
    if args.f is not None:
        cfg.f = args.f
    n = args.rows or datagen.FULL_ROWS[cfg_id]
    t = time.perf_counter()
    data = datagen.make(cfg_id, n)
    X = data["X"] if data["kind"] == "dense" else data
    y = data["y"]
    m = X.shape[1] if data["kind"] == "dense" else data["m"]
    print(f"[bench] generated {n:,} x {m} rows in {time.perf_counter() - t:.1f} s", file=sys.stderr, flush=True)

    ctx = gbt.Context(0)
    ctx.set_hist_kernel({"auto": ctx.HIST_AUTO, "plain": ctx.HIST_PLAIN, "rotated": ctx.HIST_ROTATED}[args.hist_kernel])
    t = time.perf_counter()
    mx = gbt.gbt_quantize(ctx, X, max_bin=cfg.max_bin)
    info = mx.info()
    print(f"[bench] quantized in {time.perf_counter() - t:.2f} s: w={info.symbol_bits} "
          f"row_words={info.row_words} total_bins={info.total_bins}", file=sys.stderr, flush=True)
    label = torch.from_numpy(y).cuda()
    margin = torch.full((n,), cfg.base_margin, dtype=torch.float32, device="cuda")
    sampler = ({"mvs": gbt.SAMPLE_MVS, "sgb": gbt.SAMPLE_SGB, "goss": gbt.SAMPLE_GOSS}[args.sampler],
               args.goss_a if args.sampler == "goss" else 0.0)
    P = gbt.make_train_params(loss=cfg.loss, max_depth=cfg.max_depth, eta=cfg.eta,
                              lambda_=cfg.lambda_, gamma=cfg.gamma,
                              min_child_weight=cfg.min_child_weight, f=cfg.f,
                              mvs_lambda=cfg.mvs_lambda, seed=cfg.seed, sampler=sampler[0], goss_a=sampler[1])
    ctx.set_timing(0)
    # the boosting loop: one call trains a run of trees, each queued before
    # the host reads the one before it
    P.iteration = 0
    warm = gbt.gbt_train_trees(ctx, mx, label, margin, P, args.warmup)
    first_trees = [tr.nodes.copy() for tr in warm]
    first_updates = [tr.stats.hist_updates for tr in warm]
    torch.cuda.synchronize()
    # the timed steps carry no events: a HIP event pair around each histogram
    # launch leaves the GPU idle for a few microseconds per event
    t0 = time.perf_counter()
    P.iteration = args.warmup
    stats = [tr.stats for tr in gbt.gbt_train_trees(ctx, mx, label, margin, P, args.steps)]
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    print(f"[bench] {args.steps} trees in {dt:.3f} s", file=sys.stderr, flush=True)
    # the histogram kernel's launch time: every histogram launch fills a pair
    # of HIP events on the compute stream with its own start and end, over as
    # many further timed trees of the same workload
    ctx.set_timing(1)
    estats = []
    t1 = time.perf_counter()
    for k in range(args.steps):
        P.iteration = args.warmup + args.steps + k
        estats.append(gbt.gbt_train_tree(ctx, mx, label, margin, P).stats)
    torch.cuda.synchronize()
    dt_ev = time.perf_counter() - t1

    # phase breakdown from extra trees with every phase bracketed by events
    # (outside the timed region: the events themselves add gaps)
    ctx.set_timing(2)
    pstats = []
    for k in range(3):
        P.iteration = args.warmup + 2 * args.steps + k
        pstats.append(gbt.gbt_train_tree(ctx, mx, label, margin, P).stats)
    ctx.set_timing(0)
    # the training loss after every tree of this run (warm-up, timed, event
    # and phase trees), for comparing samplers
    with torch.no_grad():
        if cfg.loss == gbt.LOSS_SQUARED:
            train_loss = float(((margin.double() - label.double()) ** 2).mean() / 2)
        else:
            z = margin.double()
            train_loss = float((torch.nn.functional.softplus(z) - label.double() * z).mean())
    n_trees_run = args.warmup + 2 * args.steps + 3
    # counter calibration: one plain device-to-device copy of known size
    src = torch.empty(CALIB_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    upd = sum(s.hist_updates for s in stats)
    hbytes = sum(s.hist_bytes for s in estats)
    hms = sum(s.ms_hist for s in estats)
    launches = sum(s.hist_launches for s in estats)
    phases = {k: round(sum(getattr(s, "ms_" + k) for s in pstats) / len(pstats), 4)
              for k in ("sample", "hist", "hist_aux", "split", "margin", "total")}
    achieved = hbytes / (hms * 1e-3) / 1e9 if hms > 0 else 0.0
    kernels = {HIST_KERNELS.get(s.hist_kernel, "k_hist_sparse") for s in stats + estats}
    kernel = kernels.pop() if len(kernels) == 1 else "+".join(sorted(kernels))
    line = {
        "metric": METRIC,
        "value": round(upd / dt / 1e9, 4),
        "unit": "G updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(dt * 1e3 / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {"workload": desc.format(n=n, f=cfg.f) + ("" if args.sampler == "mvs" or cfg.f >= 1
                                                              else f", {args.sampler.upper()} sampler"),
                   "rows": n, "features": m, "max_bin": cfg.max_bin, "max_depth": cfg.max_depth,
                   "f": cfg.f, "sampler": args.sampler if cfg.f < 1 else "none",
                   **({"goss_a": args.goss_a} if args.sampler == "goss" and cfg.f < 1 else {})},
        "sec_per_tree": round(dt / args.steps, 6),
        "rows_sampled_per_tree": round(sum(s.n_sampled for s in stats) / args.steps),
        "hist_updates_per_tree": upd // args.steps,
        "train_loss_after": {"trees": n_trees_run, "loss": round(train_loss, 6)},
        "phase_ms_per_tree_untimed_run": phases,
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": stored_traffic(workload_key(args), kernel),
                     "kernel": kernel, "launches": launches,
                     "avg_launch_us": round(hms * 1e3 / max(launches, 1), 2),
                     "algorithmic_bytes_per_launch": hbytes // max(launches, 1),
                     # of which the partition's column copy of the sampled page,
                     # written by the root pass (1 or 2 bytes per symbol)
                     "column_copy_bytes_per_launch": sum(s.hist_cols * m * s.n_sampled for s in estats)
                                                     // max(launches, 1),
                     "timing": f"start and end events of every histogram launch, filled by the launch itself "
                               f"(hipExtLaunchKernel), over {args.steps} further timed trees "
                               f"({round(dt_ev * 1e3 / args.steps, 4)} ms per tree with the events)"},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(X, y, cfg, args.cpu_trees, first_trees, first_updates, sampler)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
