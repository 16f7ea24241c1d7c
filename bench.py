#!/usr/bin/env python3
"""Benchmark of the per-window feature-fetch path on one MI355X.

One step = one window of W consecutive GraphSAGE mini-batches through the
whole path: sampling, hot-set build, owner bucketing, bulk staging and the
W per-batch gathers (with the miss path).  Inputs (CSR, feature shards,
seeds) are resident in HBM before the timed region.  Steps cycle through
the windows of one epoch.  Prints one JSON line on stdout.

value   = feature rows gathered per second over the timed steps.
roofline: the gather (gg_gather_batch) is the dominant kernel; its
          algorithmic bytes per launch (2 * row_bytes + 4 B id per row, + 4 B
          slot lookup per remote row) over its HIP-event duration, against
          8 TB/s HBM.
cpu_baseline: the single-threaded CPU oracle on one window of the same
          workload, on this host.
"""
import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PCIE5_X16_GBS = 63.0   # 32 GT/s x 16 lanes x 128/130 encoding / 8 bits
HBM_PEAK_GBS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")
GATHER_SOURCES = ["paper_2606_02916_amd/csrc/gather.hip", "paper_2606_02916_amd/csrc/gg_dev.hpp"]


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor()


def gather_source_sha():
    import hashlib
    h = hashlib.sha256()
    for f in GATHER_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def counters_path(workload):
    return os.path.join(PROFILES, f"gather_{workload}_counters.txt")


def measured_traffic(workload, per_batch):
    """HBM bytes per gather launch from the committed counter summary, or
    None when there is none for this workload or the kernel source changed."""
    path = counters_path(workload)
    if per_batch or not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.loads("".join(l for l in f if not l.startswith("#")))
    if d.get("source_sha") != gather_source_sha():
        return None
    return int(d["traffic_bytes_per_launch"])


def _short(name):
    import re
    m = re.search(r"(k_[a-z_0-9]+)(<[^>]*>)?", name)
    return (m.group(1) + (m.group(2) or "")) if m else name.split("(")[0][:48]


def summarize(args):
    """Writes profiles/ summaries from rocprofv3 databases of bench runs."""
    import sqlite3
    wl = args.config
    name = args.profile_name or wl   # file names; gather counters only for the default run
    os.makedirs(PROFILES, exist_ok=True)
    cmd = args.summary_command
    if args.trace_db:
        db = sqlite3.connect(args.trace_db)
        rows = db.execute("select name, count(*), avg(end-start), min(end-start), max(end-start), "
                          "sum(end-start) from kernels group by name order by sum(end-start) "
                          "desc").fetchall()
        tot = sum(r[5] for r in rows)
        out = [f"# rocprofv3 kernel trace of bench.py, workload {wl} ({name})",
               f"# command: {cmd}",
               f"# gather source sha: {gather_source_sha()}",
               f"{'kernel':40s} {'calls':>6s} {'avg_us':>9s} {'min_us':>9s} {'max_us':>9s} "
               f"{'total_ms':>9s} {'share':>6s}"]
        for n, c, a, mn, mx, sm in rows:
            out.append(f"{_short(n):40s} {c:6d} {a / 1e3:9.2f} {mn / 1e3:9.2f} {mx / 1e3:9.2f} "
                       f"{sm / 1e6:9.3f} {100 * sm / tot:5.1f}%")
        if args.phases:
            # the gather call's kernels per launch, split into the bench's
            # phases (pre-pass, warm-up, timed steps) by dispatch order; with
            # the look-ahead driver the pre-pass alternates the pipeline's
            # gather and the timed regather (the odd launches)
            n_pre, n_warm, n_timed = (int(x) for x in args.phases.split(","))
            per = {}
            for part in ("k_gather_rows", "k_gather_finish"):
                per[part] = [r[0] for r in db.execute(
                    "select end-start from kernels where name like ? order by start",
                    (f"%{part}%",)).fetchall()]
            n = len(per["k_gather_rows"])
            calls = [sum(per[p][i] for p in per if i < len(per[p])) for i in range(n)]
            out.append("")
            out.append("# gg_gather_batch (rows + finish) by bench phase, microseconds")
            for label, lo, hi, step in (("pre-pass, all launches", 0, n_pre, 1),
                                        ("pre-pass, odd launches", 1, n_pre, 2),
                                        ("timed steps", n - n_timed, n, 1)):
                v = calls[lo:hi:step]
                r = per["k_gather_rows"][lo:hi:step]
                if v:
                    out.append(f"{label:34s} launches {len(v):3d}  call avg {sum(v) / len(v) / 1e3:8.2f}"
                               f"  k_gather_rows avg {sum(r) / len(r) / 1e3:8.2f}")
        if args.bench_json:
            # the JSON line bench.py printed in the traced run: its HIP-event
            # gather durations, to set beside rocprofv3's
            with open(args.bench_json) as f:
                b = json.loads(f.read().strip().splitlines()[-1])
            r = b["roofline"]
            out.append("")
            out.append(f"# bench.py line of the traced run: ms_per_step {b['ms_per_step']}, "
                       f"gg_gather_batch {r['avg_launch_us']} us per launch over the timed steps "
                       f"(HIP events, frac {r['frac']}), {r['isolated']['avg_launch_us']} us "
                       f"isolated (frac {r['isolated']['frac']})")
        if args.plain_json:
            # the same command without the profiler: rocprofv3 costs the host
            # 10-40 us per launch, so a traced look-ahead run is bound by the
            # host's enqueue, its chains overlap less and its gathers run
            # with more of the chip than in the unprofiled run
            with open(args.plain_json) as f:
                b = json.loads(f.read().strip().splitlines()[-1])
            r = b["roofline"]
            out.append(f"# the same command without the profiler: ms_per_step "
                       f"{b['ms_per_step']}, gg_gather_batch {r['avg_launch_us']} us per launch "
                       f"over the timed steps (HIP events, frac {r['frac']}), "
                       f"{r['isolated']['avg_launch_us']} us isolated (frac "
                       f"{r['isolated']['frac']}); under the profiler the host's enqueue "
                       f"(10-40 us per launch) bounds the pipeline, which then overlaps less")
        copies = [r[0] for r in db.execute("select end-start from kernels where name like "
                                           "'%copyBuffer%' order by end-start desc limit 3")]
        if args.copy_calibration_mib and copies:
            # the run's plain 1 GiB device-to-device copies: the practical
            # ceiling of a streaming copy on this part
            us = sorted(copies)[len(copies) // 2] / 1e3
            nb = 2 * args.copy_calibration_mib * (1 << 20)
            out.append("")
            out.append(f"# practical ceiling: {args.copy_calibration_mib} MiB device-to-device "
                       f"copy (runtime copy kernel), median of the 3 longest: {us:.1f} us, "
                       f"{nb / (us * 1e-6) / 1e12:.2f} TB/s read+write "
                       f"({nb / (us * 1e-6) / 1e9 / HBM_PEAK_GBS:.2f} of {HBM_PEAK_GBS / 1e3:.0f} TB/s)")
        with open(os.path.join(PROFILES, f"kernels_{name}.txt"), "w") as f:
            f.write("\n".join(out) + "\n")
    if args.fetch_db and args.write_db and name == wl:
        def per_kernel(path, counter):
            db = sqlite3.connect(path)
            r = db.execute("select kernel_name, value from counters_collection where "
                           "counter_name = ?", (counter,)).fetchall()
            gather = [v for n, v in r if "k_gather_rows" in n]
            copies = sorted((v for n, v in r if "copyBuffer" in n), reverse=True)[:3]
            return sum(gather) / len(gather), sum(copies) / len(copies), len(gather)
        f_g, f_c, n_g = per_kernel(args.fetch_db, "FETCH_SIZE")
        w_g, w_c, _ = per_kernel(args.write_db, "WRITE_SIZE")
        known_kib = args.copy_calibration_mib * 1024
        fs, wsc = known_kib / f_c, known_kib / w_c
        traffic = int(round((f_g * fs + w_g * wsc) * 1024))
        d = {"kernel": "k_gather_rows", "workload": wl, "launches": n_g,
             "source_sha": gather_source_sha(),
             "fetch_kib_per_launch_raw": round(f_g, 1), "write_kib_per_launch_raw": round(w_g, 1),
             "calibration": {"copy_mib": args.copy_calibration_mib,
                             "fetch_kib_raw": round(f_c, 1), "write_kib_raw": round(w_c, 1)},
             "fetch_scale": round(fs, 4), "write_scale": round(wsc, 4),
             "traffic_bytes_per_launch": traffic}
        with open(counters_path(wl), "w") as f:
            f.write(f"# HBM counters of k_gather_rows (window-mode gather), workload {wl}\n")
            f.write(f"# command (FETCH_SIZE, then WRITE_SIZE): {cmd}\n")
            f.write("# scale = known bytes of a 1 GiB device-to-device copy / counter reading\n")
            f.write(json.dumps(d, indent=1) + "\n")
    if args.fetch_db and args.write_db and args.trace_db and args.traffic_out:
        # every kernel's HBM-side traffic: FETCH_SIZE and WRITE_SIZE per
        # dispatch, scaled by what they read for the run's 1 GiB copies,
        # beside its average duration from the kernel trace
        def per_name(path, counter):
            db = sqlite3.connect(path)
            r = db.execute("select kernel_name, value from counters_collection where "
                           "counter_name = ?", (counter,)).fetchall()
            agg, copies = {}, sorted((v for n, v in r if "copyBuffer" in n), reverse=True)[:3]
            for n, v in r:
                a = agg.setdefault(_short(n), [0, 0.0])
                a[0] += 1
                a[1] += v
            return agg, sum(copies) / len(copies)
        fa, f_c = per_name(args.fetch_db, "FETCH_SIZE")
        wa, w_c = per_name(args.write_db, "WRITE_SIZE")
        known_kib = args.copy_calibration_mib * 1024
        fs, wsc = known_kib / f_c, known_kib / w_c
        db = sqlite3.connect(args.trace_db)
        dur = {}
        for n, c, a in db.execute("select name, count(*), avg(end-start) from kernels group by "
                                  "name").fetchall():
            d = dur.setdefault(_short(n), [0, 0.0])
            d[1] = (d[1] * d[0] + a * c) / (d[0] + c)
            d[0] += c
        out = [f"# HBM-side traffic of every kernel of bench.py, workload {wl} ({name}): "
               f"FETCH_SIZE and WRITE_SIZE per dispatch",
               f"# command (trace, FETCH_SIZE, WRITE_SIZE: three runs): {cmd}",
               f"# scale: known bytes of a {args.copy_calibration_mib} MiB device-to-device copy / "
               f"counter reading (fetch x{fs:.3f}, write x{wsc:.3f}); MB = 1e6 bytes; the "
               f"counters see L2 misses, some of which the last-level (Infinity) cache serves",
               f"{'kernel':40s} {'dispatches':>10s} {'avg_us':>8s} {'fetch_MB':>9s} "
               f"{'write_MB':>9s} {'GB/s':>8s}"]
        names = sorted(fa, key=lambda k: -(fa[k][1] / fa[k][0] * fs +
                                           wa.get(k, (1, 0.0))[1] / wa.get(k, (1, 0.0))[0] * wsc))
        for k in names:
            f_mb = fa[k][1] / fa[k][0] * fs * 1024 / 1e6
            w = wa.get(k)
            w_mb = (w[1] / w[0] * wsc * 1024 / 1e6) if w else 0.0
            us = dur.get(k, [0, 0.0])[1] / 1e3
            gbs = (f_mb + w_mb) * 1e6 / (us * 1e-6) / 1e9 if us else 0.0
            out.append(f"{k:40s} {fa[k][0]:10d} {us:8.2f} {f_mb:9.2f} {w_mb:9.2f} {gbs:8.1f}")
        with open(os.path.join(PROFILES, f"{args.traffic_out}_{name}.txt"), "w") as f:
            f.write("\n".join(out) + "\n")
    if args.pmc_db:
        # per-kernel averages of every counter in a rocprofv3 --pmc run
        db = sqlite3.connect(args.pmc_db)
        rows = db.execute("select kernel_name, counter_name, count(*), avg(value) from "
                          "counters_collection group by kernel_name, counter_name").fetchall()
        per = {}
        for n, c, k, v in rows:
            per.setdefault(_short(n), {})[c] = (k, v)
        names = sorted({c for _, c, _, _ in rows})
        out = [f"# rocprofv3 counters of bench.py, workload {wl}: per-dispatch averages",
               f"# command: {cmd}",
               f"{'kernel':40s} {'dispatches':>10s} " + " ".join(f"{c:>24s}" for c in names)]
        for kn in sorted(per, key=lambda x: -max(v for _, v in per[x].values())):
            k0 = max(k for k, _ in per[kn].values())
            out.append(f"{kn:40s} {k0:10d} " + " ".join(
                f"{per[kn][c][1]:24.1f}" if c in per[kn] else f"{'-':>24s}" for c in names))
        with open(os.path.join(PROFILES, f"{args.pmc_out}_{wl}.txt"), "w") as f:
            f.write("\n".join(out) + "\n")
    print("summaries written", file=sys.stderr)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=24)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="large_sparse",
                    help="tiny | dense_mid | large_sparse | wsweep | small")
    ap.add_argument("--W", type=int, default=None, help="window size (default: the workload's)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--line-wsweep", default="1,2,4,8,16,32",
                    help="window sizes of the W sweep added to the default line (batch 4096 "
                         "on the large sparse graph, look-ahead driver); empty to skip")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="minimum oracle time for the CPU baseline sample")
    ap.add_argument("--per-batch", action="store_true",
                    help="one gather launch per batch instead of one per window (sequential "
                         "driver only)")
    ap.add_argument("--pipeline", default="lookahead",
                    choices=["sequential", "delta", "inplace", "lookahead"],
                    help="sequential: the five calls per window on one stream, full restage; "
                         "delta: the same with delta staging, retained rows copied from the "
                         "previous cache; inplace: delta staging into one persistent cache; "
                         "lookahead: in-place staging, window k+1 built and staged on a second "
                         "stream while window k is gathered")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after the timed steps, copy this many MiB device to device three "
                         "times (a plain copy of known size for scaling HBM counters)")
    ap.add_argument("--consumer", type=int, default=0, metavar="CLASSES",
                    help="also run the GraphSAGE consumer (mean aggregator, 16 hidden units, "
                         "CLASSES outputs, one layer per sampling hop) on every window's rows "
                         "inside the step, and report its time and MFMA rate")
    ap.add_argument("--breakdown", action="store_true",
                    help="record events between sampling, hot set and bucketing as well (each "
                         "event on the build stream costs a few us per window)")
    ap.add_argument("--tune", default=None, metavar="FIELD=VALUE,...",
                    help="launch tuning passed to every call (gg_tuning_t fields, e.g. "
                         "gather_blocks=768,gather_loads=8); results do not change")
    ap.add_argument("--stage-apart", type=int, default=None, choices=(0, 1),
                    help="look-ahead driver: staging on a stream of its own (1) or after the "
                         "build on the build stream (0); default: its own only with shards in "
                         "host memory")
    ap.add_argument("--sets", type=int, default=None,
                    help="buffer sets of the look-ahead pipeline (how far building may run ahead)")
    ap.add_argument("--wsweep", default=None,
                    help="comma-separated window sizes: run one epoch per W and report, per W, "
                         "hot-set size, bulk bytes per owner, rebuild delta and gather rate")
    ap.add_argument("--wsweep-table", default=None,
                    help="with --wsweep: also write the sweep as a text table to this file")
    ap.add_argument("--simulate", default=None,
                    help="comma-separated window sizes: replay one epoch per W and per hot-set "
                         "budget through the fetch path and report the simulator's event counts "
                         "z(W) and energy estimate E_phy(W) (synthetic coefficients)")
    ap.add_argument("--n-hot", default="-1",
                    help="with --simulate: comma-separated hot-set budgets (-1 = union)")
    ap.add_argument("--hot-frac", default=None,
                    help="with --simulate: budgets relative to each window, e.g. 1/10,1/4: the "
                         "top fraction of the window's distinct remote nodes; the hit ratio is "
                         "then the share of remote requests that fraction covers")
    ap.add_argument("--graph", action="store_true",
                    help="time the sequential driver launched call by call against the same "
                         "windows replayed from HIP graphs; prints one JSON line")
    ap.add_argument("--ablation", action="store_true",
                    help="measure per-row requests against bulk requests, rows per wavefront "
                         "copy step, and (host-resident shards) zero-copy staging against "
                         "pack + DMA, on the first window; prints one JSON line")
    ap.add_argument("--ablation-rows", type=int, default=100_000,
                    help="with --ablation: staged rows copied one request each")
    ap.add_argument("--summarize", action="store_true",
                    help="write profiles/ summaries from rocprofv3 databases instead of running")
    ap.add_argument("--trace-db", default=None)
    ap.add_argument("--fetch-db", default=None)
    ap.add_argument("--write-db", default=None)
    ap.add_argument("--summary-command", default="")
    ap.add_argument("--pmc-db", default=None,
                    help="with --summarize: a rocprofv3 --pmc database; writes per-kernel "
                         "averages of its counters to profiles/<pmc-out>_<config>.txt")
    ap.add_argument("--pmc-out", default="counters")
    ap.add_argument("--profile-name", default=None,
                    help="with --summarize: name of the summaries (default: the workload); the "
                         "gather's counter summary, which the bench line reads, is written only "
                         "for the default name")
    ap.add_argument("--traffic-out", default=None,
                    help="with --summarize and trace, fetch and write databases: write every "
                         "kernel's calibrated traffic and duration to profiles/<name>_<config>.txt")
    ap.add_argument("--bench-json", default=None,
                    help="with --summarize: the JSON line bench.py printed in the traced run")
    ap.add_argument("--plain-json", default=None,
                    help="with --summarize: the JSON line of the same command run without the "
                         "profiler")
    ap.add_argument("--phases", default=None,
                    help="with --trace-db: gather launches of the pre-pass (two per window "
                         "with the look-ahead driver), warm-up and timed steps, e.g. 24,1,12, "
                         "to average the gather per phase")
    args = ap.parse_args()
    if args.summarize:
        summarize(args)
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs the per-window fetch path on one GPU only; with several GPUs each "
              "would run its own partition's windows, which is not implemented here",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    from paper_2606_02916_amd import FetchPipeline, LookaheadPipeline

    dev = torch.device("cuda:0")
    wl = synth.WORKLOADS[args.config]
    if args.per_batch and args.pipeline != "sequential":
        ap.error("--per-batch needs --pipeline sequential")
    if args.wsweep:
        return wsweep(args, wl)
    if args.simulate:
        return simulate(args, wl)
    if args.ablation:
        return ablation(args, wl)
    if args.graph:
        return graph_mode(args, wl)
    W = args.W or wl.W
    t = time.time()
    inst, row_ptr_d, col_idx_d, shards_d = synth.torch_instance(args.config, dev)
    log(f"generated {args.config}: N={wl.num_nodes} E={wl.num_edges} in {time.time() - t:.1f}s")
    P, L = wl.num_parts, len(wl.fanout)
    seeds_d = torch.from_numpy(inst.seeds).to(dev)
    pcie = pcie_h2d_gbps(dev) if wl.remote_on_host else None
    pargs = (row_ptr_d, col_idx_d, P, wl.part_kind, wl.local_owner, inst.range_start, shards_d,
             [s.shape[0] for s in inst.shards], wl.row_bytes, wl.row_stride, W, wl.fanout,
             wl.batch_size)
    look = args.pipeline == "lookahead"
    inplace_cache = args.pipeline in ("lookahead", "inplace")
    tuning = parse_tuning(args.tune)
    if look:
        pipe = LookaheadPipeline(*pargs, device=dev, nsets=args.sets, tuning=tuning,
                                 stage_apart=None if args.stage_apart is None
                                 else bool(args.stage_apart))
    else:
        pipe = FetchPipeline(*pargs, device=dev, delta=args.pipeline == "delta",
                             inplace=args.pipeline == "inplace", tuning=tuning)
    boff = inst.batch_off
    nwin = synth.n_windows(boff, W)
    wins = []
    for k in range(nwin):
        b0, b1 = synth.window_batches(boff, W, k)
        so = boff[b0:b1 + 1] - boff[b0]
        wins.append((seeds_d[boff[b0]:boff[b1]], so, b0))
    cons, cons_dims = None, None
    if args.consumer:
        from paper_2606_02916_amd import SageConsumer, gg
        if args.per_batch:
            ap.error("--consumer reads whole-window gathers; drop --per-batch")
        gen = torch.Generator(device=dev).manual_seed(0)
        cons_dims = [wl.feat_dim] + [16] * (L - 1) + [args.consumer]
        layers = []
        for j in range(L):
            a, b = cons_dims[j], cons_dims[j + 1]
            layers.append((torch.randn(a, b, device=dev, generator=gen) / a ** 0.5,
                           torch.randn(a, b, device=dev, generator=gen) / a ** 0.5,
                           0.1 * torch.randn(b, device=dev, generator=gen), j < L - 1))
        cons = SageConsumer(pipe.geo, layers, device=dev,
                            x_dtype=gg.GG_F16 if wl.feat_dtype == "fp16" else gg.GG_F32)
    torch.cuda.synchronize()
    log(f"uploaded; {nwin} windows of W={W}; out_cap={pipe.geo.out_cap} "
        f"hot_cap={pipe.geo.hot_cap}; driver {args.pipeline}")

    def run_window(s, so, b0, events=None, gevs=None, cevs=None):
        """Enqueues one window; returns (Wk, object holding its statistics)."""
        if look:
            return pipe.window(s, so, b0, events=events,
                               gather_events=gevs[0] if gevs is not None else None,
                               consumer=cons, consumer_events=cevs)
        Wk = pipe.window(s, so, b0, events=events, gather_events=gevs, per_batch=pb,
                         consumer=cons, consumer_events=cevs)
        return Wk, pipe.buf

    # Pass over every window once: per-window row counts for the metric and
    # per-batch local/remote counts for the gather's algorithmic bytes.
    rb = wl.row_bytes
    mk = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    rows_w, gbytes_w, hot_w, sbytes_w, req_w, hbytes_w, lev_w = [], [], [], [], [], [], []
    pb = args.per_batch
    iso_ms = []      # gather launches with the chip to themselves
    iso_st_ms = []   # staging calls with the chip to themselves
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev) if look else None
    for k, (s, so, b0) in enumerate(wins):
        ge = [(mk(), mk()) for _ in range(W if pb else 1)]
        Wk, sb = run_window(s, so, b0, gevs=None if look else ge)
        torch.cuda.synchronize()
        if look:
            # The same gather once more on one stream after the window is
            # complete, so no cross-stream wait falls inside the interval.
            # A 512 MiB fill first evicts the window's rows from the
            # last-level cache and keeps the queue busy while the gather is
            # enqueued behind it.
            flush.fill_(k & 0xFF)
            ge[0][0].record()
            pipe.regather(sb, Wk)
            ge[0][1].record()
            torch.cuda.synchronize()
            # and its staging call, the same way (it rewrites the same slots)
            se = (mk(), mk())
            flush.fill_((k + 1) & 0xFF)
            se[0].record()
            pipe.restage()
            se[1].record()
            torch.cuda.synchronize()
            iso_st_ms.append(se[0].elapsed_time(se[1]))
        iso_ms += [a.elapsed_time(b) for a, b in ge[:Wk if pb else 1]]
        st = pipe.read_status()
        if st != 0:
            raise RuntimeError(f"device status {st} in window {k}")
        g = [sb.gather_stats_dict(b) for b in range(Wk)]
        rows_w.append(sum(x["rows"] for x in g))
        gb = [x["rows"] * (2 * rb + 4) + (x["hits"] + x["misses"]) * 4 for x in g]
        gbytes_w.append(gb if pb else [sum(gb)])
        ss = sb.stage_stats_dict()
        hot_w.append(ss["rows_total"])
        # a staged row moves 2 * row_bytes and its id and remap entry; a row
        # kept in place only its id, old and new remap entries
        kept = ss["retained"] if inplace_cache else 0
        sbytes_w.append((ss["rows_total"] - kept) * (2 * rb + 8) + kept * 12 +
                        ss["invalidated"] * 4)
        req_w.append(ss["requests_total"])
        hbytes_w.append(sum(ss["bytes"][m] for m in range(P) if not shards_d[m].is_cuda))
        fo = sb.frontier_off[:(L + 1) * Wk + 1].cpu().numpy()
        lev_w.append([int(fo[(l + 1) * Wk] - fo[l * Wk]) for l in range(L + 1)])
    del flush
    log(f"rows per window: {rows_w[:4]}... hot set: {hot_w[:4]}...")

    for i in range(args.warmup):
        s, so, b0 = wins[i % nwin]
        run_window(s, so, b0)
    torch.cuda.synchronize()

    K = args.steps
    # With staging on the build stream, the gather stream's queue holds only
    # the gathers and one end event each: the gather then starts at the
    # later of its window's staging end (events[4]) and the previous
    # gather's end, and every marker left out of that queue saves a few us.
    stage_on_build = look and pipe.stage_stream is pipe.build_stream
    hs_on_stage = look and pipe.hotset_on_stage
    # The build stream carries the critical chain and each event on it costs
    # a few us too: by default only the build's end and the staging's end
    # are recorded, and a build is taken to run from the previous window's
    # staging end (staging on the build stream) or build end (staging on a
    # stream of its own; the build then ends with the sampling when the hot
    # set and buckets follow it on the staging stream); a gather, from the
    # later of its staging's end and the previous gather's end (--breakdown:
    # every call).
    lean = look and not args.breakdown
    b_end = 1 if hs_on_stage else 3      # the event that ends a build
    evs = [[None if lean and j < 3 and j != b_end else mk() for j in range(5 if look else 6)]
           for _ in range(K)]
    gevs = [[(None if lean or stage_on_build else mk(), mk()) for _ in range(W if pb else 1)]
            for _ in range(K)]
    cevs = [(mk(), mk()) for _ in range(K)] if cons else [None] * K
    order = [(args.warmup + i) % nwin for i in range(K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i, k in enumerate(order):
        s, so, b0 = wins[k]
        run_window(s, so, b0, events=evs[i], gevs=gevs[i], cevs=cevs[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    if pipe.read_status() != 0:
        raise RuntimeError(f"device status {pipe.read_status()} after the timed steps")
    elapsed = t1 - t0
    rows = sum(rows_w[k] for k in order)
    value = rows / elapsed

    def gather_ms(gevs, i, b=None):
        """Duration of gather launch b of step i (all launches when b is
        None).  Without a start event the gather began at the later of its
        window's staging end and the previous gather's end (the first timed
        gather is charged from its staging end)."""
        if b is None:
            return sum(gather_ms(gevs, i, j) for j in range(len(gevs[i])))
        s, e = gevs[i][b]
        if s is not None:
            return s.elapsed_time(e)
        t = evs[i][4].elapsed_time(e)
        if i > 0:
            t = min(t, gevs[i - 1][-1][1].elapsed_time(e))
        return t

    g_ms, g_bytes, n_launch = 0.0, 0, 0
    stage_ms = ({"build": [], "stage": [], "gathers": []} if lean else
                {"sample": [], "hotset": [], "bucket": [], "stage": [], "gathers": []})
    st_ms, st_bytes, st_host_bytes = 0.0, 0, 0
    for i, k in enumerate(order):
        e = evs[i]
        if lean:
            if i > 0:
                stage_ms["build"].append(
                    evs[i - 1][4 if stage_on_build else b_end].elapsed_time(e[b_end]))
        else:
            for name, (a, b) in zip(stage_ms, [(0, 1), (1, 2), (2, 3)]):
                stage_ms[name].append(e[a].elapsed_time(e[b]))
        # staging starts at the buckets' end (on the staging stream too when
        # the hot set and buckets follow the sampling there); on a stream of
        # its own, at the later of that, the previous window's staging end
        # and, with more than two buffer sets, the end of the gather of
        # window k - 2, whose slots it may reuse and which it waits for
        t_st = e[3].elapsed_time(e[4])
        if look and not stage_on_build and i > 0:
            t_st = min(t_st, evs[i - 1][4].elapsed_time(e[4]))
            if i > 1 and pipe.nsets > 2:
                t_st = min(t_st, gevs[i - 2][-1][1].elapsed_time(e[4]))
        stage_ms["stage"].append(t_st)
        stage_ms["gathers"].append(gather_ms(gevs, i))
        st_ms += t_st
        st_bytes += sbytes_w[k]
        st_host_bytes += hbytes_w[k]
        for b in range(len(gbytes_w[k])):
            g_ms += gather_ms(gevs, i, b)
            g_bytes += gbytes_w[k][b]
            n_launch += 1
    win_bytes = (g_bytes + (st_bytes if pcie is None else 0)) / K
    stage_call = "gg_stage_inplace" if inplace_cache else "gg_stage_bulk"
    # per-window times: between consecutive windows' last gather ends (the
    # first timed window has no predecessor event and is left out)
    win_ms = [gevs[i - 1][-1][1].elapsed_time(gevs[i][-1][1]) for i in range(1, K)]
    avg_ms = g_ms / n_launch
    avg_bytes = g_bytes / n_launch
    achieved = avg_bytes / (avg_ms * 1e-3) / 1e9
    all_gb = [x for v in gbytes_w for x in v]
    iso_avg_ms = float(np.mean(iso_ms))
    iso_achieved = float(np.mean(all_gb)) / (iso_avg_ms * 1e-3) / 1e9
    stage_gbs = st_bytes / (st_ms * 1e-3) / 1e9
    iso_stage = None
    if iso_st_ms:
        # window 0 stages every row (no previous cache); the steady state is
        # the windows after it
        steady = list(range(1, nwin)) if nwin > 1 else [0]
        ib = float(np.mean([sbytes_w[k] for k in steady]))
        it = float(np.mean([iso_st_ms[k] for k in steady]))
        iso_stage = {"achieved": round(ib / (it * 1e-3) / 1e9, 1),
                     "frac": round(ib / (it * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "avg_call_us": round(it * 1e3, 2), "bytes_per_call": int(ib),
                     "calls": len(steady),
                     "note": "the look-ahead driver's staging call (all its kernels) launched "
                             "again on one stream after each pre-pass window, behind a 512 MiB "
                             "fill; windows after the first"}

    if args.copy_calibration_mib:
        nb = args.copy_calibration_mib << 20
        a = torch.empty(nb, dtype=torch.uint8, device=dev).fill_(1)
        b = torch.empty(nb, dtype=torch.uint8, device=dev)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        log(f"copy calibration: 3 x {args.copy_calibration_mib} MiB device-to-device")
        del a, b

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(inst, wl, W, wins[0][1], wins[0][2], args.cpu_seconds)

    line = {
        "metric": "feature rows gathered/s (per-window fetch path: sample, hot set, owner "
                  "buckets, bulk stage, per-batch gathers)",
        "value": round(value, 1),
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / K * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic R-MAT (a,b,c)=(0.57,0.19,0.19), seeded; features as opaque bytes",
        "config": {"workload": args.config, "nodes": wl.num_nodes, "edges": wl.num_edges,
                   "features": f"{wl.feat_dtype}x{wl.feat_dim}", "row_bytes": rb,
                   "fanout": list(wl.fanout), "batch": wl.batch_size, "W": W,
                   "partitions": P, "local_owner": wl.local_owner, "windows_per_epoch": nwin,
                   "gather_launch": "per batch" if pb else "per window",
                   "tuning": args.tune or "the driver's defaults",
                   "driver": args.pipeline + (f" ({pipe.nsets} buffer sets, staging on the "
                                              f"{'build' if stage_on_build else 'fetch'} stream)"
                                              if look else "")},
        "roofline": {"bound": "hbm", "kernel": "gg_gather_batch",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(args.config, pb),
                     "bytes_per_launch": int(avg_bytes), "avg_launch_us": round(avg_ms * 1e3, 2),
                     "overlapped": look,
                     "start": ("later of the window's staging end and the previous gather's end "
                               "(HIP events)" if gevs[0][0][0] is None
                               else "HIP event before the launch"),
                     "isolated": {"achieved": round(iso_achieved, 1),
                                  "frac": round(iso_achieved / HBM_PEAK_GBS, 4),
                                  "avg_launch_us": round(iso_avg_ms * 1e3, 2),
                                  "launches": len(iso_ms),
                                  "note": "pre-pass over every window, one window at a "
                                          "time" + ("; the look-ahead driver's gather launched "
                                                    "again on one stream" if look else "")}},
        "window_hbm": {"bytes_per_window": int(win_bytes),
                       "achieved": round(win_bytes / (elapsed / K) / 1e9, 1),
                       "frac": round(win_bytes / (elapsed / K) / 1e9 / HBM_PEAK_GBS, 4),
                       "unit": "GB/s",
                       "note": "algorithmic bytes of the gathers and of staging from HBM "
                               "shards over the whole window time (sampling, hot set and "
                               "bucketing not counted): the share of HBM the overlapped kernels "
                               "use together"},
        "stage_roofline": ({"kernel": stage_call, "bound": "hbm",
                            "achieved": round(stage_gbs, 1),
                            "frac": round(stage_gbs / HBM_PEAK_GBS, 4), "unit": "GB/s",
                            "bytes_per_call": int(np.mean(sbytes_w)),
                            "overlapped": look,
                            "start": ("the latest of the buckets' end, the previous staging's "
                                      "end and (staging on a stream of its own) the end of the "
                                      "gather whose slots it reuses (HIP events)" if look
                                      else "HIP event before the call"),
                            "isolated": iso_stage}
                           if pcie is None else
                           {"kernel": stage_call, "bound": "pcie",
                            "achieved": round(st_host_bytes / (st_ms * 1e-3) / 1e9, 2),
                            "peak": PCIE5_X16_GBS, "unit": "GB/s",
                            "frac": round(st_host_bytes / (st_ms * 1e-3) / 1e9 / PCIE5_X16_GBS, 4),
                            "dma_copy_gbps": round(pcie, 2),
                            "note": "host bytes the staging kernel reads over PCIe; peak is the "
                                    "PCIe 5.0 x16 link rate, dma_copy_gbps a measured "
                                    "pinned-to-device copy of 1 GiB"}),
        "window_ms": ({"median": round(float(np.median(win_ms)), 4),
                       "min": round(float(np.min(win_ms)), 4),
                       "max": round(float(np.max(win_ms)), 4), "windows": len(win_ms),
                       "note": "between consecutive windows' last gather ends"}
                      if win_ms else None),
        "stage_ms_median": {k: round(float(np.median(v)), 4) for k, v in stage_ms.items() if v},
        "rows_per_window": int(np.mean(rows_w)),
        "hot_set_rows_per_window": int(np.mean(hot_w)),
        "bulk_requests_per_window": float(np.mean(req_w)),
        "gather_rows_per_s": round(rows / (g_ms * 1e-3) if g_ms else 0.0, 1),
        "consumer": consumer_report(cons_dims, lev_w, order, cevs, wl) if cons else None,
        "cpu_baseline": cpu,
        "wsweep": None,
    }
    if args.line_wsweep and args.config == "large_sparse" and not args.consumer:
        del pipe
        torch.cuda.empty_cache()
        Ws = [int(x) for x in args.line_wsweep.split(",")]
        t_sw = time.perf_counter()
        sweep = {"workload": "wsweep", "batch": synth.WORKLOADS["wsweep"].batch_size,
                 "driver": "lookahead", "per_W": wsweep_lookahead(dev, "wsweep", Ws, tuning),
                 "note": "one untimed epoch per W (every buffer set used once), then the "
                         "epoch cycled 4 times (at least 8 windows) timed; gather rate from "
                         "HIP events as in roofline; counts from the "
                         "untimed epoch (bulk bytes per owner: the rows each owner's one request "
                         "moves, i.e. the rebuild delta); gpu_ms_per_window: mean period of the "
                         "gather ends over whole epochs of windows enqueued behind a blocker on "
                         "the caller's stream (the GPU runs them back to back, whatever the "
                         "host's enqueue rate; queued says the host finished enqueuing before "
                         "the GPU had gathered the third), host_enqueue_ms_per_window: the "
                         "host's time per window in that run"}
        sweep["wall_s"] = round(time.perf_counter() - t_sw, 1)
        line["wsweep"] = sweep
    print(json.dumps(line), flush=True)


def parse_tuning(spec):
    """--tune FIELD=VALUE,... as a gg_tuning_t (None when empty)."""
    from paper_2606_02916_amd import gg
    if not spec:
        return None
    fields = {}
    for item in spec.split(","):
        k, _, v = item.partition("=")
        fields[k.strip()] = int(v)
    return gg.make_tuning(**fields)


def consumer_report(dims, lev_w, order, cevs, wl):
    """GraphSAGE consumer per window: time (HIP events on its stream), the
    dense products' flops (layer j projects the rows of level L-j+1 from
    d_in to 2 * d_out), their rate against the fp32 MFMA peak, and the rate
    of the first layer's read of the gathered rows."""
    import numpy as np
    L = len(dims) - 1
    ms, flops, xbytes = [], 0, 0
    for i, k in enumerate(order):
        ms.append(cevs[i][0].elapsed_time(cevs[i][1]))
        lev = lev_w[k]
        for j in range(1, L + 1):
            flops += 2 * lev[L - j + 1] * dims[j - 1] * 2 * dims[j]
        xbytes += lev[L] * wl.row_bytes
    t = sum(ms) * 1e-3
    return {"layers": dims, "aggregator": "mean", "ms_per_window_median": round(float(np.median(ms)), 4),
            "flops_per_window": int(flops / len(order)),
            "tflops": round(flops / t / 1e12, 3), "peak_tflops_fp32_mfma": 157.3,
            "mfma_frac": round(flops / t / 1e12 / 157.3, 5),
            "x_read_gbps": round(xbytes / t / 1e9, 1),
            "note": "the consumer's time is on its own events; it overlaps the next window's "
                    "build under the look-ahead driver"}


def pcie_h2d_gbps(dev):
    """Pinned host to device copy rate of 1 GiB (best of 3), the PCIe ceiling
    for staging rows that live in host memory."""
    import torch
    a = torch.empty(1 << 30, dtype=torch.uint8, pin_memory=True)
    b = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    best = 1e9
    for _ in range(3):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        b.copy_(a, non_blocking=True)
        e1.record()
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1))
    del a, b
    return (1 << 30) / (best * 1e-3) / 1e9


def _hip_runtime():
    """The HIP runtime this process already uses (torch and libgg bind the
    same one), opened again by the path it is mapped from."""
    import ctypes as C
    paths = set()
    with open("/proc/self/maps") as f:
        for line in f:
            parts = line.split()
            if len(parts) >= 6 and os.path.basename(parts[5]).startswith("libamdhip64.so"):
                paths.add(parts[5])
    if len(paths) != 1:
        raise RuntimeError(f"expected one mapped HIP runtime, found {sorted(paths)}")
    hip = C.CDLL(paths.pop())
    hip.hipMemcpyAsync.restype = C.c_int
    hip.hipMemcpyAsync.argtypes = [C.c_void_p, C.c_void_p, C.c_size_t, C.c_int, C.c_void_p]
    return hip


def ablation(args, wl):
    """Measurements of three design choices on the workload's first window
    (built twice first, so everything is warm):
    - requests: one hipMemcpyAsync per staged row, on an evenly spaced
      sample of the window's hot set, against the staging call on the same
      rows (one bulk request per owner);
    - tile: rows a wavefront takes per copy step in the gather and the
      stage (1 = one wavefront per row);
    - host shards only: zero-copy staging (the kernel reads pinned host
      memory) against packing each owner's rows on the host plus one DMA
      per owner.
    Every variant's bytes are compared with the staging call's."""
    import numpy as np
    import torch

    import synth
    from paper_2606_02916_amd import FetchPipeline, gg

    dev = torch.device("cuda:0")
    inst, row_ptr_d, col_idx_d, shards_d = synth.torch_instance(args.config, dev)
    P, W, rb, stride = wl.num_parts, args.W or wl.W, wl.row_bytes, wl.row_stride
    pipe = FetchPipeline(row_ptr_d, col_idx_d, P, wl.part_kind, wl.local_owner, inst.range_start,
                         shards_d, [s.shape[0] for s in inst.shards], rb, stride, W, wl.fanout,
                         wl.batch_size, device=dev)
    seeds_d = torch.from_numpy(inst.seeds).to(dev)
    boff = inst.batch_off
    b0, b1 = synth.window_batches(boff, W, 0)
    so = boff[b0:b1 + 1] - boff[b0]
    seeds = seeds_d[boff[b0]:boff[b1]]
    for _ in range(2):
        pipe.reset_cache()
        Wk = pipe.window(seeds, so, b0)
    torch.cuda.synchronize()
    if pipe.read_status() != 0:
        raise RuntimeError(f"device status {pipe.read_status()}")
    cur = (pipe.k - 1) & 1
    H = int(pipe.hot_count[cur][0].item())
    bucket, owner_off, cache = pipe.bucket_ids[cur], pipe.owner_off, pipe.staged_cache()
    g = [pipe.buf.gather_stats_dict(b) for b in range(Wk)]
    g_rows = sum(x["rows"] for x in g)
    g_bytes = sum(x["rows"] * (2 * rb + 4) + (x["hits"] + x["misses"]) * 4 for x in g)
    s_bytes = H * (2 * rb + 8)
    mk = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    log(f"{args.config}: window 0 has {g_rows} rows, hot set {H}")

    def timed(fn, reps):
        ts = []
        for _ in range(reps):
            e0, e1 = mk(), mk()
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return float(np.median(ts))

    def stage(ids, off, n, out, slot, stats):
        gg.gg_stage_bulk(ids, off, n, pipe.part, pipe.feat, out, stride, n, slot, None, None,
                         None, None, stats, pipe.status, pipe.ws, tuning=pipe.tuning)

    def stage_full():
        stage(bucket, owner_off, pipe.hot_cap, cache, pipe.slot_of, pipe.stage_stats)

    res = {}
    # -- per-row requests against one bulk request per owner ---------------
    off_h = owner_off.cpu().numpy()
    pick = np.unique(np.linspace(0, H - 1, min(args.ablation_rows, H)).astype(np.int64))
    n = len(pick)
    own = np.searchsorted(off_h, pick, side="right") - 1
    u = bucket[:H].cpu().numpy()[pick].astype(np.int64)
    if wl.part_kind == synth.PART_RANGE:
        rows = u - np.asarray(inst.range_start, dtype=np.int64)[own]
    else:
        rows = u // P
    base = np.array([shards_d[m].data_ptr() for m in range(P)], dtype=np.int64)
    src = (base[own] + rows * stride).tolist()
    dst = torch.empty((n, stride), dtype=torch.uint8, device=dev)
    dl = (dst.data_ptr() + np.arange(n, dtype=np.int64) * stride).tolist()
    hip = _hip_runtime()
    hs = torch.cuda.current_stream().cuda_stream

    def per_row(k):
        for j in range(k):
            rc = hip.hipMemcpyAsync(dl[j], src[j], rb, 4, hs)   # hipMemcpyDefault
            if rc:
                raise RuntimeError(f"hipMemcpyAsync returned {rc}")

    per_row(min(n, 2000))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(n):
        gg.lib.gg_version()
    loop_us = (time.perf_counter() - t0) / n * 1e6
    e0, e1 = mk(), mk()
    t0 = time.perf_counter()
    e0.record()
    per_row(n)
    t_enq = time.perf_counter()
    e1.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    sub_ids = torch.from_numpy(u.astype(np.int32)).to(dev)
    cnt = np.bincount(own, minlength=P)
    sub_off = torch.from_numpy(np.concatenate([[0], np.cumsum(cnt)]).astype(np.int64)).to(dev)
    sub_cache = torch.empty((n, stride), dtype=torch.uint8, device=dev)
    sub_slot = torch.full((wl.num_nodes,), -1, dtype=torch.int32, device=dev)
    sub_stats = torch.zeros(gg.STAGE_STATS_BYTES, dtype=torch.uint8, device=dev)
    bulk_ms = timed(lambda: stage(sub_ids, sub_off, n, sub_cache, sub_slot, sub_stats), 20)
    ss = gg.stage_stats_from_bytes(sub_stats.cpu().numpy().tobytes(), P)
    same = bool(torch.equal(dst[:, :rb], sub_cache[:, :rb]))
    if not same:
        raise RuntimeError("per-row copies differ from the staging call")
    res["requests"] = {
        "rows": n, "row_bytes": rb,
        "per_row": {"requests": n, "wall_ms": round((t1 - t0) * 1e3, 3),
                    "enqueue_us_per_request": round((t_enq - t0) / n * 1e6, 3),
                    "host_loop_us_per_call": round(loop_us, 3),
                    "gpu_span_ms": round(e0.elapsed_time(e1), 3),
                    "rows_per_s": round(n / (t1 - t0), 1)},
        "bulk": {"requests": ss["requests_total"], "ms": round(bulk_ms, 4),
                 "rows_per_s": round(n / (bulk_ms * 1e-3), 1)},
        "speedup": round((t1 - t0) / (bulk_ms * 1e-3), 1)}
    log(json.dumps(res["requests"]))
    del dst, sub_cache, sub_slot

    # -- rows per wavefront copy step ---------------------------------------
    def tile_rows(max_bytes):          # staging: a power of two
        t = 64
        while t > 1 and t * rb > max_bytes:
            t //= 2
        return t

    def fill_rows(max_bytes):          # gather: as many rows as fit
        return max(1, min(64, max_bytes // rb))

    # the sequential driver's gather (eight loads, power-of-two tiles); the
    # look-ahead's shared gather fills its tiles (fill_rows), swept as well
    defaults = {"gather": tile_rows(8192), "stage": tile_rows(32768)}
    ref_out, ref_cache, tiles = None, None, []
    try:
        for t in sorted({64, 16, 4, 1, fill_rows(8192), *defaults.values()}, reverse=True):
            pipe.tuning = gg.make_tuning(tile_rows=t)
            gm = timed(lambda: pipe.gather_window(Wk), 10)
            sm = timed(stage_full, 10)
            out = pipe.win_out[:g_rows, :rb]
            if ref_out is None:
                ref_out, ref_cache = out.clone(), cache[:H, :rb].clone()
            elif not (torch.equal(out, ref_out) and torch.equal(cache[:H, :rb], ref_cache)):
                raise RuntimeError(f"rows differ with {t} rows per wave step")
            tiles.append({"rows_per_wave_step": t,
                          "default_for": [k for k, v in defaults.items() if v == t],
                          "gather_ms": round(gm, 4),
                          "gather_GBps": round(g_bytes / (gm * 1e-3) / 1e9, 1),
                          "stage_ms": round(sm, 4),
                          "stage_GBps": round(s_bytes / (sm * 1e-3) / 1e9, 1)})
            log(json.dumps(tiles[-1]))
    finally:
        pipe.tuning = None
    res["tile"] = tiles
    del ref_out, ref_cache

    # -- host shards: zero-copy against pack + DMA --------------------------
    host = [m for m in range(P) if not shards_d[m].is_cuda]
    if host:
        zc_ms = timed(stage_full, 5)
        full_own = np.searchsorted(off_h, np.arange(H), side="right") - 1
        u_all = bucket[:H].cpu().numpy().astype(np.int64)
        r_all = u_all - np.asarray(inst.range_start, dtype=np.int64)[full_own] \
            if wl.part_kind == synth.PART_RANGE else u_all // P
        host_rows = int(sum(off_h[m + 1] - off_h[m] for m in host))
        pack = torch.empty((max(host_rows, 1), stride), dtype=torch.uint8, pin_memory=True)
        dma = torch.empty((max(host_rows, 1), stride), dtype=torch.uint8, device=dev)
        idx = {m: torch.from_numpy(r_all[off_h[m]:off_h[m + 1]]) for m in host}
        best = None
        for _ in range(3):
            t0 = time.perf_counter()
            o = 0
            for m in host:
                k = len(idx[m])
                torch.index_select(shards_d[m], 0, idx[m], out=pack[o:o + k])
                o += k
            t_pack = time.perf_counter() - t0
            e0, e1 = mk(), mk()
            e0.record()
            o = 0
            for m in host:
                k = len(idx[m])
                dma[o:o + k].copy_(pack[o:o + k], non_blocking=True)
                o += k
            e1.record()
            torch.cuda.synchronize()
            t_all = time.perf_counter() - t0
            r = (t_all, t_pack, e0.elapsed_time(e1))
            best = r if best is None or r[0] < best[0] else best
        o = 0
        for m in host:
            k = len(idx[m])
            if not torch.equal(dma[o:o + k, :rb], cache[off_h[m]:off_h[m] + k, :rb]):
                raise RuntimeError(f"packed rows of owner {m} differ from the staged cache")
            o += k
        res["host_staging"] = {
            "host_rows": host_rows, "owners": host, "pack_threads": torch.get_num_threads(),
            "zero_copy_stage_ms": round(zc_ms, 3),
            "zero_copy_note": "the whole staging call, device-resident owners included",
            "pack_ms": round(best[1] * 1e3, 3), "dma_ms": round(best[2], 3),
            "pack_dma_ms": round(best[0] * 1e3, 3),
            "dma_GBps": round(host_rows * stride / (best[2] * 1e-3) / 1e9, 1)}
        log(json.dumps(res["host_staging"]))
        del pack, dma
    print(json.dumps({"ablation": args.config, "W": W, "window_rows": g_rows, "hot_set": H,
                      **res}), flush=True)


def graph_mode(args, wl):
    """The sequential driver (full restage, whole-window gather) launched call
    by call against the same windows replayed from HIP graphs captured once
    per window; one JSON line.  Every window's gathered rows from a replay
    are compared byte for byte with the eager run's."""
    import numpy as np
    import torch

    import synth
    from paper_2606_02916_amd import FetchPipeline

    dev = torch.device("cuda:0")
    inst, row_ptr_d, col_idx_d, shards_d = synth.torch_instance(args.config, dev)
    W = args.W or wl.W
    L, rb = len(wl.fanout), wl.row_bytes
    pipe = FetchPipeline(row_ptr_d, col_idx_d, wl.num_parts, wl.part_kind, wl.local_owner,
                         inst.range_start, shards_d, [s.shape[0] for s in inst.shards], rb,
                         wl.row_stride, W, wl.fanout, wl.batch_size, device=dev)
    boff = inst.batch_off
    nwin = synth.n_windows(boff, W)
    wins = []
    for k in range(nwin):
        b0, b1 = synth.window_batches(boff, W, k)
        s = torch.from_numpy(inst.seeds[boff[b0]:boff[b1]].copy()).to(dev)
        wins.append((s, boff[b0:b1 + 1] - boff[b0], b0))
    graphs = [pipe.capture_window(s, so, b0) for s, so, b0 in wins]
    torch.cuda.synchronize()

    def rows_now(Wk):
        fo = pipe.frontier_off[:(L + 1) * Wk + 1].cpu().numpy()
        return int(fo[-1] - fo[L * Wk])

    nrows, same = [], True
    for k, (s, so, b0) in enumerate(wins):
        pipe.reset_cache()
        Wk = pipe.window(s, so, b0)
        torch.cuda.synchronize()
        n = rows_now(Wk)
        ref = pipe.win_out[:n, :rb].clone()
        graphs[k][0].replay()
        torch.cuda.synchronize()
        same = same and rows_now(Wk) == n and bool(torch.equal(pipe.win_out[:n, :rb], ref))
        nrows.append(n)
        del ref
    if pipe.read_status() != 0 or not same:
        raise RuntimeError("graph replays differ from the eager windows")
    K = args.steps
    order = [i % nwin for i in range(K)]

    def timed(fn):
        for k in order[:nwin]:
            fn(k)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in order:
            fn(k)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / K * 1e3

    def eager(k):
        s, so, b0 = wins[k]
        pipe.reset_cache()
        pipe.window(s, so, b0)

    e_ms = timed(eager)
    g_ms = timed(lambda k: graphs[k][0].replay())
    rows = sum(nrows[k] for k in order) / K
    print(json.dumps({"graph": args.config, "W": W, "windows": nwin, "steps": K,
                      "rows_per_window": round(rows, 1),
                      "eager_ms_per_window": round(e_ms, 4),
                      "graph_ms_per_window": round(g_ms, 4),
                      "speedup": round(e_ms / g_ms, 3),
                      "graph_rows_per_s": round(rows / (g_ms * 1e-3), 1),
                      "replays_equal_eager": same}), flush=True)


def wsweep(args, wl):
    """One epoch per window size W on the same graph, seeds and features:
    counts and a timed epoch with the sequential driver (full restage), then
    the same windows timed through the look-ahead driver."""
    import numpy as np
    import torch

    import synth
    from paper_2606_02916_amd import FetchPipeline
    dev = torch.device("cuda:0")
    inst, row_ptr_d, col_idx_d, shards_d = synth.torch_instance(args.config, dev)
    P, rb = wl.num_parts, wl.row_bytes
    seeds_d = torch.from_numpy(inst.seeds).to(dev)
    boff = inst.batch_off
    results = []
    for W in [int(x) for x in args.wsweep.split(",")]:
        pipe = FetchPipeline(row_ptr_d, col_idx_d, P, wl.part_kind, wl.local_owner,
                             inst.range_start, shards_d, [s.shape[0] for s in inst.shards], rb,
                             wl.row_stride, W, wl.fanout, wl.batch_size, device=dev)
        nwin = synth.n_windows(boff, W)
        wins = []
        for k in range(nwin):
            b0, b1 = synth.window_batches(boff, W, k)
            wins.append((seeds_d[boff[b0]:boff[b1]], boff[b0:b1 + 1] - boff[b0], b0))
        # untimed pass: counts; then one timed epoch
        hot, delta, owner_bytes, rows, remote, gbytes, requests = [], [], [], [], [], [], []
        for s, so, b0 in wins:
            Wk = pipe.window(s, so, b0)
            torch.cuda.synchronize()
            if pipe.read_status() != 0:
                raise RuntimeError(f"device status {pipe.read_status()} at W={W}")
            st = pipe.stage_stats_dict()
            g = [pipe.gather_stats_dict(b) for b in range(Wk)]
            hot.append(st["rows_total"])
            delta.append(sum(st["delta_rows"]))
            owner_bytes.append(st["bytes"])
            requests.append(st["requests_total"])
            rows.append(sum(x["rows"] for x in g))
            remote.append(sum(x["hits"] + x["misses"] for x in g))
            gbytes.append(sum(x["rows"] * (2 * rb + 4) + (x["hits"] + x["misses"]) * 4 for x in g))
        pipe.reset_cache()
        mk = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
        gev = [(mk(), mk()) for _ in wins]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for (s, so, b0), ge in zip(wins, gev):
            pipe.window(s, so, b0, gather_events=[ge])
        torch.cuda.synchronize()
        el = time.perf_counter() - t0
        g_ms = sum(a.elapsed_time(b) for a, b in gev)
        del pipe
        torch.cuda.empty_cache()
        r = {"W": W, "windows": nwin, "hot_set_rows_per_window": float(np.mean(hot)),
             "bulk_bytes_per_owner_per_window": [float(x) for x in np.mean(owner_bytes, axis=0)],
             "bulk_requests_per_epoch": int(sum(requests)),
             "delta_rows_per_window": float(np.mean(delta)),
             "rows_gathered_per_epoch": int(sum(rows)),
             "reuse_factor": round(sum(remote) / max(1, sum(hot)), 3),
             "epoch_ms": round(el * 1e3, 3), "rows_per_s": round(sum(rows) / el, 1),
             "gather_GBps": round(sum(gbytes) / (g_ms * 1e-3) / 1e9, 1)}
        log(json.dumps(r))
        results.append(r)
    # the same windows through the look-ahead driver (persistent cache), as
    # the default line's sweep measures them (it uploads its own copy)
    del row_ptr_d, col_idx_d, shards_d, seeds_d
    torch.cuda.empty_cache()
    for r, la in zip(results, wsweep_lookahead(dev, args.config, [r["W"] for r in results],
                                               parse_tuning(args.tune))):
        assert la["W"] == r["W"]
        r["lookahead_ms_per_window"] = la["ms_per_window"]
        r["lookahead_rows_per_s"] = la["rows_per_s"]
        r["lookahead_gather_GBps"] = la["gather_GBps"]
        r["lookahead_gpu_ms_per_window"] = la["gpu_ms_per_window"]
        r["lookahead_host_enqueue_ms_per_window"] = la["host_enqueue_ms_per_window"]
        r["lookahead_queued"] = la["queued"]
    pick = next((r for r in results if r["W"] == wl.W), results[-1])
    line = {"metric": "feature rows gathered/s vs W (per-window fetch path)",
            "value": pick["rows_per_s"], "unit": "rows/s", "n_gpus": 1,
            "steps": pick["windows"], "warmup": 1, "ms_per_step": round(pick["epoch_ms"] /
                                                                      pick["windows"], 4),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u8",
            "data": "synthetic R-MAT (a,b,c)=(0.57,0.19,0.19), seeded; features as opaque bytes",
            "config": {"workload": args.config, "nodes": wl.num_nodes, "edges": wl.num_edges,
                       "features": f"{wl.feat_dtype}x{wl.feat_dim}", "fanout": list(wl.fanout),
                       "batch": wl.batch_size, "W_reported": pick["W"]},
            "w_sweep": results}
    if args.wsweep_table:
        write_wsweep_table(args, wl, results)
    print(json.dumps(line), flush=True)


def write_wsweep_table(args, wl, results):
    """The --wsweep results as a text table (the sweep's profile summary)."""
    batches = results[0]["windows"] * results[0]["W"]
    lines = [
        f"# command: python3 bench.py --config {args.config} --wsweep {args.wsweep} "
        f"--wsweep-table <file> (env SYNTH_CACHE_DIR=/tmp/synth_cache), one MI355X",
        f"# {wl.num_nodes / 1e6:.2f}M-node / {wl.num_edges / 1e6:.0f}M-edge R-MAT, "
        f"{wl.feat_dtype}x{wl.feat_dim} rows, fanout {list(wl.fanout)}, batch {wl.batch_size}, "
        f"about {batches} batches per epoch",
        "# columns 3-10: sequential driver (full restage of the hot set every window), one "
        "timed epoch after an untimed one",
        "# look: the look-ahead driver (persistent cache, delta staging) over the same windows, "
        "epoch cycled 4 times after an untimed epoch",
        "# look GPU ms/win: mean period over whole epochs of windows enqueued behind a blocker "
        "(the GPU's own rate); host ms/win: the host's enqueue per window in that run",
        "  W windows hot rows/win  delta/win bulk req/epoch  reuse  epoch ms       rows/s "
        "gather GB/s | look ms/win  look rows/s look gather GB/s look GPU ms/win host ms/win",
    ]
    for r in results:
        lines.append(
            f"{r['W']:3d} {r['windows']:7d} {r['hot_set_rows_per_window']:12.0f} "
            f"{r['delta_rows_per_window']:10.0f} {r['bulk_requests_per_epoch']:14d} "
            f"{r['reuse_factor']:6.2f} {r['epoch_ms']:9.3f} {r['rows_per_s']:12.4g} "
            f"{r['gather_GBps']:11.1f} | {r['lookahead_ms_per_window']:11.4f} "
            f"{r['lookahead_rows_per_s']:12.4g} {r['lookahead_gather_GBps']:16.1f} "
            f"{r['lookahead_gpu_ms_per_window']:15.4f}{'' if r['lookahead_queued'] else '*'} "
            f"{r['lookahead_host_enqueue_ms_per_window']:11.4f}")
    if not all(r["lookahead_queued"] for r in results):
        lines.append("# *: the GPU reached the third queued window before the host had "
                     "enqueued them all (not a clean GPU-only period)")
    lines.append("# bulk bytes per owner per window, sequential driver (full restage; owners "
                 f"0..{wl.num_parts - 1}, owner {wl.local_owner} local):")
    for r in results:
        lines.append(f"#  W={r['W']:2d}: " + ", ".join(
            f"{x / 1e6:.1f} MB" for x in r["bulk_bytes_per_owner_per_window"]))
    with open(args.wsweep_table, "w") as f:
        f.write("\n".join(lines) + "\n")


def wsweep_lookahead(dev, name, Ws, tuning=None, reps=4):
    """The W sweep as the default bench reports it: for each W, one epoch of
    the workload `name` through the look-ahead driver (the benchmarked
    configuration), after one untimed epoch, cycled `reps` times (at least
    8 windows).  Per W: rows gathered/s over the timed windows, the
    gather's rate from HIP events (the same method as the main line: a
    gather ends at its end event and started at the later of its window's
    staging end and the previous gather's end), and the epoch's counts from
    the untimed pass: hot-set rows, bulk bytes per owner and rebuild-delta
    rows per window, bulk requests per epoch and the reuse factor."""
    import numpy as np
    import torch

    import synth
    from paper_2606_02916_amd import LookaheadPipeline
    wl = synth.WORKLOADS[name]
    inst, row_ptr_d, col_idx_d, shards_d = synth.torch_instance(name, dev)
    P, rb = wl.num_parts, wl.row_bytes
    seeds_d = torch.from_numpy(inst.seeds).to(dev)
    boff = inst.batch_off
    mk = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    out = []
    look = None
    for W in Ws:
        t_w = time.perf_counter()
        # the previous W's buffers go back to the device before this W's
        # are allocated (at W = 32 one set's output alone is about 31 GB)
        look = None
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        look = LookaheadPipeline(row_ptr_d, col_idx_d, P, wl.part_kind, wl.local_owner,
                                 inst.range_start, shards_d, [s.shape[0] for s in inst.shards],
                                 rb, wl.row_stride, W, wl.fanout, wl.batch_size, device=dev,
                                 tuning=tuning)
        nwin = synth.n_windows(boff, W)
        wins = []
        for k in range(nwin):
            b0, b1 = synth.window_batches(boff, W, k)
            wins.append((seeds_d[boff[b0]:boff[b1]], boff[b0:b1 + 1] - boff[b0], b0))
        hot, delta, owner_bytes, requests, rows, remote, gbytes = [], [], [], [], [], [], []
        for s_, so, b0 in wins:          # untimed epoch: counts
            Wk, bufs = look.window(s_, so, b0)
            look.synchronize()
            st = bufs.stage_stats_dict()
            g = [bufs.gather_stats_dict(b) for b in range(Wk)]
            hot.append(st["rows_total"])
            delta.append(sum(st["delta_rows"]))
            owner_bytes.append(st["bytes"])
            requests.append(st["requests_total"])
            rows.append(sum(x["rows"] for x in g))
            remote.append(sum(x["hits"] + x["misses"] for x in g))
            gbytes.append(sum(x["rows"] * (2 * rb + 4) + (x["hits"] + x["misses"]) * 4
                              for x in g))
        for i in range(nwin, look.nsets):
            # every buffer set runs once before the timed windows (its
            # output is allocated on first use)
            look.window(*wins[i % nwin])
        if look.read_status() != 0:
            raise RuntimeError(f"device status {look.read_status()} at W={W}")
        K = max(reps * nwin, 8)
        order = [i % nwin for i in range(K)]
        sev = [mk() for _ in range(K)]
        gev = [mk() for _ in range(K)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i, k in enumerate(order):
            s_, so, b0 = wins[k]
            look.window(s_, so, b0, events=[None, None, None, None, sev[i]],
                        gather_events=(None, gev[i]))
        look.synchronize()
        el = time.perf_counter() - t0
        if look.read_status() != 0:
            raise RuntimeError(f"device status {look.read_status()} at W={W}")
        g_ms = 0.0
        for i in range(K):
            t = sev[i].elapsed_time(gev[i])
            if i > 0:
                t = min(t, gev[i - 1].elapsed_time(gev[i]))
            g_ms += t
        g_bytes = sum(gbytes[k] for k in order)
        g_gbs = g_bytes / (g_ms * 1e-3) / 1e9
        # The GPU's own period: the same windows enqueued behind a blocker on
        # the caller's stream (every window waits on that stream, as in the
        # timed run), so the GPU runs them back to back whatever the host's
        # enqueue rate (about 0.15-0.2 ms per window; the blocker lasts
        # longer than the whole enqueue).  The period is the mean over whole
        # epochs from the third window on (an epoch's windows may differ in
        # size).
        Kq = 3 + nwin * max(1, 37 // nwin)
        qev = [mk() for _ in range(Kq)]
        blocker = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
        torch.cuda.synchronize()
        for i in range(Kq * 3):          # ~0.1 ms of GPU time per fill
            blocker.fill_(i & 0xFF)
        t1 = time.perf_counter()
        for i in range(Kq):
            s_, so, b0 = wins[i % nwin]
            look.window(s_, so, b0, gather_events=(None, qev[i]))
        host_q = (time.perf_counter() - t1) / Kq
        queued = not qev[2].query()
        look.synchronize()
        del blocker
        q_ms = qev[2].elapsed_time(qev[Kq - 1]) / (Kq - 3)
        r = {"W": W, "windows_per_epoch": nwin,
             "rows_per_s": round(sum(rows[k] for k in order) / el, 1),
             "ms_per_window": round(el / K * 1e3, 4),
             "gather_GBps": round(g_gbs, 1), "gather_frac": round(g_gbs / HBM_PEAK_GBS, 4),
             "hot_set_rows_per_window": round(float(np.mean(hot)), 1),
             "bulk_bytes_per_owner_per_window": [round(float(x), 1)
                                                 for x in np.mean(owner_bytes, axis=0)],
             "delta_rows_per_window": round(float(np.mean(delta)), 1),
             "bulk_requests_per_epoch": int(sum(requests)),
             "reuse_factor": round(sum(remote) / max(1, sum(hot)), 3),
             "gpu_ms_per_window": round(q_ms, 4),
             "host_enqueue_ms_per_window": round(host_q * 1e3, 4), "queued": queued,
             "wall_s": None}
        del look
        torch.cuda.empty_cache()
        r["wall_s"] = round(time.perf_counter() - t_w, 2)
        log(f"wsweep W={W}: " + json.dumps(r))
        out.append(r)
    return out


def sim_coefficients(wl):
    """Synthetic coefficients of the analytical energy model, the same for
    every owner: a 500 us request initiation at 50 W, rows at 1.25 GB/s
    (one 10 GbE link) at 50 W, a 1.25 GB/s aggregate ceiling and 30 W idle
    power.  A one-row request is then almost all initiation and a request
    of about 1,500 rows of 400 B is half initiation."""
    link = 1.25e9
    lam_init, lam_row = 500e-6, wl.row_bytes / link
    return dict(eps_init=50.0 * lam_init, eps_row=50.0 * lam_row, lam_init=lam_init,
                lam_row=lam_row, bw_bytes_per_s=link, row_bytes=wl.row_bytes, p_idle=30.0)


def simulate(args, wl):
    """The window-size simulator on the GPU: one epoch per (budget, W)
    through the fetch path, the per-window rebuild-delta and miss counters
    priced into z(W) and E_phy(W) on the device."""
    import numpy as np
    import torch

    import synth
    from paper_2606_02916_amd import FetchPipeline, gg
    dev = torch.device("cuda:0")
    inst, row_ptr_d, col_idx_d, shards_d = synth.torch_instance(args.config, dev)
    P, rb = wl.num_parts, wl.row_bytes
    seeds_d = torch.from_numpy(inst.seeds).to(dev)
    boff = inst.batch_off
    cd = sim_coefficients(wl)
    coeffs = gg.make_sim_coeffs(P, **cd)
    results = []
    if args.hot_frac:
        budgets = [(-1, tuple(int(v) for v in f.split("/"))) for f in args.hot_frac.split(",")]
    else:
        budgets = [(int(x), None) for x in args.n_hot.split(",")]
    for n_hot, frac in budgets:
        for W in [int(x) for x in args.simulate.split(",")]:
            pipe = FetchPipeline(row_ptr_d, col_idx_d, P, wl.part_kind, wl.local_owner,
                                 inst.range_start, shards_d, [s.shape[0] for s in inst.shards],
                                 rb, wl.row_stride, W, wl.fanout, wl.batch_size, n_hot=n_hot,
                                 device=dev, delta=True, hot_frac=frac)
            nwin = synth.n_windows(boff, W)
            wins = []
            for k in range(nwin):
                b0, b1 = synth.window_batches(boff, W, k)
                wins.append((seeds_d[boff[b0]:boff[b1]], boff[b0:b1 + 1] - boff[b0], b0))
            acc = torch.zeros(gg.SIM_ACC_BYTES, dtype=torch.uint8, device=dev)
            for s, so, b0 in wins:                       # warm-up epoch
                pipe.window(s, so, b0)
            pipe.reset_cache()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for s, so, b0 in wins:
                pipe.window(s, so, b0, sim=(coeffs, acc))
            torch.cuda.synchronize()
            el = time.perf_counter() - t0
            if pipe.read_status() != 0:
                raise RuntimeError(f"device status {pipe.read_status()} at W={W}")
            a = gg.sim_acc_from_bytes(acc.cpu().numpy().tobytes())
            r = {"n_hot": n_hot if frac is None else f"{frac[0]}/{frac[1]} of each window",
                 "W": W, "windows": a["windows"],
                 "z": {"rebuild_events": a["rebuild_events"], "miss_events": a["miss_events"],
                       "t_stall_s": a["t_stall"],
                       "hit_ratio": a["hits"] / a["remote_rows"] if a["remote_rows"] else 1.0},
                 "rebuild_rows": a["rebuild_rows"], "miss_rows": a["miss_rows"],
                 "remote_requests": a["remote_rows"],
                 "E_rebuild_J": a["e_rebuild"], "E_miss_J": a["e_miss"],
                 "E_stall_J": a["e_stall"], "E_phy_J": a["e_phy"],
                 "epoch_ms": round(el * 1e3, 3)}
            log(json.dumps(r))
            results.append(r)
            del pipe
            torch.cuda.empty_cache()
    best = {}
    for r in results:
        if r["n_hot"] not in best or r["E_phy_J"] < best[r["n_hot"]]["E_phy_J"]:
            best[r["n_hot"]] = r
    line = {"metric": "window-size simulator: z(W) and E_phy(W) per candidate W",
            "value": round(sum(r["epoch_ms"] for r in results), 3), "unit": "ms (whole sweep)",
            "n_gpus": 1, "higher_is_better": False, "dtype": "int64+f64",
            "data": "synthetic R-MAT (a,b,c)=(0.57,0.19,0.19), seeded; synthetic cost coefficients",
            "config": {"workload": args.config, "nodes": wl.num_nodes, "edges": wl.num_edges,
                       "fanout": list(wl.fanout), "batch": wl.batch_size,
                       "coefficients": cd},
            "W_star": {str(k): v["W"] for k, v in best.items()},
            "sweep": results}
    print(json.dumps(line), flush=True)


def cpu_baseline(inst, wl, W, so, b0, min_seconds):
    """The CPU oracle, untuned and single-threaded, on window 0 of the same
    workload; repeated until at least min_seconds of work when one window is
    shorter than that.  The calling thread (the oracle runs no threads of its
    own) is pinned to one core for the duration, and each step of the path
    is timed on its own."""
    import numpy as np

    from oracle import ggref
    P = wl.num_parts
    part = ggref.make_part(P, wl.part_kind, wl.local_owner, wl.num_nodes, inst.range_start)
    feat = ggref.make_feat(wl.row_bytes, inst.shards, [wl.row_stride] * P)
    boff = inst.batch_off
    seeds = inst.seeds[boff[b0]:boff[b0 + len(so) - 1]]
    slot_of = np.full(wl.num_nodes, -1, dtype=np.int32)
    cache = None
    reps, rows = 0, 0
    steps = {"sample": 0.0, "hotset": 0.0, "bucket": 0.0, "stage": 0.0, "gather": 0.0}
    affinity = os.sched_getaffinity(0)
    core = max(affinity)
    os.sched_setaffinity(0, {core})
    try:
        while True:
            Wk, L = len(so) - 1, len(wl.fanout)
            t0 = time.perf_counter()
            fids, foff, nids, noff = ggref.sample_window(inst.row_ptr, inst.col_idx, seeds, so,
                                                         wl.fanout, 0, 0, b0)
            t1 = time.perf_counter()
            hot, freq = ggref.build_hotset(fids, foff, Wk, L, part, -1)
            t2 = time.perf_counter()
            bucket, owner_off = ggref.bucket_by_owner(hot, part)
            t3 = time.perf_counter()
            steps["sample"] += t1 - t0
            steps["hotset"] += t2 - t1
            steps["bucket"] += t3 - t2
            if cache is None or cache.shape[0] < len(hot):              # not timed
                cache = np.zeros((len(hot), wl.row_stride), dtype=np.uint8)
            slot_of.fill(-1)
            t0 = time.perf_counter()
            ggref.stage_bulk(bucket, owner_off, part, feat, cache, wl.row_stride, slot_of, None)
            steps["stage"] += time.perf_counter() - t0
            for b in range(Wk):
                s = L * Wk + b
                ids = fids[foff[s]:foff[s + 1]]
                out = np.empty((len(ids), wl.row_stride), dtype=np.uint8)  # not timed
                t0 = time.perf_counter()
                ggref.gather_batch(ids, part, feat, cache, wl.row_stride, slot_of, out,
                                   wl.row_stride)
                steps["gather"] += time.perf_counter() - t0
                rows += len(ids)
            reps += 1
            if sum(steps.values()) >= min_seconds or reps >= 1000:
                break
    finally:
        os.sched_setaffinity(0, affinity)
    total = sum(steps.values())
    log(f"cpu oracle: {reps} window(s), {rows} rows in {total:.1f}s on core {core}")
    return {"value": round(rows / total, 1), "unit": "rows/s", "cores": 1, "kind": "oracle",
            "sample": f"{reps} x window 0 of {wl.name} (W={len(so) - 1}, {rows // reps} rows per "
                      f"window), single-threaded C++ oracle pinned to one core, excluding input "
                      f"generation and buffer allocation",
            "seconds_per_window": {k: round(v / reps, 4) for k, v in steps.items()},
            "host_cpu": cpu_model(), "host_nproc": os.cpu_count(), "pinned_core": core}


if __name__ == "__main__":
    main()
