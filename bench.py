"""Benchmark of the error-feedback compression step on one MI355X.

Workload (default, the largest one-GPU configuration): d = 1,500,000,000
fp32 elements, Gaussian g with std 1e-3 except a fixed seeded 5 % of
coordinates at std 0.1 (sparse large outliers), lr = 0.1, e carried from
step to step; hard threshold at the lambda that keeps 0.1 % at the first
step, Top-k with k = 1,500,000.  Gradients rotate through a pool of two
(12 GB, far beyond the 256 MB Infinity Cache), resident in HBM before any
timing.

Timed regions (HIP events at their two ends only, on the stream the
kernels run on; a barrier and a device synchronisation on both sides):
  * `value`: K error-feedback steps of the hard threshold (ht_compress,
    one launch of ht_fused_kernel per step); value = d / (time per step),
    G grad-elements/s; ms_per_step is that time.  `ht_steps` holds the
    p10 / p50 / p90 of the same steps replayed one call at a time, and
    `ht_cold` five further calls each after a 1 GiB write that evicts the
    caches.
  * `topk`: K steps of the Top-k baseline (topk_compress, its own error
    vector and workspace) on the same gradients.
  * `average`: K exchange-and-average calls (sparse_accumulate) of the
    eight-worker 25,557,032-element workload's first-step hard-threshold
    payloads, the output rotating over four buffers.
Each reports its rate against the HBM roofline (8 TB/s) on the algorithmic
bytes: 12 d + 8 k_t for the hard threshold, 12 d + 8 k for Top-k (the
information it must move), 4 d + 8 (sum of counts) for the average.

`roofline` is the hard-threshold kernel on the default workload: the
algorithmic bytes per launch over its launch duration (the timed steps are
back-to-back launches of that kernel alone).  `traffic` is the HBM bytes
per launch from two rocprofv3 --pmc runs of this script (FETCH_SIZE, then
WRITE_SIZE), each scaled by what the same counter reads for the copy probe
moving a known 8 d bytes in the same run; null when the summary was taken
from other kernel sources.  `cpu_baseline` is the CPU oracle on the same
workload (its multi-core build on all host cores; `cpu_baseline_1core` the
single-threaded build).  `extra` holds the 25,557,032-element workload's
figures and the fused model updates.
"""
import argparse
import csv
import glob
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
HT_KERNEL = "ht_fused_kernel"
HT_PLAIN = HT_KERNEL + "<true, false>"
COPY_KERNEL = "copy_kernel"
HT_SOURCES = ["ht.hip", "device_common.hpp"]
T0 = time.time()


def say(*a):
    print("[bench %6.1fs]" % (time.time() - T0), *a, file=sys.stderr, flush=True)


def traffic_file(name):
    return os.path.join(ROOT, "profiles", "ht_fused_kernel_%s_pmc.txt" % name)


def kernel_source_digest():
    """sha256 over the sources that determine the hard-threshold kernel."""
    import hashlib
    h = hashlib.sha256()
    for name in HT_SOURCES:
        with open(os.path.join(ROOT, "paper_2108_00951_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def read_traffic(path):
    """Counter-derived bytes per launch, or None when the file is absent or
    was taken from a different version of the kernel sources."""
    if not path or not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            parts = line.split()
            if len(parts) == 2 and not line.startswith("#"):
                fields[parts[0]] = parts[1]
    if fields.get("kernel_source_sha256") != kernel_source_digest():
        return None
    return int(float(fields["ht_bytes_per_launch"]))


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20, help="timed steps (the workload runs 20)")
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=5, choices=(2, 3, 5),
                    help="workload of the hard-threshold and Top-k timings: 5 = 1.5e9 outliers "
                         "(default), 2 = 25,557,032 segments, 3 = 110e6 Student-t")
    ap.add_argument("--pool", type=int, default=None,
                    help="distinct gradients in the rotation (default: 2 for the 1.5e9 "
                         "workload, 4 for the others, always beyond the 256 MB Infinity Cache)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baselines")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the 25.6e6 workload's figures and the fused model updates")
    ap.add_argument("--parse-trace", metavar="TRACE_DIR",
                    help="print the kernel statistics of a rocprofv3 --kernel-trace --stats "
                         "run of this script, with the average over the timed run of "
                         "hard-threshold launches")
    ap.add_argument("--parse-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarise two rocprofv3 --pmc output folders and exit")
    ap.add_argument("--layerwise-only", action="store_true",
                    help="time only the 20,000-layer layer-wise Top-k and print its figures "
                         "(not the contract line)")
    ap.add_argument("--radix-only", action="store_true",
                    help="time only Top-k from a fresh workspace (the radix path) on the "
                         "workload's first gradient, as drawn and quantised to 2^-16 and 2^-10 "
                         "(ties at the threshold to split), and print its figures (not the "
                         "contract line)")
    ap.add_argument("--trace-last", type=int, metavar="N",
                    help="with --parse-trace: per-kernel statistics over each kernel's last N "
                         "dispatches only (the timed calls of a run that times N)")
    return ap.parse_args()


def _pmc_rows(folder, counter):
    """(kernel name, value) of every dispatch in a rocprofv3 counter CSV, in
    dispatch order."""
    rows = []
    for path in glob.glob(os.path.join(folder, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as f:
            for r in csv.DictReader(f):
                if r.get("Counter_Name") == counter:
                    rows.append((int(r.get("Dispatch_Id") or 0), r["Kernel_Name"],
                                 float(r["Counter_Value"])))
    rows.sort()
    return [(k, v) for _, k, v in rows]


def parse_pmc(fetch_dir, write_dir, d, ht_launches):
    """HBM bytes per launch of the hard-threshold kernel, scaled by the copy probe.

    FETCH_SIZE and WRITE_SIZE are in KiB per dispatch.  The copy probe moves
    exactly 4n bytes in and 4n bytes out (n = d); the ratio of those bytes to
    what the counters report for it is the scale applied to the kernel.  The
    kernel's figure averages its first `ht_launches` dispatches: the
    hard-threshold phase on the workload (warm-up, timed steps, and the same
    steps again for k_t); the average's payloads come from later, smaller
    launches of the same kernel."""
    out = {}
    for name, folder in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = _pmc_rows(folder, name)
        ht = [v for k, v in rows if HT_PLAIN in k][:ht_launches]
        cp = [v for k, v in rows if COPY_KERNEL in k]
        if not ht or not cp:
            raise SystemExit("no %s rows for %s / %s in %s" % (name, HT_PLAIN, COPY_KERNEL, folder))
        ht_b = 1024.0 * sum(ht) / len(ht)
        cp_b = 1024.0 * sum(cp) / len(cp)
        scale = 4.0 * d / cp_b
        out[name] = {"ht_kib_per_launch": ht_b / 1024, "copy_kib_per_launch": cp_b / 1024,
                     "copy_expected_kib": 4.0 * d / 1024, "scale": scale,
                     "ht_bytes_scaled": ht_b * scale, "launches": len(ht)}
        # every other kernel of the run, the same scale applied
        by = {}
        for k, v in rows:
            by.setdefault(_short_kernel_name(k), []).append(v)
        out[name]["kernels"] = {k: (1024.0 * sum(v) / len(v) * scale, len(v)) for k, v in by.items()}
    out["ht_bytes_per_launch"] = out["FETCH_SIZE"]["ht_bytes_scaled"] + out["WRITE_SIZE"]["ht_bytes_scaled"]
    return out


def _short_kernel_name(name):
    name = name.replace("efs::(anonymous namespace)::", "").replace("efs::", "")
    name = name.replace("void ", "")
    return re.sub(r"\(.*", "", name)[:34]


def parse_trace(folder, steps):
    """Per-kernel statistics of a rocprofv3 kernel trace, and the average of
    the first run of exactly `steps` consecutive dispatches of the
    hard-threshold kernel (its plain variant) that no other kernel
    interrupts: the timed steps, which the script delimits with other
    kernels."""
    stats = list(csv.DictReader(open(os.path.join(folder, "run_kernel_stats.csv"))))
    trace = list(csv.DictReader(open(os.path.join(folder, "run_kernel_trace.csv"))))
    trace.sort(key=lambda r: int(r["Start_Timestamp"]))
    total = sum(float(r["TotalDurationNs"]) for r in stats)
    lines = ["%-36s %6s %9s %9s %9s %7s" % ("kernel", "calls", "avg_us", "min_us", "max_us", "pct")]
    for r in sorted(stats, key=lambda r: -float(r["TotalDurationNs"])):
        if float(r["TotalDurationNs"]) / total < 0.0005:
            continue
        lines.append("%-36s %6s %9.2f %9.2f %9.2f %7.2f" % (
            _short_kernel_name(r["Name"]), r["Calls"], float(r["AverageNs"]) / 1e3,
            float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3,
            100 * float(r["TotalDurationNs"]) / total))
    runs, cur = [], []
    for r in trace:
        if HT_PLAIN in r["Kernel_Name"]:
            cur.append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
        else:
            if cur:
                runs.append(cur)
            cur = []
    if cur:
        runs.append(cur)
    timed = [x for x in runs if len(x) == steps]
    lines.append("")
    if timed:
        x = timed[0]
        lines.append("# %s, the %d timed steps: avg %.2f us, min %.2f, max %.2f"
                     % (HT_PLAIN, steps, sum(x) / len(x), min(x), max(x)))
    else:
        lines.append("# no run of %d back-to-back %s dispatches in the trace" % (steps, HT_PLAIN))
    return "\n".join(lines) + "\n"


def parse_trace_last(folder, n):
    """Per-kernel duration statistics of a rocprofv3 kernel trace over the
    last `n` dispatches of each kernel (every kernel of a run that ends with
    n timed calls)."""
    trace = list(csv.DictReader(open(os.path.join(folder, "run_kernel_trace.csv"))))
    trace.sort(key=lambda r: int(r["Start_Timestamp"]))
    by = {}
    for r in trace:
        us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        by.setdefault(_short_kernel_name(r["Kernel_Name"]), []).append(us)
    lines = ["%-36s %6s %9s %9s %9s" % ("kernel", "calls", "avg_us", "min_us", "max_us")]
    rows = []
    for name, xs in by.items():
        x = xs[-n:]
        rows.append((sum(x) / len(x), name, len(x), min(x), max(x)))
    for avg, name, cnt, lo, hi in sorted(rows, reverse=True):
        lines.append("%-36s %6d %9.2f %9.2f %9.2f" % (name, cnt, avg, lo, hi))
    return "\n".join(lines) + "\n"


def format_traffic(res, workload, args):
    lines = ["# HBM traffic of %s per launch from rocprofv3 counters, %s" % (HT_PLAIN, workload),
             "# (KiB per dispatch, averaged over the kernel's first %d dispatches, the"
             % (args.warmup + 2 * args.steps),
             "# hard-threshold phase with --warmup %d --steps %d; each counter scaled by"
             % (args.warmup, args.steps),
             "# expected/measured for %s moving 4*d bytes each way)" % COPY_KERNEL]
    for name in ("FETCH_SIZE", "WRITE_SIZE"):
        r = res[name]
        lines.append("# %s: kernel %.1f KiB, copy probe %.1f KiB (expected %.1f), scale %.5f, "
                     "%d launches" % (name, r["ht_kib_per_launch"], r["copy_kib_per_launch"],
                                      r["copy_expected_kib"], r["scale"], r["launches"]))
    fk, wk = res["FETCH_SIZE"].get("kernels", {}), res["WRITE_SIZE"].get("kernels", {})
    if fk or wk:
        lines.append("# every kernel of the run (all its dispatches, of any size), scaled the same "
                     "way: MB fetched + MB written per launch (launches)")
        names = sorted(set(fk) | set(wk),
                       key=lambda n: -(fk.get(n, (0.0, 0))[0] + wk.get(n, (0.0, 0))[0]))
        for n in names:
            f, nf = fk.get(n, (0.0, 0))
            w, nw = wk.get(n, (0.0, 0))
            lines.append("#   %-34s %9.2f + %9.2f MB  (%d)" % (n, f / 1e6, w / 1e6, max(nf, nw)))
    lines.append("ht_bytes_per_launch %d" % round(res["ht_bytes_per_launch"]))
    lines.append("kernel_source_sha256 %s" % kernel_source_digest())
    return "\n".join(lines) + "\n"


def stats_us(xs):
    import numpy as np
    a = np.sort(np.asarray(xs, dtype=np.float64))
    return {"mean_us": round(float(a.mean()), 2),
            "p10_us": round(float(a[int(0.1 * (a.size - 1))]), 2),
            "p50_us": round(float(np.median(a)), 2),
            "p90_us": round(float(a[int(0.9 * (a.size - 1))]), 2)}


def rate(nbytes, us):
    gbps = nbytes / (us * 1e-6) / 1e9
    return {"gbps": round(gbps, 1), "frac": round(gbps / HBM_PEAK_GBPS, 4)}


class Timer:
    """HIP events at the two ends of a region on one stream, with a device
    synchronisation on both sides."""

    def __init__(self, torch, stream):
        self.torch, self.stream = torch, stream

    def __enter__(self):
        self.a = self.torch.cuda.Event(enable_timing=True)
        self.b = self.torch.cuda.Event(enable_timing=True)
        self.torch.cuda.synchronize()
        self.a.record(self.stream)
        return self

    def __exit__(self, *exc):
        self.b.record(self.stream)
        self.torch.cuda.synchronize()
        self.us = self.a.elapsed_time(self.b) * 1e3


def to_device(torch, host, dev, chunk=1 << 26):
    out = torch.empty(host.size, dtype=torch.float32, device=dev)
    for lo in range(0, host.size, chunk):
        out[lo:lo + chunk].copy_(torch.from_numpy(host[lo:lo + chunk]))
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(got --gpus %d)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import numpy as np

    from paper_2108_00951_amd import synth

    wl = synth.WORKLOADS[args.workload]
    d, k, density = wl.d, wl.topk_k[0], wl.densities[0]
    if args.parse_pmc:
        res = parse_pmc(args.parse_pmc[0], args.parse_pmc[1], d, args.warmup + 2 * args.steps)
        sys.stdout.write(format_traffic(res, wl.name, args))
        return
    if args.parse_trace:
        if args.trace_last:
            sys.stdout.write(parse_trace_last(args.parse_trace, args.trace_last))
        else:
            sys.stdout.write(parse_trace(args.parse_trace, args.steps))
        return

    import torch

    from paper_2108_00951_amd import binding as efs

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    efs.load_library()
    cur = torch.cuda.current_stream()
    if args.layerwise_only:
        print(json.dumps(bench_many_layers(efs, torch, synth, cur)), flush=True)
        return
    if args.radix_only:
        print(json.dumps(bench_radix(efs, torch, synth, cur, wl, dev)), flush=True)
        return
    lr = synth.LR
    if args.pool is None:
        args.pool = 2 if d >= 100_000_000 else 4
    lam = synth.stored_lambda(wl.ident, density)
    stream = synth.Stream(wl.ident)
    threads = min(16, os.cpu_count() or 1)
    say("drawing %d gradients of %s (d=%d)" % (args.pool, wl.name, d))
    pool_host = [stream.gradient(t, threads=threads) for t in range(args.pool)]
    pool = [to_device(torch, g, dev) for g in pool_host]
    say("inputs resident: lambda=%r k=%d" % (float(lam), k))
    delimiter = torch.empty(4096, dtype=torch.float32, device=dev)

    def mark():
        # a short kernel of another name between phases, so that a kernel
        # trace shows the timed launches as one run
        efs.stream_probe(delimiter, delimiter, 2)

    # ---- hard threshold: K timed steps --------------------------------------
    e_ht = torch.zeros(d, dtype=torch.float32, device=dev)
    cap = d   # k_t grows under error feedback with a fixed lambda (past d/8 on heavy tails)
    idx = torch.empty(cap, dtype=torch.int32, device=dev)
    val = torch.empty(cap, dtype=torch.float32, device=dev)
    ctr = efs.new_counter(dev)
    for s in range(args.warmup):
        efs.ht_compress(pool[s % len(pool)], e_ht, lr, lam, idx, val, ctr)
    e_snap = e_ht.clone()
    mark()
    with Timer(torch, cur) as tm:
        for s in range(args.steps):
            efs.ht_compress(pool[(args.warmup + s) % len(pool)], e_ht, lr, lam, idx, val, ctr)
    mark()
    ht_us = tm.us / args.steps
    # k_t and the time of every timed step: the same calls again from the
    # same state, one at a time
    e_ht.copy_(e_snap)
    kts, ht_each = [], []
    for s in range(args.steps):
        with Timer(torch, cur) as t1:
            efs.ht_compress(pool[(args.warmup + s) % len(pool)], e_ht, lr, lam, idx, val, ctr)
        ht_each.append(t1.us)
        kts.append(efs.counter_value(ctr))
    if max(kts) > cap:
        raise RuntimeError("hard-threshold payload capacity exceeded")
    # cold calls: a 1 GiB write before each evicts the caches (the
    # trajectory continues from the replayed steps)
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    ht_cold = []
    for s in range(5):
        flush.fill_(float(s))
        with Timer(torch, cur) as t1:
            efs.ht_compress(pool[(args.warmup + s) % len(pool)], e_ht, lr, lam, idx, val, ctr)
        ht_cold.append(t1.us)
    del flush
    kt = float(np.mean(kts))
    ht_bytes = 12.0 * d + 8.0 * kt
    say("hard threshold: %.1f us per step, k_t %d..%d" % (ht_us, kts[0], kts[-1]))
    del e_snap, idx, val
    torch.cuda.empty_cache()

    # ---- Top-k: K timed steps on its own error vector -------------------------
    e_tk = torch.zeros(d, dtype=torch.float32, device=dev)
    tidx = torch.empty(k, dtype=torch.int32, device=dev)
    tval = torch.empty(k, dtype=torch.float32, device=dev)
    ws = efs.new_topk_workspace(d, k, dev)
    for s in range(args.warmup):
        efs.topk_compress(pool[s % len(pool)], e_tk, lr, k, tidx, tval, ws)
    # the error vector and the workspace (its threshold history) as the timed
    # steps found them, so that the replay below repeats those steps
    e_snap, ws_snap = e_tk.clone(), ws.clone()
    mark()
    with Timer(torch, cur) as tt:
        for s in range(args.steps):
            efs.topk_compress(pool[(args.warmup + s) % len(pool)], e_tk, lr, k, tidx, tval, ws)
    mark()
    tk_us = tt.us / args.steps
    # which selection each timed step took, and its time alone
    e_tk.copy_(e_snap)
    ws.copy_(ws_snap)
    paths, tk_each = [], []
    for s in range(args.steps):
        with Timer(torch, cur) as t1:
            efs.topk_compress(pool[(args.warmup + s) % len(pool)], e_tk, lr, k, tidx, tval, ws)
        tk_each.append(t1.us)
        paths.append(efs.topk_took_bracket_path(ws))
    tk_ideal = 12.0 * d + 8.0 * k
    say("Top-k: %.1f us per step, bracket path in %d of %d" % (tk_us, sum(paths), len(paths)))
    del e_snap, ws_snap, e_tk, tidx, tval, ws
    torch.cuda.empty_cache()

    # copy probe over d elements (also the scale of the traffic counters)
    with Timer(torch, cur) as tc:
        for s in range(3):
            efs.copy_probe(pool[s % len(pool)], pool[(s + 1) % len(pool)])
    copy_us = tc.us / 3
    ceiling = stream_ceiling(efs, torch, cur, pool, d)
    ceiling["ht_frac_over_best_2r1w"] = round(
        ht_bytes / (ht_us * 1e-6) / 1e9 / HBM_PEAK_GBPS / ceiling["best_2r1w_frac"], 3)
    del pool
    torch.cuda.empty_cache()

    # ---- exchange-and-average: eight workers' first-step payloads -------------
    average = bench_average(efs, torch, synth, cur, args.steps, args.warmup, threads)

    line = {
        "metric": "G grad-elements/s compressed (hard-threshold, Top-k) + achieved HBM GB/s",
        "value": round(d / (ht_us * 1e-6) / 1e9, 2),
        "unit": "G grad-elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ht_us / 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "%s: d=%s fp32, %s, lr=0.1, e carried; hard threshold at lambda=%.6g "
                        "(0.1%% first-step density), error-feedback steps; Top-k k=%s and the "
                        "8-worker average of the 25,557,032-element workload timed alongside"
                        % (wl.name, format(d, ","), describe(wl), float(lam), format(k, ",")),
            "d": d, "k": k, "lambda": float(lam), "lr": float(lr), "pool": args.pool,
            "step": "one hard-threshold error-feedback iteration (ht_compress)",
        },
        "hbm_gbps": round(ht_bytes / (ht_us * 1e-6) / 1e9, 1),
        "ht_steps": dict(stats_us(ht_each), note="each timed step replayed alone, synchronised "
                         "on both sides"),
        "ht_cold": dict(stats_us(ht_cold), calls=len(ht_cold),
                        note="one call after a 1 GiB write that evicts the caches"),
        "roofline": dict(
            kernel=HT_PLAIN, bound="hbm",
            achieved=round(ht_bytes / (ht_us * 1e-6) / 1e9, 1), peak=HBM_PEAK_GBPS, unit="GB/s",
            frac=round(ht_bytes / (ht_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
            traffic=read_traffic(traffic_file(wl.name)),
            launch_us=round(ht_us, 2), bytes_per_launch=ht_bytes, k_t_mean=kt,
            k_t_first=kts[0], k_t_last=kts[-1],
            bytes_model="12 d + 8 k_t (read g, read e, write e', 8 bytes per kept pair)"),
        "topk": dict(
            stats_us(tk_each), us_per_step=round(tk_us, 2),
            gelem_s=round(d / (tk_us * 1e-6) / 1e9, 2), bracket_path_steps=int(sum(paths)),
            bytes_ideal=tk_ideal, **rate(tk_ideal, tk_us),
            bytes_model="12 d + 8 k: what the step must move (frac is against this)"),
        "average": average,
        "copy_probe": {"us": round(copy_us, 2), "bytes": 8.0 * d, **rate(8.0 * d, copy_us)},
        "stream_ceiling": ceiling,
    }
    if not args.no_extra:
        line["extra"] = {"segments_25.6m": bench_segments(efs, torch, synth, cur, threads),
                         "layerwise_20000_layers": bench_many_layers(efs, torch, synth, cur),
                         "sparse_apply_8_workers": average.pop("_apply", None)}
    average.pop("_apply", None)
    if not args.no_cpu:
        line["cpu_baseline"], line["cpu_baseline_1core"] = cpu_baselines(pool_host, wl, lam)
    print(json.dumps(line), flush=True)


def stream_ceiling(efs, torch, cur, pool, d, calls=6):
    """Plain streaming kernels over the workload's d elements, per traffic
    mix, in the hard threshold's persistent grid and with one workgroup per
    4096-element tile: what a kernel with the hard threshold's traffic
    (2r1w: read g, read e, write e in place) reaches on this GPU.  The calls
    rotate over pairs of the pool's buffers, so that the data comes from HBM
    (the pool spans more than the 256 MB Infinity Cache)."""
    pairs = [(pool[i], pool[(i + 1) % len(pool)]) for i in range(0, max(len(pool), 2), 2)]
    if len(pool) < 2:
        pairs = [(pool[0], torch.empty_like(pool[0]))]
    whole = d // 4096 * 4096
    out = {"note": "us per call, back to back; bytes per call: copy 8d, read 4d, write 4d, "
                   "2r1w 12d (whole 4096-element tiles)"}
    best = 0.0
    for name, mode, nbytes in (("copy", 0, 8.0 * d), ("read", 1, 4.0 * whole),
                               ("write", 2, 4.0 * whole), ("2r1w", 3, 12.0 * whole)):
        for shape, bit in (("persistent", 0), ("tile_per_workgroup", 4)):
            for x, y in pairs:
                efs.stream_probe(x, y, mode + bit)
            with Timer(torch, cur) as t:
                for c in range(calls):
                    x, y = pairs[c % len(pairs)]
                    efs.stream_probe(x, y, mode + bit)
            us = t.us / calls
            r = rate(nbytes, us)
            out["%s_%s" % (name, shape)] = dict(us=round(us, 2), **r)
            if name == "2r1w":
                best = max(best, r["frac"])
    out["best_2r1w_frac"] = best
    return out


def describe(wl):
    return {"outliers": "Gaussian g std 1e-3 with a fixed 5% of coordinates at std 0.1",
            "segments": "161 log-uniform segments, Gaussian g with per-segment std "
                        "log-uniform [1e-5,1e-2]",
            "student_t": "200 segments, Student-t (nu=3) g scaled by 1e-4 x per-segment "
                         "log-uniform [0.1,10]",
            "gauss": "Gaussian g std 1e-3"}[wl.kind]


def bench_average(efs, torch, synth, cur, steps, warmup, threads):
    """sparse_accumulate over the eight workers' first-step hard-threshold
    payloads of the 8-worker workload (d = 25,557,032), the output rotating
    over four buffers; then the fused model updates on the same payloads."""
    st = synth.Stream(4)
    w = st.w
    d = w.d
    lam = synth.stored_lambda(4, w.densities[0])
    payloads = []
    for wk in range(w.n_workers):
        g = torch.from_numpy(st.gradient(0, worker=wk, threads=threads)).to("cuda")
        e = torch.zeros(d, dtype=torch.float32, device="cuda")
        cap = d // 100
        idx = torch.empty(cap, dtype=torch.int32, device="cuda")
        val = torch.empty(cap, dtype=torch.float32, device="cuda")
        ctr = efs.new_counter("cuda")
        efs.ht_compress(g, e, synth.LR, lam, idx, val, ctr)
        payloads.append((idx, val, ctr))
        del g, e
    pairs = sum(efs.counter_value(p[2]) for p in payloads)
    ws = efs.new_apply_workspace(payloads, d, "cuda")
    outs = [torch.empty(d, dtype=torch.float32, device="cuda") for _ in range(4)]
    calls = [efs.prepare_sparse_accumulate(payloads, d, o, ws) for o in outs]
    for s in range(warmup):
        calls[s % 4]()
    with Timer(torch, cur) as t:
        for s in range(steps):
            calls[s % 4]()
    us = t.us / steps
    # each call's own time: events between the same back-to-back calls
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    evs[0].record(cur)
    for s in range(steps):
        calls[s % 4]()
        evs[s + 1].record(cur)
    torch.cuda.synchronize()
    per_call = [evs[i].elapsed_time(evs[i + 1]) * 1e3 for i in range(steps)]
    status = efs.sparse_status(ws)
    nbytes = 4.0 * d + 8.0 * pairs
    res = {"workers": w.n_workers, "d": d, "pairs": pairs, "us": round(us, 2),
           "per_call": dict(stats_us(per_call), note="events between back-to-back calls"),
           "status": status,
           "bytes_min": nbytes, **rate(nbytes, us),
           "bytes_model": "4 d + 8 per pair (dense output write, payload read)"}
    say("average of %d payloads (%d pairs): %.1f us" % (w.n_workers, pairs, us))
    # the fused model updates on the same payloads, (x, m) rotating over four sets
    touched_idx = torch.unique(torch.cat(
        [p[0][:efs.counter_value(p[2])] for p in payloads]))
    touched = int(touched_idx.numel())
    # the SGD update reads and writes x only where a payload touches it:
    # scattered 4-byte updates, each moving its 128-byte cache line
    lines = int(torch.unique(touched_idx // 32).numel())
    ms = [torch.zeros(d, dtype=torch.float32, device="cuda") for _ in range(4)]
    upd = {"touched": touched, "lines_128b": lines}
    for mode, name, nb in ((efs.APPLY_SGD, "sgd", 8.0 * pairs + 8.0 * touched),
                           (efs.APPLY_MOMENTUM, "momentum", 8.0 * pairs + 16.0 * d)):
        fns = [efs.prepare_sparse_apply(payloads, d, mode, outs[r], ws, m=ms[r], beta=0.9,
                                        gamma=0.05) for r in range(4)]
        for s in range(4):
            fns[s]()
        with Timer(torch, cur) as t:
            for s in range(steps):
                fns[s % 4]()
        upd[name] = {"us": round(t.us / steps, 2), "bytes": nb, **rate(nb, t.us / steps)}
        if mode == efs.APPLY_SGD:
            lb = 8.0 * pairs + 2 * 128.0 * lines
            upd[name]["line_traffic"] = {
                "bytes": lb, **rate(lb, t.us / steps),
                "model": "8 per pair read + each touched 128-byte line of x read and written"}
    res["_apply"] = upd
    del ws, outs, ms, payloads
    torch.cuda.empty_cache()
    return res


def bench_segments(efs, torch, synth, cur, threads):
    """The 25,557,032-element, 161-segment workload: hard threshold, flat and
    layer-wise Top-k, each K = 20 back-to-back error-feedback steps on four
    gradients in turn after 30 untimed steps."""
    import numpy as np
    st = synth.Stream(2)
    w = st.w
    d, k = w.d, w.topk_k[0]
    lam = synth.stored_lambda(2, w.densities[0])
    pool = [torch.from_numpy(st.gradient(t, threads=threads)).to("cuda") for t in range(4)]
    lr = synth.LR
    reps, pre = 20, 30
    res = {"d": d}
    e = torch.zeros(d, dtype=torch.float32, device="cuda")
    idx = torch.empty(d, dtype=torch.int32, device="cuda")
    val = torch.empty(d, dtype=torch.float32, device="cuda")
    ctr = efs.new_counter("cuda")
    for s in range(pre):
        efs.ht_compress(pool[s % 4], e, lr, lam, idx, val, ctr)
    with Timer(torch, cur) as t:
        for s in range(reps):
            efs.ht_compress(pool[s % 4], e, lr, lam, idx, val, ctr)
    kt = efs.counter_value(ctr)
    us = t.us / reps
    res["ht_compress"] = {"us": round(us, 2), "k_t_last": kt,
                          "gelem_s": round(d / (us * 1e-6) / 1e9, 1), **rate(12.0 * d + 8.0 * kt, us)}
    e.zero_()
    tidx, tval = idx[:k], val[:k]
    ws = efs.new_topk_workspace(d, k, "cuda")
    for s in range(pre):
        efs.topk_compress(pool[s % 4], e, lr, k, tidx, tval, ws)
    each, paths = [], 0
    for s in range(reps):
        with Timer(torch, cur) as t:
            efs.topk_compress(pool[s % 4], e, lr, k, tidx, tval, ws)
        each.append(t.us)
        paths += efs.topk_took_bracket_path(ws)
    with Timer(torch, cur) as t:
        for s in range(reps):
            efs.topk_compress(pool[s % 4], e, lr, k, tidx, tval, ws)
    us = t.us / reps
    res["topk_compress"] = dict(stats_us(each), us_back_to_back=round(us, 2),
                                bracket_path_steps=paths, **rate(12.0 * d + 8.0 * k, us))
    ks = synth.layerwise_k(st.bounds, w.densities[0])
    kt = int(ks.sum())
    offd = torch.from_numpy(st.bounds.astype(np.int64)).to("cuda")
    kd = torch.from_numpy(ks).to("cuda")
    sidx = torch.empty(kt, dtype=torch.int32, device="cuda")
    sval = torch.empty(kt, dtype=torch.float32, device="cuda")
    sws = efs.new_topk_segmented_workspace(ks.size, kt, "cuda")
    e.zero_()
    for s in range(pre):
        efs.topk_segmented_compress(pool[s % 4], e, lr, offd, kd, sidx, sval, sws)
    with Timer(torch, cur) as t:
        for s in range(reps):
            efs.topk_segmented_compress(pool[s % 4], e, lr, offd, kd, sidx, sval, sws)
    us = t.us / reps
    res["topk_segmented_compress"] = {
        "us": round(us, 2), "segments": int(ks.size), "k_total": kt,
        "bracket_segments_last_call": efs.topk_segmented_bracket_segments(sws),
        **rate(12.0 * d + 8.0 * kt, us)}
    say("25.6e6 workload: %s" % res)
    del pool, e, idx, val, ws, sws
    torch.cuda.empty_cache()
    return res


def bench_many_layers(efs, torch, synth, cur):
    """Layer-wise Top-k over a model with 20,000 tensors: d = 25,600,000 split
    into 20,000 layers of log-uniform sizes (1 to 10^4 before scaling to d),
    k_s = ceil(0.1 % of each layer), Gaussian gradients; K = 20 back-to-back
    error-feedback steps on four gradients in turn after 30 untimed steps."""
    import numpy as np
    d, nseg = 25_600_000, 20_000
    sizes = synth.segment_sizes(7, nseg, d, lo=1.0, hi=1e4)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    ks = synth.layerwise_k(off, 0.001)
    kt = int(ks.sum())
    pool = [torch.from_numpy(synth.small_gradient(3000 + t, d)).to("cuda") for t in range(4)]
    lr = synth.LR
    reps, pre = 20, 30
    e = torch.zeros(d, dtype=torch.float32, device="cuda")
    sidx = torch.empty(kt, dtype=torch.int32, device="cuda")
    sval = torch.empty(kt, dtype=torch.float32, device="cuda")
    sws = efs.new_topk_segmented_workspace(nseg, kt, "cuda")
    offd = torch.from_numpy(off).to("cuda")
    kd = torch.from_numpy(ks).to("cuda")
    for s in range(pre):
        efs.topk_segmented_compress(pool[s % 4], e, lr, offd, kd, sidx, sval, sws)
    with Timer(torch, cur) as t:
        for s in range(reps):
            efs.topk_segmented_compress(pool[s % 4], e, lr, offd, kd, sidx, sval, sws)
    us = t.us / reps
    # layers touching more than one 4096-element block of the vector
    first, last = off[:-1] // 4096, (off[1:] - 1) // 4096
    multi = int(np.sum((sizes > 0) & (last > first)))
    res = {"d": d, "segments": nseg, "multi_tile_segments": multi,
           "k_total": kt, "us": round(us, 2),
           "bracket_segments_last_call": efs.topk_segmented_bracket_segments(sws),
           **rate(12.0 * d + 8.0 * kt, us)}
    say("20,000-layer layer-wise Top-k: %s" % res)
    del pool, e, sidx, sval, sws
    torch.cuda.empty_cache()
    return res


def bench_radix(efs, torch, synth, cur, wl, dev, calls=4):
    """Top-k from a fresh workspace (no threshold recorded, so the radix path)
    with e = 0 on the workload's first gradient: as drawn, and rounded to
    multiples of 2^-16 and 2^-10, which put ties at the threshold that must
    be split by index (a few hundred, listed; tens of thousands, counted per
    tile).  Each call timed alone with events on the stream it runs on."""
    import numpy as np
    d, k = wl.d, wl.topk_k[0]
    host = synth.Stream(wl.ident).gradient(0, threads=min(16, os.cpu_count() or 1))
    g = to_device(torch, host, dev)
    del host
    e = torch.zeros(d, dtype=torch.float32, device=dev)
    idx = torch.empty(k, dtype=torch.int32, device=dev)
    val = torch.empty(k, dtype=torch.float32, device=dev)
    ws = efs.new_topk_workspace(d, k, dev)
    res = {"workload": wl.name, "d": d, "k": k}
    for q in (0, 16, 10):
        if q:
            g.mul_(2.0 ** q).round_().div_(2.0 ** q)   # multiples of 2^-q, exact in fp32
        each = []
        for _ in range(calls):
            e.zero_()
            ws.zero_()
            with Timer(torch, cur) as t:
                efs.topk_compress(g, e, synth.LR, k, idx, val, ws)
            assert not efs.topk_took_bracket_path(ws)
            each.append(t.us)
        key = "as_drawn" if q == 0 else "multiples_of_2^-%d" % q
        res[key] = dict(stats_us(each), **rate(12.0 * d + 8.0 * k, float(np.median(each))))
        say("Top-k radix path, %s: %s" % (key, res[key]))
    del g, e, idx, val, ws
    torch.cuda.empty_cache()
    return res


def cpu_baselines(pool_host, wl, lam):
    """The CPU oracle on the same workload, a bounded sample of about 10-20 s
    of CPU work: error-feedback steps of the hard threshold over the whole
    vector (e from 0, the pool's gradients in turn), and Top-k on a leading
    slice of the first gradient (k = 0.1 % of the slice); the multi-core build
    on all host cores, then the single-threaded build with fewer steps and a
    smaller slice."""
    import numpy as np

    import oracle

    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    d = pool_host[0].size
    cap = 4 * int(round(wl.densities[0] * d)) + 1024
    out = []
    for mt, steps, slice_n in ((True, 4, min(d, 500_000_000)), (False, 2, min(d, 100_000_000))):
        e = np.zeros(d, np.float32)
        t0 = time.perf_counter()
        for s in range(steps):
            _, _, e, _ = oracle.ht(pool_host[s % len(pool_host)], e, synth_lr(), lam, cap=cap, mt=mt)
        ht_s = time.perf_counter() - t0
        del e
        sl = pool_host[0][:slice_n]
        ks = max(1, int(round(0.001 * slice_n)))
        t0 = time.perf_counter()
        oracle.topk(sl, np.zeros(slice_n, np.float32), synth_lr(), ks, mt=mt)
        tk_s = time.perf_counter() - t0
        cores = oracle.mt_threads() if mt else 1
        out.append({
            "value": round(steps * d / ht_s / 1e9, 4), "unit": "G grad-elements/s",
            "cores": cores, "kind": "oracle", "cpu_model": model, "host_cpus": os.cpu_count(),
            "build": "oracle.c + oracle_mt.c, OpenMP" if mt else "oracle.c, one thread",
            "topk_gelem_s": round(slice_n / tk_s / 1e9, 5),
            "sample": "%d hard-threshold error-feedback steps over the whole d=%d vector "
                      "(%.2f s); Top-k on the first %d elements of the first gradient with "
                      "k=%d (%.2f s)" % (steps, d, ht_s, slice_n, ks, tk_s)})
        say("CPU oracle (%d cores): %s" % (cores, out[-1]["sample"]))
    return out[0], out[1]


def synth_lr():
    from paper_2108_00951_amd import synth
    return synth.LR


if __name__ == "__main__":
    main()
