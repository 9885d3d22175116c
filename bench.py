"""Benchmark of the error-feedback compression step on one MI355X.

One step = one pass of the whole path over one synthetic gradient of the
25,557,032-element, 161-segment workload (Gaussian, per-segment std
log-uniform in [1e-5, 1e-2], lr = 0.1):
    hard threshold  ht_compress    (lambda giving 0.1 % density at the first step)
    Top-k           topk_compress  (k = 25,557, its own error vector)
    average         sparse_accumulate of the hard-threshold payload (n = 1)
Gradients rotate through a pool larger than the 256 MB Infinity Cache, so
every step reads them from HBM; the error vectors are carried from step to
step as in training.  Inputs are resident on the device before timing.

Prints one JSON line.  value = gradient elements compressed per second over
the whole step (2 d per step: d by each compressor); the K timed steps carry
HIP events only at their two ends.  The per-operation breakdown ("ops") comes
from a second pass over the same steps with events between the operations.

The roofline entry is for the hard-threshold kernel: algorithmic bytes
(12 per element + 8 per kept pair) over its launch duration, from HIP events
around back-to-back launches on four error-feedback states taken in turn, so
that g and e come from HBM as they do inside the step (ops also reports one
state carried from launch to launch, where part of e stays in the Infinity
Cache, and launches after a cache flush).  --traffic takes the counter-derived HBM
bytes per launch written by --parse-pmc from two rocprofv3 --pmc runs of this
script (FETCH_SIZE, then WRITE_SIZE), scaled by what the same counters read
for the copy probe of known size.
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
COPY_KERNEL = "copy_kernel"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "ht_fused_kernel_segments_25.6m_pmc.txt")
HT_SOURCES = ["ht.hip", "device_common.hpp"]


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
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--pool", type=int, default=4, help="distinct gradients in the rotation")
    ap.add_argument("--b2b", type=int, default=20,
                    help="back-to-back launches timed for the kernel roofline")
    ap.add_argument("--cpu-steps", type=int, default=2,
                    help="steps of the CPU oracle for the baseline (0 to skip)")
    ap.add_argument("--traffic", type=str, default=TRAFFIC_FILE,
                    help="summary written by --parse-pmc (HBM bytes per hard-threshold launch)")
    ap.add_argument("--parse-trace", metavar="TRACE_DIR",
                    help="print the kernel statistics of a rocprofv3 --kernel-trace --stats "
                         "run of this script (run_kernel_stats.csv, run_kernel_trace.csv), "
                         "with the average of the back-to-back hard-threshold launches that "
                         "roofline.launch_us times")
    ap.add_argument("--parse-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarise two rocprofv3 --pmc output folders and exit")
    ap.add_argument("--no-apply", action="store_true",
                    help="skip the fused update timings (sparse_apply, 1 and 8 workers)")
    ap.add_argument("--sweep", action="store_true",
                    help="also time the hard-threshold kernel on the 110e6 Student-t and "
                         "1.5e9 outlier workloads (adds ~1 min of input generation)")
    return ap.parse_args()


def _pmc_rows(folder, counter):
    """(kernel name, value) of every dispatch in a rocprofv3 counter CSV."""
    rows = []
    for path in glob.glob(os.path.join(folder, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as f:
            for r in csv.DictReader(f):
                if r.get("Counter_Name") == counter:
                    rows.append((r["Kernel_Name"], float(r["Counter_Value"])))
    return rows


def parse_pmc(fetch_dir, write_dir, d):
    """HBM bytes per launch of the hard-threshold kernel, scaled by the copy probe.

    FETCH_SIZE and WRITE_SIZE are in KiB per dispatch.  The copy probe moves
    exactly 4n bytes in and 4n bytes out (n = d); the ratio of those bytes to
    what the counters report for it is the scale applied to the kernel."""
    out = {}
    for name, folder in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = _pmc_rows(folder, name)
        ht = [v for k, v in rows if HT_KERNEL in k]
        cp = [v for k, v in rows if COPY_KERNEL in k]
        if not ht or not cp:
            raise SystemExit("no %s rows for %s / %s in %s" % (name, HT_KERNEL, COPY_KERNEL, folder))
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


def parse_trace(folder, b2b):
    """Per-kernel statistics of a rocprofv3 kernel trace, and the average of
    the first `b2b` consecutive dispatches of the hard-threshold kernel (its
    plain variant) that no other kernel interrupts: the launches
    roofline.launch_us times with HIP events."""
    import csv
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
    plain = HT_KERNEL + "<true, false>"
    runs, cur = [], []
    for r in trace:
        if plain in r["Kernel_Name"]:
            cur.append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
        else:
            if cur:
                runs.append(cur)
            cur = []
    if cur:
        runs.append(cur)
    b2b_runs = [x for x in runs if len(x) == b2b]
    lines.append("")
    if b2b_runs:
        x = b2b_runs[0]
        lines.append("# %s, the %d back-to-back launches timed for roofline.launch_us: "
                     "avg %.2f us, min %.2f, max %.2f" % (plain, b2b, sum(x) / len(x), min(x), max(x)))
    else:
        lines.append("# no run of %d back-to-back %s dispatches in the trace" % (b2b, plain))
    return "\n".join(lines) + "\n"


def format_traffic(res):
    lines = ["# HBM traffic of %s per launch from rocprofv3 counters" % HT_KERNEL,
             "# (KiB per dispatch, averaged over the kernel's dispatches; each counter",
             "# scaled by expected/measured for %s moving 4*d bytes each way)" % COPY_KERNEL]
    for name in ("FETCH_SIZE", "WRITE_SIZE"):
        r = res[name]
        lines.append("# %s: kernel %.1f KiB, copy probe %.1f KiB (expected %.1f), scale %.5f, "
                     "%d launches" % (name, r["ht_kib_per_launch"], r["copy_kib_per_launch"],
                                      r["copy_expected_kib"], r["scale"], r["launches"]))
    fk, wk = res["FETCH_SIZE"].get("kernels", {}), res["WRITE_SIZE"].get("kernels", {})
    if fk or wk:
        lines.append("# every kernel of the run, scaled the same way: MB fetched + MB written per "
                     "launch (launches)")
        names = sorted(set(fk) | set(wk),
                       key=lambda n: -(fk.get(n, (0.0, 0))[0] + wk.get(n, (0.0, 0))[0]))
        for n in names:
            f, nf = fk.get(n, (0.0, 0))
            w, nw = wk.get(n, (0.0, 0))
            lines.append("#   %-34s %9.2f + %9.2f MB  (%d)" % (n, f / 1e6, w / 1e6, max(nf, nw)))
    lines.append("ht_bytes_per_launch %d" % round(res["ht_bytes_per_launch"]))
    lines.append("kernel_source_sha256 %s" % kernel_source_digest())
    return "\n".join(lines) + "\n"


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(got --gpus %d)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import numpy as np

    from paper_2108_00951_amd import synth

    wl = synth.WORKLOADS[2]
    d, k, density = wl.d, wl.topk_k[0], wl.densities[0]
    if args.parse_pmc:
        sys.stdout.write(format_traffic(parse_pmc(args.parse_pmc[0], args.parse_pmc[1], d)))
        return
    if args.parse_trace:
        sys.stdout.write(parse_trace(args.parse_trace, args.b2b))
        return

    import torch

    from paper_2108_00951_amd import binding as efs

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    efs.load_library()

    lr = synth.LR
    stream = synth.Stream(2)
    t0 = time.time()
    pool_host = [stream.gradient(t, threads=16) for t in range(args.pool)]
    lam = synth.calibrate_lambda(pool_host[0], density, lr)
    pool = [torch.from_numpy(g).to(dev) for g in pool_host]
    print("inputs ready: d=%d pool=%d lambda=%.6g k=%d (%.1fs)"
          % (d, args.pool, float(lam), k, time.time() - t0), file=sys.stderr, flush=True)

    e_ht = torch.zeros(d, dtype=torch.float32, device=dev)
    e_tk = torch.zeros(d, dtype=torch.float32, device=dev)
    cap = d   # k_t grows under error feedback with a fixed lambda; never truncate
    idx = torch.empty(cap, dtype=torch.int32, device=dev)
    val = torch.empty(cap, dtype=torch.float32, device=dev)
    ctr = efs.new_counter(dev)
    tidx = torch.empty(k, dtype=torch.int32, device=dev)
    tval = torch.empty(k, dtype=torch.float32, device=dev)
    ws = efs.new_topk_workspace(d, k, dev)
    out = torch.empty(d, dtype=torch.float32, device=dev)
    cur = torch.cuda.current_stream()

    def ev():
        return torch.cuda.Event(enable_timing=True)

    def step(s, evs=None):
        g = pool[s % len(pool)]
        if evs is not None:
            evs[0].record(cur)
        efs.ht_compress(g, e_ht, lr, lam, idx, val, ctr)
        if evs is not None:
            evs[1].record(cur)
        efs.topk_compress(g, e_tk, lr, k, tidx, tval, ws)
        if evs is not None:
            evs[2].record(cur)
        efs.sparse_accumulate([(idx, val, ctr)], d, out)
        if evs is not None:
            evs[3].record(cur)

    for s in range(args.warmup):
        step(s)
    torch.cuda.synchronize()
    e_ht_start = e_ht.clone()
    e_tk_start = e_tk.clone()

    # ---- timed region: K whole steps, events only at its two ends -------
    begin, end = ev(), ev()
    torch.cuda.synchronize()
    begin.record(cur)
    for s in range(args.steps):
        step(args.warmup + s)
    end.record(cur)
    torch.cuda.synchronize()
    e_ht_end = e_ht.clone()
    e_tk_end = e_tk.clone()

    # ---- per-operation breakdown: the same K steps again from the same
    # state, with events between the operations (the event packets add
    # dispatch gaps, so this pass is reported but not used for the step time)
    e_ht.copy_(e_ht_start)
    e_tk.copy_(e_tk_start)
    evs = [[ev() for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    for s in range(args.steps):
        step(args.warmup + s, evs[s])
    torch.cuda.synchronize()

    # k_t of every timed step, from a deterministic replay of the
    # hard-threshold calls (same inputs, same starting e).
    e_ht.copy_(e_ht_start)
    kts = []
    for s in range(args.steps):
        efs.ht_compress(pool[(args.warmup + s) % len(pool)], e_ht, lr, lam, idx, val, ctr)
        kts.append(efs.counter_value(ctr))

    # Which Top-k selection each timed step took (same replay idea).
    e_tk.copy_(e_tk_start)
    bracket_hits = 0
    for s in range(args.steps):
        efs.topk_compress(pool[(args.warmup + s) % len(pool)], e_tk, lr, k, tidx, tval, ws)
        bracket_hits += efs.topk_took_bracket_path(ws)

    # ---- kernel durations: back-to-back launches -------------------------
    # Hard threshold on four error-feedback states continuing from the end of
    # the timed region, taken in turn, each with its own gradient sequence:
    # g and e of every launch come from HBM, as inside the step, where the
    # other operations evict them from the 256 MB Infinity Cache.
    e_rot = [e_ht_end.clone() for _ in range(4)]
    ctr_rot = [efs.new_counter(dev) for _ in range(4)]

    def ht_rot(s, telemetry=None):
        r = s % 4
        g = pool[(s + s // 4) % len(pool)]
        if telemetry is None:
            efs.ht_compress(g, e_rot[r], lr, lam, idx, val, ctr_rot[r])
        else:
            efs.ht_compress_telemetry(g, e_rot[r], lr, lam, idx, val, ctr_rot[r], telemetry)

    a, b = ev(), ev()
    torch.cuda.synchronize()
    a.record(cur)
    for s in range(args.b2b):
        ht_rot(s)
    b.record(cur)
    torch.cuda.synchronize()
    ht_b2b_us = a.elapsed_time(b) * 1e3 / args.b2b
    kt_b2b = float(np.mean([efs.counter_value(c) for c in ctr_rot]))
    # the same with the fused telemetry (total error, pairs sent, max |e'|)
    tel = efs.new_telemetry(dev)
    a, b = ev(), ev()
    torch.cuda.synchronize()
    a.record(cur)
    for s in range(args.b2b):
        ht_rot(s, tel)
    b.record(cur)
    torch.cuda.synchronize()
    ht_tel_us = a.elapsed_time(b) * 1e3 / args.b2b
    # copy probe over the same element count, destinations in turn
    a, b = ev(), ev()
    a.record(cur)
    for s in range(args.b2b):
        efs.copy_probe(pool[s % len(pool)], e_rot[(s + 1) % 4])
    b.record(cur)
    torch.cuda.synchronize()
    copy_us = a.elapsed_time(b) * 1e3 / args.b2b
    del e_rot
    # one state carried from launch to launch (an EF loop with nothing in
    # between): part of e then stays in the Infinity Cache
    e_ht.copy_(e_ht_end)
    a, b = ev(), ev()
    torch.cuda.synchronize()
    a.record(cur)
    for s in range(args.b2b):
        efs.ht_compress(pool[s % len(pool)], e_ht, lr, lam, idx, val, ctr)
    b.record(cur)
    torch.cuda.synchronize()
    ht_one_us = a.elapsed_time(b) * 1e3 / args.b2b
    kt_one = efs.counter_value(ctr)
    # cold: a 1 GiB write (stream probe) before every launch evicts the 256 MB
    # Infinity Cache, so g and e come from HBM; events around the launch only
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    cold = []
    for s in range(args.b2b):
        efs.stream_probe(flush, flush, 2)
        a, b = ev(), ev()
        a.record(cur)
        efs.ht_compress(pool[s % len(pool)], e_ht, lr, lam, idx, val, ctr)
        b.record(cur)
        torch.cuda.synchronize()
        cold.append(a.elapsed_time(b) * 1e3)
    del flush
    ht_cold_us = float(np.median(cold))
    kt_cold = efs.counter_value(ctr)
    # layer-wise Top-k over the workload's 161 segments, k_s = ceil(0.1 % d_s)
    seg_ks = synth.layerwise_k(stream.bounds, density)
    seg_ktot = int(seg_ks.sum())
    seg_off_d = torch.from_numpy(stream.bounds.astype(np.int64)).to(dev)
    seg_k_d = torch.from_numpy(seg_ks).to(dev)
    seg_idx = torch.empty(seg_ktot, dtype=torch.int32, device=dev)
    seg_val = torch.empty(seg_ktot, dtype=torch.float32, device=dev)
    seg_ws = efs.new_topk_segmented_workspace(seg_ks.size, seg_ktot, dev)
    e_seg = torch.zeros(d, dtype=torch.float32, device=dev)
    seg_ws.zero_()
    # as many untimed calls as the step loop has run (warmup + timed steps), so
    # the error vector is as far into training as the step's own
    for s in range(args.warmup + args.steps):
        efs.topk_segmented_compress(pool[s % len(pool)], e_seg, lr, seg_off_d, seg_k_d, seg_idx,
                                    seg_val, seg_ws)
    a, b = ev(), ev()
    torch.cuda.synchronize()
    a.record(cur)
    for s in range(args.b2b):
        efs.topk_segmented_compress(pool[s % len(pool)], e_seg, lr, seg_off_d, seg_k_d, seg_idx,
                                    seg_val, seg_ws)
    b.record(cur)
    torch.cuda.synchronize()
    seg_us = a.elapsed_time(b) * 1e3 / args.b2b
    seg_hits = efs.topk_segmented_bracket_segments(seg_ws)
    del e_seg, seg_ws

    total_ms = begin.elapsed_time(end)
    ms_step = total_ms / args.steps
    ht_ms = [x[0].elapsed_time(x[1]) for x in evs]
    tk_ms = [x[1].elapsed_time(x[2]) for x in evs]
    ac_ms = [x[2].elapsed_time(x[3]) for x in evs]
    kt = float(np.mean(kts))

    def stats(xs):
        a = np.sort(np.asarray(xs))
        return {"mean_us": round(float(a.mean()) * 1e3, 2),
                "p10_us": round(float(a[int(0.1 * (a.size - 1))]) * 1e3, 2),
                "p50_us": round(float(np.median(a)) * 1e3, 2),
                "p90_us": round(float(a[int(0.9 * (a.size - 1))]) * 1e3, 2)}

    ht_bytes = 12.0 * d + 8.0 * kt
    ht_bytes_b2b = 12.0 * d + 8.0 * kt_b2b
    tk_bytes_ideal = 12.0 * d + 8.0 * k
    tk_bytes_twolook = 16.0 * d + 8.0 * k
    ac_bytes = 4.0 * d + 8.0 * kt
    ht_s = float(np.mean(ht_ms)) / 1e3
    tk_s = float(np.mean(tk_ms)) / 1e3
    ac_s = float(np.mean(ac_ms)) / 1e3
    roof_gbps = ht_bytes_b2b / (ht_b2b_us * 1e-6) / 1e9

    traffic = read_traffic(args.traffic)

    line = {
        "metric": "G grad-elements/s compressed (hard-threshold, Top-k) + achieved HBM GB/s",
        "value": round(2.0 * d / (ms_step / 1e3) / 1e9, 3),
        "unit": "G grad-elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "d=25,557,032 fp32 in 161 log-uniform segments, Gaussian g with "
                        "per-segment std log-uniform [1e-5,1e-2], lr=0.1; hard threshold at "
                        "0.1%% first-step density (lambda=%.6g) + Top-k k=25,557 + average of "
                        "the hard-threshold payload" % float(lam),
            "d": d, "k": k, "lambda": float(lam), "lr": float(lr), "pool": args.pool,
        },
        "hbm_gbps_step": round((ht_bytes + tk_bytes_twolook + ac_bytes) / (ms_step / 1e3) / 1e9, 1),
        "roofline": {
            "kernel": HT_KERNEL,
            "bound": "hbm",
            "achieved": round(roof_gbps, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(roof_gbps / HBM_PEAK_GBPS, 4),
            "traffic": traffic,
            "launch_us": round(ht_b2b_us, 2),
            "bytes_per_launch": ht_bytes_b2b,
            "k_t": kt_b2b,
        },
        "copy_probe": {"us": round(copy_us, 2), "gbps": round(8.0 * d / (copy_us * 1e-6) / 1e9, 1),
                       "bytes": 8.0 * d},
        "ops": {
            "ht_compress_telemetry": {"launch_us": round(ht_tel_us, 2)},
            "ht_compress_one_state": {
                "launch_us": round(ht_one_us, 2), "k_t": kt_one,
                "gbps": round((12.0 * d + 8.0 * kt_one) / (ht_one_us * 1e-6) / 1e9, 1)},
            "ht_compress_cold": {
                "median_us": round(ht_cold_us, 2), "p10_us": round(float(np.percentile(cold, 10)), 2),
                "p90_us": round(float(np.percentile(cold, 90)), 2),
                "gbps": round((12.0 * d + 8.0 * kt_cold) / (ht_cold_us * 1e-6) / 1e9, 1),
                "vs_b2b": round(ht_cold_us / ht_b2b_us, 3)},
            "topk_segmented_compress": {
                "launch_us": round(seg_us, 2), "segments": int(seg_ks.size), "k_total": seg_ktot,
                "bracket_segments_last_call": seg_hits,
                "gelem_s": round(d / (seg_us * 1e-6) / 1e9, 2),
                "gbps_ideal": round((12.0 * d + 8.0 * seg_ktot) / (seg_us * 1e-6) / 1e9, 1),
                "gbps_two_pass": round((16.0 * d + 8.0 * seg_ktot) / (seg_us * 1e-6) / 1e9, 1)},
            "ht_compress": dict(stats(ht_ms), gelem_s=round(d / ht_s / 1e9, 2),
                                gbps=round(ht_bytes / ht_s / 1e9, 1), k_t_mean=kt,
                                k_t_first=kts[0], k_t_last=kts[-1]),
            "topk_compress": dict(stats(tk_ms), gelem_s=round(d / tk_s / 1e9, 2),
                                  bracket_path_steps=bracket_hits,
                                  gbps_ideal=round(tk_bytes_ideal / tk_s / 1e9, 1),
                                  gbps_twolook=round(tk_bytes_twolook / tk_s / 1e9, 1)),
            "sparse_accumulate": dict(stats(ac_ms),
                                      gbps_min=round(ac_bytes / ac_s / 1e9, 1)),
        },
    }

    if not args.no_apply:
        line["sparse_apply"] = apply_bench(efs, torch, synth, cur, args.b2b, (idx, val, ctr), d)
    if args.sweep:
        del pool, e_tk, out, ws
        line["ht_sweep"] = ht_sweep(efs, torch, synth, cur, args.b2b)
    if args.cpu_steps > 0:
        line["cpu_baseline"] = cpu_baseline(pool_host, d, k, lam, lr, args.cpu_steps)
    print(json.dumps(line), flush=True)


def ht_sweep(efs, torch, synth, cur, reps):
    """Back-to-back launches on the larger workloads, two distinct gradients
    alternating, e carried: the hard threshold (0.1 % first-step density),
    the streaming ceilings, Top-k at the workload's densities and, where the
    workload has layers, the layer-wise Top-k at 1 %."""
    import numpy as np
    res = {}
    for wid in (3, 5):
        st = synth.Stream(wid)
        d = st.w.d
        gh = st.gradient(0, threads=16)
        lam = synth.calibrate_lambda(gh, 0.001)
        gs = [torch.from_numpy(gh).to("cuda")]
        del gh
        gs.append(torch.from_numpy(st.gradient(1, threads=16)).to("cuda"))
        e = torch.zeros(d, dtype=torch.float32, device="cuda")
        cap = d // 4
        idx = torch.empty(cap, dtype=torch.int32, device="cuda")
        val = torch.empty(cap, dtype=torch.float32, device="cuda")
        ctr = efs.new_counter("cuda")
        for s in range(2):
            efs.ht_compress(gs[s % 2], e, synth.LR, lam, idx, val, ctr)
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(cur)
        for s in range(reps):
            efs.ht_compress(gs[s % 2], e, synth.LR, lam, idx, val, ctr)
        b.record(cur)
        torch.cuda.synchronize()
        us = a.elapsed_time(b) * 1e3 / reps
        kt = efs.counter_value(ctr)
        if kt > cap:
            raise RuntimeError("sweep payload capacity exceeded")
        gbps = (12.0 * d + 8.0 * kt) / (us * 1e-6) / 1e9
        res[st.w.name] = {"d": d, "launch_us": round(us, 2), "k_t": kt,
                          "gbps": round(gbps, 1), "frac": round(gbps / HBM_PEAK_GBPS, 4),
                          "gelem_s": round(d / (us * 1e-6) / 1e9, 1)}
        del e, idx, val
        torch.cuda.empty_cache()
        # Top-k on the same gradients, its own e from zero: 5 calls, then
        # `reps` back-to-back calls timed (bytes: 12 per element + 8 per pair
        # ideal, 16 + 8 per pair for the two-look radix path)
        dens = (0.01, 0.001, 0.0001) if wid == 3 else (0.001,)
        res[st.w.name]["topk"] = {}
        for rho in dens:
            k = max(1, int(round(rho * d)))
            e = torch.zeros(d, dtype=torch.float32, device="cuda")
            tidx = torch.empty(k, dtype=torch.int32, device="cuda")
            tval = torch.empty(k, dtype=torch.float32, device="cuda")
            ws = efs.new_topk_workspace(d, k, "cuda")
            for s in range(5):
                efs.topk_compress(gs[s % 2], e, synth.LR, k, tidx, tval, ws)
            torch.cuda.synchronize()
            a.record(cur)
            for s in range(reps):
                efs.topk_compress(gs[s % 2], e, synth.LR, k, tidx, tval, ws)
            b.record(cur)
            torch.cuda.synchronize()
            us = a.elapsed_time(b) * 1e3 / reps
            res[st.w.name]["topk"]["k=%d" % k] = {
                "launch_us": round(us, 2), "gelem_s": round(d / (us * 1e-6) / 1e9, 1),
                "gbps_ideal": round((12.0 * d + 8.0 * k) / (us * 1e-6) / 1e9, 1),
                "gbps_twolook": round((16.0 * d + 8.0 * k) / (us * 1e-6) / 1e9, 1),
                "last_call_bracket": efs.topk_took_bracket_path(ws)}
            del e, tidx, tval, ws
            torch.cuda.empty_cache()
        if st.bounds is not None:
            # layer-wise Top-k over the workload's segments at 1 %
            ks = synth.layerwise_k(st.bounds, 0.01)
            kt = int(ks.sum())
            offd = torch.from_numpy(st.bounds.astype(np.int64)).to("cuda")
            kd = torch.from_numpy(ks).to("cuda")
            e = torch.zeros(d, dtype=torch.float32, device="cuda")
            tidx = torch.empty(kt, dtype=torch.int32, device="cuda")
            tval = torch.empty(kt, dtype=torch.float32, device="cuda")
            ws = efs.new_topk_segmented_workspace(ks.size, kt, "cuda")
            ws.zero_()
            for s in range(5):
                efs.topk_segmented_compress(gs[s % 2], e, synth.LR, offd, kd, tidx, tval, ws)
            torch.cuda.synchronize()
            a.record(cur)
            for s in range(reps):
                efs.topk_segmented_compress(gs[s % 2], e, synth.LR, offd, kd, tidx, tval, ws)
            b.record(cur)
            torch.cuda.synchronize()
            us = a.elapsed_time(b) * 1e3 / reps
            res[st.w.name]["topk_layerwise_1pct"] = {
                "segments": int(ks.size), "k_total": kt, "launch_us": round(us, 2),
                "gelem_s": round(d / (us * 1e-6) / 1e9, 1),
                "gbps_ideal": round((12.0 * d + 8.0 * kt) / (us * 1e-6) / 1e9, 1),
                "bracket_segments_last_call": efs.topk_segmented_bracket_segments(ws)}
            del e, tidx, tval, ws
        # streaming ceilings on the same buffers (whole tiles): copy, read,
        # write, and two reads + one write (the hard threshold's pattern);
        # last, because the write probes overwrite the second gradient
        nt = (d // 4096) * 4096
        ceil = {}
        for mode, name, nbytes in ((0, "copy", 8.0), (1, "read", 4.0), (2, "write", 4.0),
                                   (3, "2r1w", 12.0)):
            a.record(cur)
            for s in range(reps):
                efs.stream_probe(gs[0][:nt], gs[1][:nt], mode)
            b.record(cur)
            torch.cuda.synchronize()
            pus = a.elapsed_time(b) * 1e3 / reps
            ceil[name] = round(nbytes * nt / (pus * 1e-6) / 1e9, 1)
        res[st.w.name]["ceiling_gbps"] = ceil
        print("sweep %s: %s" % (st.w.name, res[st.w.name]), file=sys.stderr, flush=True)
        del gs
        torch.cuda.empty_cache()
    return res


def apply_bench(efs, torch, synth, cur, reps, ht_payload, d):
    """Back-to-back sparse_apply launches in each mode: on the step's own
    hard-threshold payload (1 worker), and on 8 workers' payloads of the
    8-worker workload (same d and segment layout, 0.1 % first-step density),
    next to sparse_accumulate on the same payloads; the launches take four
    output sets in turn.  Algorithmic bytes:
    average 8 per pair + 4 d; sgd 8 per pair + 8 per touched coordinate;
    momentum 8 per pair + 16 d."""
    import numpy as np

    def timed(fns):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        for fn in fns:
            fn()
        torch.cuda.synchronize()
        a.record(cur)
        for s in range(reps):
            fns[s % len(fns)]()
        b.record(cur)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / reps

    def measure(payloads):
        pairs = sum(efs.counter_value(p[2]) for p in payloads)
        touched = int(torch.unique(torch.cat(
            [p[0][:efs.counter_value(p[2])] for p in payloads])).numel())
        ws = efs.new_apply_workspace(payloads, d, "cuda")
        # four (x, m) sets taken in turn, so that they come from HBM as the
        # parameters and momentum of a training step would
        xs = [torch.zeros(d, dtype=torch.float32, device="cuda") for _ in range(4)]
        ms = [torch.zeros(d, dtype=torch.float32, device="cuda") for _ in range(4)]
        res = {"pairs": pairs, "touched": touched, "workspace_mb": round(ws.numel() / 2 ** 20, 1)}
        for mode, name, nbytes in (
                (efs.APPLY_AVERAGE, "average", 8.0 * pairs + 4.0 * d),
                (efs.APPLY_SGD, "sgd", 8.0 * pairs + 8.0 * touched),
                (efs.APPLY_MOMENTUM, "momentum", 8.0 * pairs + 16.0 * d)):
            us = timed([efs.prepare_sparse_apply(payloads, d, mode, xs[r], ws, m=ms[r], beta=0.9,
                                                 gamma=0.05) for r in range(4)])
            res[name] = {"us": round(us, 2), "gbps": round(nbytes / (us * 1e-6) / 1e9, 1)}
        us = timed([efs.prepare_sparse_accumulate(payloads, d, x) for x in xs])
        res["sparse_accumulate_us"] = round(us, 2)
        del ws, xs, ms
        return res

    res = {"workers_1": measure([ht_payload])}
    st = synth.Stream(4)
    w = st.w
    assert w.d == d
    lam = synth.calibrate_lambda(st.gradient(0, worker=0, threads=16), w.densities[0])
    payloads = []
    for wk in range(w.n_workers):
        g = torch.from_numpy(st.gradient(0, worker=wk, threads=16)).to("cuda")
        e = torch.zeros(d, dtype=torch.float32, device="cuda")
        cap = d // 100
        idx = torch.empty(cap, dtype=torch.int32, device="cuda")
        val = torch.empty(cap, dtype=torch.float32, device="cuda")
        ctr = efs.new_counter("cuda")
        efs.ht_compress(g, e, synth.LR, lam, idx, val, ctr)
        if efs.counter_value(ctr) > cap:
            raise RuntimeError("apply bench payload capacity exceeded")
        payloads.append((idx, val, ctr))
        del g, e
    res["workers_8"] = measure(payloads)
    print("sparse_apply: %s" % res, file=sys.stderr, flush=True)
    torch.cuda.empty_cache()
    return res


def cpu_baseline(pool_host, d, k, lam, lr, steps):
    """The CPU oracle (single-threaded C, as written) on the same step."""
    import numpy as np

    import oracle

    e_ht = np.zeros(d, dtype=np.float32)
    e_tk = np.zeros(d, dtype=np.float32)
    t0 = time.perf_counter()
    for s in range(steps):
        g = pool_host[s % len(pool_host)]
        ridx, rval, e_ht, _ = oracle.ht(g, e_ht, lr, lam)
        _, _, e_tk = oracle.topk(g, e_tk, lr, k)
        oracle.accumulate([(ridx, rval)], d)
    dt = time.perf_counter() - t0
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": round(2.0 * d * steps / dt / 1e9, 5), "unit": "G grad-elements/s",
            "cores": 1, "kind": "oracle", "cpu_model": model, "host_cpus": os.cpu_count(),
            "sample": "%d full steps (d=%d: hard threshold + Top-k + average) of the same "
                      "workload, single-threaded C oracle, %.1f s" % (steps, d, dt)}


if __name__ == "__main__":
    main()
