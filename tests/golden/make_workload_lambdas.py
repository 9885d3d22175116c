"""Writes workload_lambdas.json: the hard-threshold lambda of every workload
at each of its first-step densities, computed by the oracle only.

    python tests/golden/make_workload_lambdas.py

For each (workload, density) the threshold is oracle.calibrate_lambda on the
workload's first gradient g_0 (worker 0): the K-th largest |fl(lr * g_0)|,
K = round(density * d), the upper end of Lemma 3's interval.  The file also
records K and the number of coordinates the oracle's hard threshold keeps at
the first iteration with that lambda (e_0 = 0): K, or more when the K-th
magnitude is tied.  The inputs come from the seeded generator module, which
holds none of the method's arithmetic.  Takes a few minutes (the 1.5e9
workload draws 6 GB).
"""
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2108_00951_amd import synth  # noqa: E402

OUT = os.path.join(HERE, synth.LAMBDA_FILE)
CHUNK = 1 << 26


def first_step_count(g, lam):
    """Coordinates the oracle's hard threshold keeps at t = 0 (e_0 = 0),
    chunk by chunk (the threshold is element-wise)."""
    total = 0
    zeros = np.zeros(min(CHUNK, g.size), np.float32)
    for lo in range(0, g.size, CHUNK):
        hi = min(g.size, lo + CHUNK)
        total += oracle.ht(g[lo:hi], zeros[:hi - lo], synth.LR, lam, cap=0, mt=True)[3]
    return total


def main():
    threads = min(16, os.cpu_count() or 1)
    table = {"lr": float(synth.LR), "lambda_bits": {}, "lambda": {}, "K": {},
             "first_step_count": {}}
    for wid, w in sorted(synth.WORKLOADS.items()):
        st = synth.Stream(wid)
        g = st.gradient(0, worker=0, threads=threads)
        for density in w.densities:
            lam = oracle.calibrate_lambda(g, density, synth.LR)
            key = "%d/%g/%d" % (wid, density, 0)
            table["lambda_bits"][key] = int(np.array([lam], np.float32).view(np.uint32)[0])
            table["lambda"][key] = repr(float(lam))
            table["K"][key] = min(max(int(round(density * w.d)), 1), w.d)
            table["first_step_count"][key] = int(first_step_count(g, lam))
            print("%s: lambda=%r K=%d kept=%d" % (key, float(lam), table["K"][key],
                                                   table["first_step_count"][key]), flush=True)
        del g
    with open(OUT, "w") as f:
        json.dump(table, f, indent=1, sort_keys=True)
        f.write("\n")
    print("wrote", OUT)


if __name__ == "__main__":
    main()
