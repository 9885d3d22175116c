"""Seeded synthetic gradient streams and parameter recipes.

This module holds no part of the compression arithmetic: it only draws the
inputs (gradients g_t, per worker and iteration) with numpy's counter-free
PCG64 generator keyed by a SeedSequence, and holds the workload parameters
(sizes, densities, k, the layer-wise budgets).  Both the HIP path and the
CPU oracle are fed from here.  The threshold lambda that gives a workload's
first-step density is a selection on fl(lr * g_0), so it is computed by the
oracle (a committed script stores each workload's value, read by
`stored_lambda`).

The paper trains real models (Table 1 of Appendix C lists ResNet-18 with
11,173,962 parameters, an LSTM with 28,949,319 and NCF with 31,832,577);
those gradient streams are not available, so the workloads below stand in
for them with synthetic vectors of that size class and a layer-wise
(segment) structure, up to 1.5e9 elements.

Draws are made per fixed block of BLOCK elements, each block with its own
seed, so any element range of any gradient can be regenerated on its own
(used to stream the 1.5e9-element case through the oracle chunk by chunk).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

ROOT_ENTROPY = 2108_00951
BLOCK = 1 << 22            # elements per independently seeded draw block
LR = np.float32(0.1)       # step size gamma used by every workload


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic gradient stream.

    kind       "gauss" | "segments" | "student_t" | "outliers"
    d          vector length
    iters      EF iterations the workload runs
    densities  hard-threshold target densities at the first iteration
    topk_k     Top-k k values (one per density)
    n_workers  simulated workers (>1 only for the aggregation workload)
    nseg       number of contiguous segments (layer stand-ins)
    """
    ident: int
    name: str
    kind: str
    d: int
    iters: int
    densities: tuple
    topk_k: tuple
    n_workers: int = 1
    nseg: int = 0


WORKLOADS = {
    1: Workload(1, "gauss_1m", "gauss", 1_000_000, 10, (0.01,), (1_000,)),
    2: Workload(2, "segments_25.6m", "segments", 25_557_032, 100, (0.001,), (25_557,),
                nseg=161),
    3: Workload(3, "student_t_110m", "student_t", 110_000_000, 50,
                (0.01, 0.001, 0.0001), (1_100_000, 110_000, 11_000), nseg=200),
    4: Workload(4, "segments_25.6m_x8", "segments", 25_557_032, 100, (0.001,), (25_557,),
                n_workers=8, nseg=161),
    5: Workload(5, "outliers_1.5b", "outliers", 1_500_000_000, 20, (0.001,), (1_500_000,)),
}


def _rng(*key):
    ss = np.random.SeedSequence(entropy=ROOT_ENTROPY, spawn_key=tuple(int(k) for k in key))
    return np.random.Generator(np.random.PCG64(ss))


def segment_sizes(workload_id: int, nseg: int, d: int, lo: float = 64.0,
                  hi: float = 2.4e6) -> np.ndarray:
    """Contiguous segment sizes, log-uniform in [lo, hi], rescaled to sum d.

    Sizes are floored after scaling; the remainder goes one element each to
    the largest segments; every segment keeps at least one element.
    """
    rng = _rng(workload_id, 0, 0, 1)
    raw = np.exp(rng.uniform(math.log(lo), math.log(hi), size=nseg))
    scaled = raw * (d / raw.sum())
    sizes = np.maximum(np.floor(scaled).astype(np.int64), 1)
    rem = d - int(sizes.sum())
    order = np.argsort(-scaled, kind="stable")
    j = 0
    while rem != 0:
        s = order[j % nseg]
        if rem > 0:
            sizes[s] += 1
            rem -= 1
        elif sizes[s] > 1:
            sizes[s] -= 1
            rem += 1
        j += 1
    assert int(sizes.sum()) == d
    return sizes


def segment_scales(workload_id: int, nseg: int, lo: float, hi: float) -> np.ndarray:
    """Per-segment scale, log-uniform in [lo, hi], drawn once per workload."""
    rng = _rng(workload_id, 0, 0, 2)
    return np.exp(rng.uniform(math.log(lo), math.log(hi), size=nseg)).astype(np.float32)


class Stream:
    """Gradient stream g_{w,t} of one workload (all workers share the layout)."""

    def __init__(self, workload_id: int):
        self.w = WORKLOADS[workload_id]
        w = self.w
        self.bounds = None
        self.scales = None
        if w.kind == "segments":
            sizes = segment_sizes(w.ident if w.ident != 4 else 2, w.nseg, w.d)
            self.bounds = np.concatenate([[0], np.cumsum(sizes)])
            self.scales = segment_scales(w.ident if w.ident != 4 else 2, w.nseg, 1e-5, 1e-2)
        elif w.kind == "student_t":
            sizes = segment_sizes(w.ident, w.nseg, w.d)
            self.bounds = np.concatenate([[0], np.cumsum(sizes)])
            self.scales = (np.float32(1e-4) *
                           segment_scales(w.ident, w.nseg, 0.1, 10.0)).astype(np.float32)

    def _fill_block(self, worker: int, t: int, b: int, o: np.ndarray) -> None:
        """Writes g_{worker,t}[b*BLOCK : b*BLOCK + o.size] into o (in place)."""
        w = self.w
        start = b * BLOCK
        n = o.size
        rng = _rng(w.ident, worker, t, 100 + b)
        if w.kind == "student_t":
            np.copyto(o, rng.standard_t(3, size=n), casting="same_kind")
        else:
            rng.standard_normal(out=o, dtype=np.float32)
        if w.kind == "gauss":
            o *= np.float32(1e-3)
        elif w.kind in ("segments", "student_t"):
            self._scale_segments(o, start)
            if w.n_workers > 1:
                shift = np.empty(n, dtype=np.float32)
                _rng(w.ident, worker, 0, 1_000_000 + b).standard_normal(out=shift,
                                                                        dtype=np.float32)
                shift *= np.float32(1e-4)   # fixed per-worker offset mu_w ~ N(0, 1e-4^2)
                o += shift
        elif w.kind == "outliers":
            # fixed Bernoulli(0.05) set of large-gradient coordinates
            u = np.empty(n, dtype=np.float32)
            _rng(w.ident, 0, 0, 2_000_000 + b).random(out=u, dtype=np.float32)
            big = u < np.float32(0.05)
            np.multiply(o, np.float32(0.1), out=o, where=big)
            np.multiply(o, np.float32(1e-3), out=o, where=~big)
        else:
            raise ValueError(w.kind)

    def _scale_segments(self, o: np.ndarray, start: int) -> None:
        stop = start + o.size
        j0 = int(np.searchsorted(self.bounds, start, side="right")) - 1
        j = j0
        while j < self.scales.size and self.bounds[j] < stop:
            lo = max(start, int(self.bounds[j]))
            hi = min(stop, int(self.bounds[j + 1]))
            o[lo - start:hi - start] *= self.scales[j]
            j += 1

    def gradient(self, t: int, worker: int = 0, start: int = 0, stop: int | None = None,
                 out: np.ndarray | None = None, threads: int = 1) -> np.ndarray:
        """g_{worker,t}[start:stop] as float32 (blocks drawn by `threads` threads)."""
        d = self.w.d
        stop = d if stop is None else stop
        assert 0 <= start <= stop <= d
        if out is None:
            out = np.empty(stop - start, dtype=np.float32)
        b0 = start // BLOCK
        b1 = (stop + BLOCK - 1) // BLOCK

        def one(b):
            bs = b * BLOCK
            be = min(d, bs + BLOCK)
            lo, hi = max(start, bs), min(stop, be)
            if lo == bs and hi == be:
                self._fill_block(worker, t, b, out[lo - start:hi - start])
            else:
                tmp = np.empty(be - bs, dtype=np.float32)
                self._fill_block(worker, t, b, tmp)
                out[lo - start:hi - start] = tmp[lo - bs:hi - bs]

        if threads > 1 and b1 - b0 > 1:
            from concurrent.futures import ThreadPoolExecutor
            with ThreadPoolExecutor(threads) as ex:
                list(ex.map(one, range(b0, b1)))
        else:
            for b in range(b0, b1):
                one(b)
        return out


def small_gradient(seed: int, d: int, scale: float = 1e-3) -> np.ndarray:
    """A small Gaussian vector for unit and parity tests."""
    rng = _rng(9, seed, d, 3)
    return (rng.standard_normal(d, dtype=np.float32) * np.float32(scale))


def long_gradient(seed: int, d: int, scale: float = 1e-3, threads: int = 1) -> np.ndarray:
    """A Gaussian vector of any length (tests up to 2^31 - 1 elements),
    N(0, scale^2) in float32, drawn per BLOCK elements each from its own
    seed, `threads` blocks at a time."""
    out = np.empty(d, dtype=np.float32)

    def one(b):
        lo, hi = b * BLOCK, min(d, (b + 1) * BLOCK)
        _rng(10, seed, b).standard_normal(out=out[lo:hi], dtype=np.float32)
        out[lo:hi] *= np.float32(scale)

    blocks = range((d + BLOCK - 1) // BLOCK)
    if threads > 1:
        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(one, blocks))
    else:
        for b in blocks:
            one(b)
    return out


LAMBDA_FILE = "workload_lambdas.json"


def stored_lambda(workload_id: int, density: float, worker: int = 0) -> np.float32:
    """The threshold of a workload at a first-step density, as stored by the
    oracle's calibration script (the K-th largest |fl(lr * g_0)| of that
    workload's first gradient, K = round(density * d)), bit for bit."""
    import json
    import os
    path = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                        "tests", "golden", LAMBDA_FILE)
    with open(path) as f:
        table = json.load(f)
    key = "%d/%g/%d" % (workload_id, density, worker)
    if key not in table["lambda_bits"]:
        raise KeyError("no stored threshold for workload %d at density %g (worker %d)"
                       % (workload_id, density, worker))
    return np.array([table["lambda_bits"][key]], dtype=np.uint32).view(np.float32)[0]


def lambda_from_k(k: int) -> float:
    """Tuning rule lambda ~ 1/(2 sqrt(k)) of Appendix D (used for Table 5)."""
    return 1.0 / (2.0 * math.sqrt(k))


def lambda_in_update_units(lam_paper: float, lr=LR) -> np.float32:
    """Algorithm 1 compresses p/gamma; its threshold in units of p is gamma*lambda."""
    return np.float32(np.float32(lr) * np.float32(lam_paper))


def layerwise_k(bounds, density: float) -> np.ndarray:
    """Per-layer budgets for layer-wise Top-k at a density: k_s = ceil(rho d_s)
    for each segment [bounds[s], bounds[s+1]) (at least one coordinate of a
    non-empty segment, never more than the segment holds)."""
    sizes = np.diff(np.asarray(bounds, dtype=np.int64))
    k = np.ceil(sizes * float(density)).astype(np.int64)
    return np.minimum(np.maximum(k, (sizes > 0).astype(np.int64)), sizes)
