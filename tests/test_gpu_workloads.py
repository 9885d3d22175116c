"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times (the same entry points, grid sizing and vector path).

Hard threshold: every output against the oracle (streamed in chunks for the
1.5e9-element vector, which the element-wise definition allows).  Top-k: the
oracle's qsort definition at the 1e6 size and once at 25.6e6; at every size
the properties that fix the Top-k payload uniquely (check_topk_properties /
check_topk_chunked).  Average: against the oracle, bit for bit.
"""
import os
import time

import numpy as np
import pytest

import oracle
from paper_2108_00951_amd import synth
from tests._checks import (assert_bits_equal, assert_payload_equal, canonical,
                           check_topk_chunked, check_topk_properties)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2108_00951_amd import binding as efs  # noqa: E402

DEV = "cuda"
LR = synth.LR
THREADS = min(16, os.cpu_count() or 1)
T0 = time.time()


def say(*a):
    print("[%6.1fs]" % (time.time() - T0), *a, flush=True)


def _repeat_topk_from_the_bracket(tk, g_dev, k):
    """Repeats the last Top-k call of `tk` from e = 0 on the same workspace
    (its threshold is recorded there, so the call selects from the bracket)
    and checks the result equals the last call's bit for bit."""
    first_i, first_v = tk.payload(k)
    first_e = tk.e.cpu().numpy()
    tk.e.zero_()
    tk.topk(g_dev, k)
    assert efs.topk_took_bracket_path(tk.ws)
    gi, gv = tk.payload(k)
    o1, o2 = np.argsort(first_i), np.argsort(gi)
    np.testing.assert_array_equal(gi[o2], first_i[o1])
    assert_bits_equal(gv[o2], first_v[o1], "values from the bracket")
    assert_bits_equal(tk.e.cpu().numpy(), first_e, "e' from the bracket")


class Worker:
    """Hard-threshold and Top-k EF state of one worker on the device."""

    def __init__(self, d, cap, k=None):
        self.d = d
        self.cap = cap
        self.e = torch.zeros(d, dtype=torch.float32, device=DEV)
        self.idx = torch.empty(cap, dtype=torch.int32, device=DEV)
        self.val = torch.empty(cap, dtype=torch.float32, device=DEV)
        self.ctr = efs.new_counter(DEV)
        if k is not None:
            self.ws = efs.new_topk_workspace(d, k, DEV)

    def ht(self, g_dev, lam):
        efs.ht_compress(g_dev, self.e, LR, lam, self.idx, self.val, self.ctr)
        k = efs.counter_value(self.ctr)
        assert k <= self.cap, "payload capacity %d exceeded (k_t=%d)" % (self.cap, k)
        return k

    def topk(self, g_dev, k):
        efs.topk_compress(g_dev, self.e, LR, k, self.idx[:k], self.val[:k], self.ws)

    def payload(self, n):
        return self.idx[:n].cpu().numpy(), self.val[:n].cpu().numpy()


def test_workload1_gauss_1m_all_iterations():
    st = synth.Stream(1)
    w = st.w
    gs = [st.gradient(t) for t in range(w.iters)]
    lam = oracle.calibrate_lambda(gs[0], w.densities[0])
    k = w.topk_k[0]
    ht, tk = Worker(w.d, w.d), Worker(w.d, k, k=k)
    e_ht = np.zeros(w.d, np.float32)
    e_tk = np.zeros(w.d, np.float32)
    for t, g in enumerate(gs):
        g_dev = torch.from_numpy(g).to(DEV)
        n = ht.ht(g_dev, lam)
        ri, rv, e_ht, rk = oracle.ht(g, e_ht, LR, lam)
        assert n == rk
        if t == 0:
            assert rk == int(round(w.densities[0] * w.d))
        assert_payload_equal(*ht.payload(n), ri, rv, "ht t=%d" % t)
        assert_bits_equal(ht.e.cpu().numpy(), e_ht, "ht e' t=%d" % t)
        tk.topk(g_dev, k)
        ri, rv, e_tk = oracle.topk(g, e_tk, LR, k)
        assert_payload_equal(*tk.payload(k), ri, rv, "topk t=%d" % t)
        assert_bits_equal(tk.e.cpu().numpy(), e_tk, "topk e' t=%d" % t)
    say("workload 1: %d iterations, last k_t=%d" % (w.iters, rk))


def test_workload2_segments_25m():
    st = synth.Stream(2)
    w = st.w
    T = 4
    gs = [st.gradient(t, threads=THREADS) for t in range(T)]
    lam = oracle.calibrate_lambda(gs[0], w.densities[0])
    k = w.topk_k[0]
    ht, tk = Worker(w.d, w.d), Worker(w.d, k, k=k)
    e_ht = np.zeros(w.d, np.float32)
    e_tk = np.zeros(w.d, np.float32)
    for t, g in enumerate(gs):
        g_dev = torch.from_numpy(g).to(DEV)
        n = ht.ht(g_dev, lam)
        ri, rv, e_ht, rk = oracle.ht(g, e_ht, LR, lam)
        assert n == rk
        assert_payload_equal(*ht.payload(n), ri, rv, "ht t=%d" % t)
        assert_bits_equal(ht.e.cpu().numpy(), e_ht, "ht e' t=%d" % t)
        acc = oracle.ht(g, e_tk, LR, np.inf)[2]
        tk.topk(g_dev, k)
        gi, gv = tk.payload(k)
        e_tk = tk.e.cpu().numpy()
        if t == 0:
            ri, rv, re = oracle.topk(g, np.zeros(w.d, np.float32), LR, k)
            assert_payload_equal(gi, gv, ri, rv, "topk t=0 vs oracle")
            assert_bits_equal(e_tk, re, "topk e' t=0")
            _repeat_topk_from_the_bracket(tk, g_dev, k)
        check_topk_properties(acc, k, gi, gv, e_tk)
        say("workload 2 t=%d: ht k_t=%d, topk ok" % (t, n))


def _segmented(d, bounds, ks):
    """Device buffers for layer-wise Top-k over the given layout."""
    k_total = int(ks.sum())
    return dict(off=torch.from_numpy(np.asarray(bounds, np.int64)).to(DEV),
                k=torch.from_numpy(np.asarray(ks, np.int64)).to(DEV),
                idx=torch.empty(k_total, dtype=torch.int32, device=DEV),
                val=torch.empty(k_total, dtype=torch.float32, device=DEV),
                ws=efs.new_topk_segmented_workspace(len(ks), k_total, DEV),
                e=torch.zeros(d, dtype=torch.float32, device=DEV))


def _check_segments(acc, bounds, ks, gi, gv, e_next):
    pos = 0
    for s in range(len(ks)):
        lo, hi, n = int(bounds[s]), int(bounds[s + 1]), int(ks[s])
        check_topk_properties(acc[lo:hi], n, gi[pos:pos + n] - lo, gv[pos:pos + n], e_next[lo:hi])
        pos += n


def _bracket_eligible(bounds, ks):
    """Segments that can select from a bracket: more than one 4096-element
    tile and 0 < k < size."""
    lo, hi = np.asarray(bounds[:-1], np.int64), np.asarray(bounds[1:], np.int64)
    size = hi - lo
    tiles = np.where(size > 0, (hi - 1) // 4096 - lo // 4096 + 1, 0)
    return int(np.sum((tiles > 1) & (ks > 0) & (ks < size)))


def _repeat_from_the_bracket(g_dev, b, ks, bounds):
    """Runs the call of `b` again from e = 0 on the same workspace: the
    threshold of each segment is the one the last call recorded, so the
    segments select from the bracket; the result must equal the last call's
    bit for bit (results never depend on the path)."""
    first_i, first_v, first_e = (b["idx"].cpu().numpy(), b["val"].cpu().numpy(),
                                 b["e"].cpu().numpy())
    b["e"].zero_()
    efs.topk_segmented_compress(g_dev, b["e"], LR, b["off"], b["k"], b["idx"], b["val"], b["ws"])
    assert efs.topk_segmented_status(b["ws"]) == 0
    hits = efs.topk_segmented_bracket_segments(b["ws"])
    gi, gv, ge = b["idx"].cpu().numpy(), b["val"].cpu().numpy(), b["e"].cpu().numpy()
    pos = 0
    for s in range(len(ks)):
        n = int(ks[s])
        o1, o2 = np.argsort(first_i[pos:pos + n]), np.argsort(gi[pos:pos + n])
        np.testing.assert_array_equal(gi[pos:pos + n][o2], first_i[pos:pos + n][o1],
                                      "segment %d" % s)
        assert_bits_equal(gv[pos:pos + n][o2], first_v[pos:pos + n][o1], "segment %d" % s)
        pos += n
    assert_bits_equal(ge, first_e, "e' from the bracket")
    eligible = _bracket_eligible(bounds, ks)
    say("  repeated from the bracket: %d of %d eligible segments" % (hits, eligible))
    assert hits >= 0.9 * eligible


def test_workload2_layerwise_topk():
    # layer-wise Top-k over the 161 segments, k_s = ceil(0.1 % of d_s), e
    # carried for three steps: the oracle at t = 0 and 1, properties after
    st = synth.Stream(2)
    w = st.w
    ks = synth.layerwise_k(st.bounds, w.densities[0])
    b = _segmented(w.d, st.bounds, ks)
    e_ref = np.zeros(w.d, np.float32)
    for t in range(3):
        g = st.gradient(t, threads=THREADS)
        acc = oracle.ht(g, e_ref, LR, np.inf)[2]
        efs.topk_segmented_compress(torch.from_numpy(g).to(DEV), b["e"], LR, b["off"], b["k"],
                                    b["idx"], b["val"], b["ws"])
        assert efs.topk_segmented_status(b["ws"]) == 0
        gi, gv, ge = b["idx"].cpu().numpy(), b["val"].cpu().numpy(), b["e"].cpu().numpy()
        if t < 2:
            ri, rv, re = oracle.topk_segmented(g, e_ref, LR, st.bounds, ks)
            pos = 0
            for s in range(ks.size):
                n = int(ks[s])
                assert_payload_equal(gi[pos:pos + n], gv[pos:pos + n], ri[pos:pos + n],
                                     rv[pos:pos + n], "segment %d t=%d" % (s, t))
                pos += n
            assert_bits_equal(ge, re, "layer-wise e' t=%d" % t)
        _check_segments(acc, st.bounds, ks, gi, gv, ge)
        say("workload 2 layer-wise t=%d: %d pairs in %d segments ok" % (t, ks.sum(), ks.size))
        if t == 0:
            # the oracle-checked first call, repeated from the bracket
            _repeat_from_the_bracket(torch.from_numpy(g).to(DEV), b, ks, st.bounds)
        e_ref = b["e"].cpu().numpy()


def test_workload3_layerwise_topk():
    # 110e6 elements in 200 segments at 1 % and 0.01 % per segment
    st = synth.Stream(3)
    w = st.w
    g = st.gradient(0, threads=THREADS)
    acc = oracle.ht(g, np.zeros(w.d, np.float32), LR, np.inf)[2]   # p with e = 0
    g_dev = torch.from_numpy(g).to(DEV)
    for rho in (0.01, 0.0001):
        ks = synth.layerwise_k(st.bounds, rho)
        b = _segmented(w.d, st.bounds, ks)
        efs.topk_segmented_compress(g_dev, b["e"], LR, b["off"], b["k"], b["idx"], b["val"],
                                    b["ws"])
        assert efs.topk_segmented_status(b["ws"]) == 0
        _check_segments(acc, st.bounds, ks, b["idx"].cpu().numpy(), b["val"].cpu().numpy(),
                        b["e"].cpu().numpy())
        say("workload 3 layer-wise rho=%g: %d pairs ok" % (rho, ks.sum()))
        _repeat_from_the_bracket(g_dev, b, ks, st.bounds)
        del b
        torch.cuda.empty_cache()


def test_workload3_student_t_110m():
    st = synth.Stream(3)
    w = st.w
    gs = [st.gradient(t, threads=THREADS) for t in range(2)]
    say("workload 3 inputs ready")
    g_devs = [torch.from_numpy(g).to(DEV) for g in gs]
    for density, k in zip(w.densities, w.topk_k):
        lam = oracle.calibrate_lambda(gs[0], density)
        ht = Worker(w.d, w.d // 8)
        e_ht = np.zeros(w.d, np.float32)
        for t in range(2):
            n = ht.ht(g_devs[t], lam)
            ri, rv, e_ht, rk = oracle.ht(gs[t], e_ht, LR, lam, cap=w.d // 8)
            assert n == rk
            assert_payload_equal(*ht.payload(n), ri, rv, "ht rho=%g t=%d" % (density, t))
            assert_bits_equal(ht.e.cpu().numpy(), e_ht, "ht e' rho=%g t=%d" % (density, t))
        del ht
        tk = Worker(w.d, k, k=k)
        acc = oracle.ht(gs[0], np.zeros(w.d, np.float32), LR, np.inf)[2]
        tk.topk(g_devs[0], k)
        check_topk_properties(acc, k, *tk.payload(k), tk.e.cpu().numpy())
        _repeat_topk_from_the_bracket(tk, g_devs[0], k)
        del tk, acc
        say("workload 3 rho=%g: ht k_t=%d, topk k=%d ok" % (density, n, k))


def test_workload4_eight_workers_average():
    st = synth.Stream(4)
    w = st.w
    lam = oracle.calibrate_lambda(st.gradient(0, worker=0, threads=THREADS), w.densities[0])
    workers = [Worker(w.d, w.d // 4) for _ in range(w.n_workers)]
    e_ref = [np.zeros(w.d, np.float32) for _ in range(w.n_workers)]
    out = torch.empty(w.d, dtype=torch.float32, device=DEV)
    # model state for the fused update (Algorithm 2's momentum form and
    # Algorithm 1's x - avg on a copy)
    rng = np.random.default_rng(4)
    x_ref = rng.standard_normal(w.d).astype(np.float32)
    m_ref = np.zeros(w.d, np.float32)
    x, m = torch.from_numpy(x_ref).to(DEV), torch.from_numpy(m_ref).to(DEV)
    p_dev = [(o.idx, o.val, o.ctr) for o in workers]
    ws = efs.new_apply_workspace(p_dev, w.d, DEV)
    for t in range(2):
        payloads = []
        for wk in range(w.n_workers):
            g = st.gradient(t, worker=wk, threads=THREADS)
            n = workers[wk].ht(torch.from_numpy(g).to(DEV), lam)
            ri, rv, e_ref[wk], rk = oracle.ht(g, e_ref[wk], LR, lam)
            assert n == rk
            gi, gv = workers[wk].payload(n)
            assert_payload_equal(gi, gv, ri, rv, "worker %d t=%d" % (wk, t))
            # the device payload, in its own (unspecified) order, is what is averaged
            payloads.append((gi, gv))
        efs.sparse_accumulate(p_dev, w.d, out, ws)
        ref = oracle.accumulate(payloads, w.d)
        assert_bits_equal(out.cpu().numpy(), ref, "average t=%d" % t)
        assert efs.sparse_status(ws) == 0
        say("workload 4 t=%d: 8 workers averaged, k_t=%s" % (
            t, [efs.counter_value(o.ctr) for o in workers]))
        x_sgd = x.clone()
        efs.sparse_apply(p_dev, w.d, efs.APPLY_SGD, x_sgd, ws)
        want_sgd, _ = oracle.update(payloads, x_ref, 1)
        assert_bits_equal(x_sgd.cpu().numpy(), want_sgd, "sgd update t=%d" % t)
        del x_sgd, want_sgd
        efs.sparse_apply(p_dev, w.d, efs.APPLY_MOMENTUM, x, ws, m=m, beta=0.9, gamma=0.05)
        x_ref, m_ref = oracle.update(payloads, x_ref, 2, m=m_ref, beta=0.9, gamma=0.05)
        assert_bits_equal(m.cpu().numpy(), m_ref, "momentum m t=%d" % t)
        assert_bits_equal(x.cpu().numpy(), x_ref, "momentum x t=%d" % t)
        say("workload 4 t=%d: fused sgd and momentum updates ok" % t)


@pytest.mark.timeout(900)
def test_workload5_outliers_1_5b_streamed():
    st = synth.Stream(5)
    w = st.w
    d = w.d
    chunk = 1 << 26
    say("workload 5: drawing g_0 (%d elements)" % d)
    g = st.gradient(0, threads=THREADS)
    lam = synth.stored_lambda(5, w.densities[0])
    g_dev = torch.empty(d, dtype=torch.float32, device=DEV)
    for lo in range(0, d, chunk):
        g_dev[lo:lo + chunk].copy_(torch.from_numpy(g[lo:lo + chunk]))
    say("workload 5: g_0 on device, lambda=%g" % float(lam))

    # hard threshold, two iterations (e carried), streamed comparison
    cap = 1 << 26
    ht = Worker(d, cap)
    e_ref = np.zeros(d, np.float32)
    for t in range(2):
        if t == 1:
            g = st.gradient(1, threads=THREADS)
            for lo in range(0, d, chunk):
                g_dev[lo:lo + chunk].copy_(torch.from_numpy(g[lo:lo + chunk]))
        n = ht.ht(g_dev, lam)
        gi, gv = canonical(*ht.payload(n))
        total = 0
        for lo in range(0, d, chunk):
            hi = min(d, lo + chunk)
            ri, rv, e_chunk, rk = oracle.ht(g[lo:hi], e_ref[lo:hi], LR, lam, cap=hi - lo)
            e_ref[lo:hi] = e_chunk
            a, b = np.searchsorted(gi, [lo, hi])
            assert_payload_equal(gi[a:b] - lo, gv[a:b], ri, rv, "ht t=%d chunk %d" % (t, lo))
            assert_bits_equal(ht.e[lo:hi].cpu().numpy(), e_chunk, "ht e' t=%d chunk %d" % (t, lo))
            total += rk
        assert n == total
        if t == 0:
            assert n == w.topk_k[0]   # the stored lambda keeps exactly K at the first step
        say("workload 5 ht t=%d: k_t=%d matches" % (t, n))
    del ht, e_ref

    # Top-k on g_1 from e = 0 (the acc is then fl(lr * g_1)): the radix path
    k = w.topk_k[0]
    tk = Worker(d, k, k=k)
    tk.ws.zero_()    # no threshold recorded yet
    tk.topk(g_dev, k)
    assert not efs.topk_took_bracket_path(tk.ws)
    gi, gv = tk.payload(k)
    zeros = np.zeros(chunk, np.float32)
    check_topk_chunked(
        d, k, gi, gv,
        acc_fn=lambda lo, hi: oracle.ht(g[lo:hi], zeros[:hi - lo], LR, np.inf, cap=0, mt=True)[2],
        e_next_fn=lambda lo, hi: tk.e[lo:hi].cpu().numpy(),
        chunk=chunk)
    say("workload 5 topk k=%d ok (radix path)" % k)

    # Error feedback on the same workspace: e carried, the same gradient
    # again, so the threshold drifts up steadily and a later call selects
    # from the bracket around the extrapolated threshold (24 M candidate
    # slots, 64-bit offsets).  That call is checked in full.
    e_before = torch.empty_like(tk.e)
    for t in range(1, 9):
        e_before.copy_(tk.e)
        tk.topk(g_dev, k)
        if efs.topk_took_bracket_path(tk.ws):
            break
    assert efs.topk_took_bracket_path(tk.ws), "no call took the bracket path"
    say("workload 5 topk call %d took the bracket path; checking it" % t)
    gi, gv = tk.payload(k)
    check_topk_chunked(
        d, k, gi, gv,
        acc_fn=lambda lo, hi: oracle.ht(g[lo:hi], e_before[lo:hi].cpu().numpy(), LR, np.inf,
                                        cap=0, mt=True)[2],
        e_next_fn=lambda lo, hi: tk.e[lo:hi].cpu().numpy(),
        chunk=chunk)
    say("workload 5 topk k=%d ok (bracket path, call %d)" % (k, t))
