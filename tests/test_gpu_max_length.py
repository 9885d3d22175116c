"""GPU parity at the largest vector length the ABI takes, d = 2^31 - 1
(int32 indices; 8.6 GB per fp32 vector): the hard threshold over two
error-feedback steps with its telemetry, the flat Top-k on its radix path
and then from its bracket, the layer-wise Top-k over five layers (first
call and a later one from the brackets), the average of the first two
payloads and the same average fused with the momentum update, each against
the oracle chunk by chunk.  Large magnitudes are planted at the last elements of the
vector (the ragged last tile) and around the last 4096-element boundary, so
that pairs with the largest indices are kept."""
import os
import time

import numpy as np
import pytest

from paper_2108_00951_amd import synth
from tests._checks import assert_bits_equal, assert_payload_equal, canonical, check_topk_chunked

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import oracle  # noqa: E402
from paper_2108_00951_amd import binding as efs  # noqa: E402

DEV = "cuda"
LR = synth.LR
D = 2 ** 31 - 1
CHUNK = 1 << 26
THREADS = min(16, os.cpu_count() or 1)


def say(t0, *a):
    print("[%6.1fs]" % (time.time() - t0), *a, flush=True)


def to_dev(host):
    out = torch.empty(host.size, dtype=torch.float32, device=DEV)
    for lo in range(0, host.size, CHUNK):
        out[lo:lo + CHUNK].copy_(torch.from_numpy(host[lo:lo + CHUNK]))
    return out


def test_vector_of_two_to_the_31_minus_one_elements():
    t0 = time.time()
    g = synth.long_gradient(31, D, threads=THREADS)
    last_block = (D // 4096) * 4096
    plant = np.array([D - 1, D - 2, D - 3, last_block, last_block - 1, D - 4096, 0, 1])
    g[plant] = np.array([0.9, -0.8, 0.7, -0.6, 0.5, -0.45, 0.4, -0.35], dtype=np.float32)
    g_dev = to_dev(g)
    say(t0, "g on the device, d=%d" % D)

    # hard threshold, two steps with e carried (the same gradient twice)
    # 4.4 sigma of lr*g at the first step (about 23,000 pairs), 2.2 sigma at the
    # second, where p is about 2 lr g (about 60 M pairs)
    lam = np.float32(4.4e-4)
    cap = 1 << 27
    e = torch.zeros(D, dtype=torch.float32, device=DEV)
    idx = torch.empty(cap, dtype=torch.int32, device=DEV)
    val = torch.empty(cap, dtype=torch.float32, device=DEV)
    ctr = efs.new_counter(DEV)
    e_ref = np.zeros(D, np.float32)
    payload0 = None
    tel = efs.new_telemetry(DEV)
    err2, sent, maxbits = 0.0, 0, 0
    for t in range(2):
        efs.ht_compress_telemetry(g_dev, e, LR, lam, idx, val, ctr, tel)
        n = efs.counter_value(ctr)
        assert n <= cap
        gi, gv = canonical(idx[:n].cpu().numpy(), val[:n].cpu().numpy())
        if t == 0:
            payload0 = (gi.copy(), gv.copy())
        assert np.all(np.isin(plant, gi)), "a planted magnitude was not kept"
        total = 0
        for lo in range(0, D, CHUNK):
            hi = min(D, lo + CHUNK)
            ri, rv, e_chunk, rk = oracle.ht(g[lo:hi], e_ref[lo:hi], LR, lam, cap=hi - lo, mt=True)
            e_ref[lo:hi] = e_chunk
            a, b = np.searchsorted(gi, [lo, hi])
            assert_payload_equal(gi[a:b] - lo, gv[a:b], ri, rv, "ht t=%d chunk %d" % (t, lo))
            assert_bits_equal(e[lo:hi].cpu().numpy(), e_chunk, "ht e' t=%d chunk %d" % (t, lo))
            total += rk
            err2 += float(np.sum(e_chunk.astype(np.float64) ** 2))
            maxbits = max(maxbits, int(np.max(e_chunk.view(np.uint32) & np.uint32(0x7FFFFFFF))))
        assert n == total
        sent += n
        say(t0, "hard threshold t=%d: k_t=%d, last index %d" % (t, n, gi[-1]))
    got = efs.read_telemetry(tel)
    assert got["calls"] == 2 and got["sent_total"] == sent
    assert got["max_abs_bits"] == maxbits
    assert abs(got["err2_total"] - err2) <= 1e-9 * err2
    say(t0, "telemetry ok: sum ||e'||^2 %.6g, max |e'| %.6g" % (err2, got["max_abs"]))
    del e, e_ref, idx, val
    torch.cuda.empty_cache()

    # Top-k: the radix path from a zeroed workspace, then error feedback on
    # the same workspace until a call selects from the bracket
    k = 1000
    et = torch.zeros(D, dtype=torch.float32, device=DEV)
    tidx = torch.empty(k, dtype=torch.int32, device=DEV)
    tval = torch.empty(k, dtype=torch.float32, device=DEV)
    ws = efs.new_topk_workspace(D, k, DEV)
    ws.zero_()
    zeros = np.zeros(CHUNK, np.float32)
    efs.topk_compress(g_dev, et, LR, k, tidx, tval, ws)
    assert not efs.topk_took_bracket_path(ws)
    ti, tv = tidx.cpu().numpy(), tval.cpu().numpy()
    assert np.all(np.isin(plant, ti))
    check_topk_chunked(
        D, k, ti, tv,
        acc_fn=lambda lo, hi: oracle.ht(g[lo:hi], zeros[:hi - lo], LR, np.inf, cap=0, mt=True)[2],
        e_next_fn=lambda lo, hi: et[lo:hi].cpu().numpy(), chunk=CHUNK)
    payload1 = canonical(ti, tv)
    say(t0, "Top-k radix path ok")
    e_before = torch.empty_like(et)
    for t in range(1, 9):
        e_before.copy_(et)
        efs.topk_compress(g_dev, et, LR, k, tidx, tval, ws)
        if efs.topk_took_bracket_path(ws):
            break
    assert efs.topk_took_bracket_path(ws), "no call took the bracket path"
    check_topk_chunked(
        D, k, tidx.cpu().numpy(), tval.cpu().numpy(),
        acc_fn=lambda lo, hi: oracle.ht(g[lo:hi], e_before[lo:hi].cpu().numpy(), LR, np.inf,
                                        cap=0, mt=True)[2],
        e_next_fn=lambda lo, hi: et[lo:hi].cpu().numpy(), chunk=CHUNK)
    say(t0, "Top-k bracket path ok (call %d)" % t)
    del et, ws
    torch.cuda.empty_cache()

    # layer-wise Top-k: a one-element layer, a light two-tile layer, a
    # one-tile layer and two layers of about 10^9 elements; the first call
    # ranks every layer by its radix path, a later call (e carried) selects
    # the large layers from their brackets; each layer checked chunk by chunk
    off = np.array([0, 1, 1 + 4097, 1 + 4097 + 1000, 1_000_000_000, D], dtype=np.int64)
    ks = np.array([1, 10, 5, 700, 1500], dtype=np.int64)
    kt = int(ks.sum())
    es = torch.zeros(D, dtype=torch.float32, device=DEV)
    sidx = torch.empty(kt, dtype=torch.int32, device=DEV)
    sval = torch.empty(kt, dtype=torch.float32, device=DEV)
    sws = efs.new_topk_segmented_workspace(ks.size, kt, DEV)
    sws.zero_()
    offd, kd = torch.from_numpy(off).to(DEV), torch.from_numpy(ks).to(DEV)

    def check_layers(prev, what):
        gi, gv = sidx.cpu().numpy(), sval.cpu().numpy()
        pos = 0
        for s_ in range(ks.size):
            lo_s, hi_s, k_s = int(off[s_]), int(off[s_ + 1]), int(ks[s_])
            check_topk_chunked(
                hi_s - lo_s, k_s, gi[pos:pos + k_s] - lo_s, gv[pos:pos + k_s],
                acc_fn=lambda lo, hi: oracle.ht(g[lo_s + lo:lo_s + hi], prev(lo_s + lo, lo_s + hi), LR,
                                                np.inf, cap=0, mt=True)[2],
                e_next_fn=lambda lo, hi: es[lo_s + lo:lo_s + hi].cpu().numpy(), chunk=CHUNK)
            pos += k_s
        say(t0, "layer-wise %s ok (bracket in %d layers)" % (what, efs.topk_segmented_bracket_segments(sws)))

    efs.topk_segmented_compress(g_dev, es, LR, offd, kd, sidx, sval, sws)
    assert efs.topk_segmented_status(sws) == 0
    check_layers(lambda lo, hi: zeros[:hi - lo], "first call")
    for t in range(1, 9):
        e_before.copy_(es)
        efs.topk_segmented_compress(g_dev, es, LR, offd, kd, sidx, sval, sws)
        if efs.topk_segmented_bracket_segments(sws) >= 2:
            break
    assert efs.topk_segmented_bracket_segments(sws) >= 2, "the large layers never used their brackets"
    check_layers(lambda lo, hi: e_before[lo:hi].cpu().numpy(), "call %d" % t)
    del es, e_before, sws, g_dev
    torch.cuda.empty_cache()

    # the average of the two payloads over d = 2^31 - 1 coordinates
    ps = [(torch.from_numpy(p[0]).to(DEV), torch.from_numpy(p[1]).to(DEV)) for p in (payload0, payload1)]
    out = torch.empty(D, dtype=torch.float32, device=DEV)
    aws = efs.new_apply_workspace(ps, D, DEV, layout="packed")
    efs.sparse_accumulate(ps, D, out, aws)
    assert efs.sparse_status(aws) == 0
    ref = oracle.accumulate([payload0, payload1], D)
    for lo in range(0, D, CHUNK):
        assert_bits_equal(out[lo:lo + CHUNK].cpu().numpy(), ref[lo:lo + CHUNK], "average chunk %d" % lo)
    say(t0, "average of the two payloads ok")
    del out, ref
    torch.cuda.empty_cache()

    # the same average fused with the momentum update of Algorithm 2
    m_host = synth.long_gradient(32, D, threads=THREADS)
    x_dev, m_dev = to_dev(g), to_dev(m_host)
    efs.sparse_apply(ps, D, efs.APPLY_MOMENTUM, x_dev, aws, m=m_dev, beta=0.9, gamma=0.05)
    assert efs.sparse_status(aws) == 0
    rx, rm = oracle.update([payload0, payload1], g, 2, m=m_host, beta=0.9, gamma=0.05)
    for lo in range(0, D, CHUNK):
        assert_bits_equal(m_dev[lo:lo + CHUNK].cpu().numpy(), rm[lo:lo + CHUNK], "m chunk %d" % lo)
        assert_bits_equal(x_dev[lo:lo + CHUNK].cpu().numpy(), rx[lo:lo + CHUNK], "x chunk %d" % lo)
    say(t0, "momentum update ok")
