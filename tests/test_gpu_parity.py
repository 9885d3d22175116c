"""GPU parity: the HIP path through the C ABI against the CPU oracle, element
by element, at sizes that span many 4096-element tiles and ragged tails,
plus the edge cases of the method.  Bit-exact throughout: indices, counts,
values and residuals are integer or copy results of one fp32 mul and add
that both sides round the same way; the average is an in-order fp32 sum
divided once, bit-exact as well (the 1e-6 relative bound is never needed).
"""
import numpy as np
import pytest

import oracle
from paper_2108_00951_amd import synth
from tests._checks import (assert_bits_equal, assert_payload_equal, bits, canonical,
                           check_topk_properties)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2108_00951_amd import binding as efs  # noqa: E402

LR = np.float32(0.1)
DEV = "cuda"


def say(*a):
    print(*a, flush=True)


def to_dev(a, unaligned=False):
    """Copy a host array to the device; unaligned=True offsets it by one
    element so the 16-byte vector path is not taken."""
    a = np.ascontiguousarray(a)
    if not unaligned:
        return torch.from_numpy(a).to(DEV)
    buf = torch.empty(a.size + 1, dtype=torch.from_numpy(a[:0]).dtype, device=DEV)
    v = buf[1:]
    v.copy_(torch.from_numpy(a))
    return v


class HT:
    """One worker's hard-threshold EF state on the device."""

    def __init__(self, d, cap=None, unaligned=False):
        self.d = d
        self.cap = d if cap is None else cap
        self.e = to_dev(np.zeros(d, dtype=np.float32), unaligned)
        self.idx = torch.empty(max(self.cap, 1), dtype=torch.int32, device=DEV)[:self.cap]
        self.val = torch.empty(max(self.cap, 1), dtype=torch.float32, device=DEV)[:self.cap]
        self.ctr = efs.new_counter(DEV)
        self.unaligned = unaligned

    def step(self, g_host, lam, lr=LR):
        g = to_dev(g_host, self.unaligned)
        efs.ht_compress(g, self.e, lr, lam, self.idx, self.val, self.ctr)
        k = efs.counter_value(self.ctr)
        n = min(k, self.cap)
        return self.idx[:n].cpu().numpy(), self.val[:n].cpu().numpy(), self.e.cpu().numpy(), k


def topk_gpu(g_host, e_host, k, lr=LR, unaligned=False):
    d = g_host.size
    g = to_dev(g_host, unaligned)
    e = to_dev(e_host, unaligned)
    idx = torch.empty(max(k, 1), dtype=torch.int32, device=DEV)[:k]
    val = torch.empty(max(k, 1), dtype=torch.float32, device=DEV)[:k]
    ws = efs.new_topk_workspace(d, k, DEV)
    efs.topk_compress(g, e, lr, k, idx, val, ws)
    return idx.cpu().numpy(), val.cpu().numpy(), e.cpu().numpy()


SIZES = [1, 3, 63, 64, 65, 1023, 4095, 4096, 4097, 8191, 12_289, 100_003, 1_000_000]


@pytest.mark.parametrize("unaligned", [False, True])
@pytest.mark.parametrize("d", SIZES)
def test_ht_ef_loop_matches_oracle(d, unaligned):
    say("ht parity d=%d unaligned=%s" % (d, unaligned))
    gs = [synth.small_gradient(10 + t, d) for t in range(3)]
    lam = oracle.calibrate_lambda(gs[0], 0.01)
    st = HT(d, unaligned=unaligned)
    e_ref = np.zeros(d, dtype=np.float32)
    for t in range(3):
        gi, gv, ge, gk = st.step(gs[t], lam)
        ri, rv, e_ref, rk = oracle.ht(gs[t], e_ref, LR, lam)
        assert gk == rk
        assert_payload_equal(gi, gv, ri, rv, "t=%d" % t)
        assert_bits_equal(ge, e_ref, "e' t=%d" % t)


@pytest.mark.parametrize("unaligned", [False, True])
def test_ht_long_sweep(unaligned):
    # 34 tiles per workgroup and a ragged last tile (the sweeps of 256 tiles
    # per workgroup and more, walked XCD by XCD, are checked on the 1.5e9
    # workload)
    d = 70_000_003
    say("ht parity long sweep d=%d unaligned=%s" % (d, unaligned))
    gs = [synth.small_gradient(20 + t, d) for t in range(2)]
    lam = oracle.calibrate_lambda(gs[0], 0.001)
    st = HT(d, cap=d // 8, unaligned=unaligned)
    e_ref = np.zeros(d, dtype=np.float32)
    for t in range(2):
        gi, gv, ge, gk = st.step(gs[t], lam)
        ri, rv, e_ref, rk = oracle.ht(gs[t], e_ref, LR, lam, mt=True)
        assert gk == rk
        assert_payload_equal(gi, gv, ri, rv, "t=%d" % t)
        assert_bits_equal(ge, e_ref, "e' t=%d" % t)


def test_ht_lambda_zero_and_infinity():
    d = 70_001
    g = synth.small_gradient(1, d)
    g[17] = np.float32(-0.0)
    st = HT(d)
    gi, gv, ge, gk = st.step(g, 0.0)
    ri, rv, re, rk = oracle.ht(g, np.zeros(d, np.float32), LR, 0.0)
    assert gk == rk == d
    assert_payload_equal(gi, gv, ri, rv)
    assert np.all(bits(ge) == 0)
    st = HT(d)
    gi, gv, ge, gk = st.step(g, np.inf)
    assert gk == 0
    assert_bits_equal(ge, oracle.ht(g, np.zeros(d, np.float32), LR, np.inf)[2])


def test_ht_special_values():
    d = 4099
    g = synth.small_gradient(2, d)
    e = np.zeros(d, dtype=np.float32)
    g[0], g[1], g[2], g[3] = np.nan, np.inf, -np.inf, np.float32(-0.0)
    e[4] = np.frombuffer(np.uint32(7).tobytes(), dtype=np.float32)[0]   # subnormal
    g[4] = 0.0
    e[5] = np.frombuffer(np.uint32(0x807FFFFF).tobytes(), dtype=np.float32)[0]
    g[5] = 0.0
    lam = np.frombuffer(np.uint32(6).tobytes(), dtype=np.float32)[0]
    for lam_ in (lam, np.float32(1e-4)):
        st = HT(d)
        st.e.copy_(torch.from_numpy(e))
        gi, gv, ge, gk = st.step(g, lam_)
        ri, rv, re, rk = oracle.ht(g, e, LR, lam_)
        assert gk == rk
        assert_payload_equal(gi, gv, ri, rv)
        assert_bits_equal(ge, re)


def test_ht_empty_vector():
    st = HT(0, cap=0)
    st.ctr.fill_(0)
    st.ctr[0] = 12345
    gi, gv, ge, gk = st.step(np.zeros(0, np.float32), 1e-3)
    assert gk == 0 and gi.size == 0


def test_ht_capacity_overflow():
    d = 300_007
    g = synth.small_gradient(3, d)
    lam = oracle.calibrate_lambda(g, 0.05)
    cap = 1000
    st = HT(d, cap=cap)
    gi, gv, ge, gk = st.step(g, lam)
    ri, rv, re, rk = oracle.ht(g, np.zeros(d, np.float32), LR, lam)
    assert gk == rk > cap
    assert gi.size == cap
    # the cap written pairs are distinct members of the true payload
    ci, cv = canonical(gi, gv)
    assert np.all(np.diff(ci) > 0)
    pos = np.searchsorted(ri, ci)
    assert np.all(ri[pos] == ci)
    assert_bits_equal(cv, rv[pos])
    assert_bits_equal(ge, re)


def test_ht_counter_returns_to_zero_between_calls():
    st = HT(200_000)
    for t, d in enumerate([200_000, 5, 4096 * 7 + 1, 0, 123_457]):
        g = synth.small_gradient(40 + t, d)
        e = torch.zeros(d, dtype=torch.float32, device=DEV)
        efs.ht_compress(to_dev(g), e, LR, np.float32(1e-4), st.idx, st.val, st.ctr)
        words = st.ctr.cpu().numpy()
        assert words[2] == 0 and words[3] == 0
        assert words[0] == oracle.ht(g, np.zeros(d, np.float32), LR, np.float32(1e-4))[3]


def test_ht_repeat_is_deterministic():
    d = 1_000_000
    g = synth.small_gradient(5, d)
    lam = oracle.calibrate_lambda(g, 0.02)
    outs = []
    for _ in range(3):
        st = HT(d)
        gi, gv, ge, gk = st.step(g, lam)
        outs.append((canonical(gi, gv), bits(ge).copy(), gk))
    for o in outs[1:]:
        assert o[2] == outs[0][2]
        np.testing.assert_array_equal(o[0][0], outs[0][0][0])
        np.testing.assert_array_equal(bits(o[0][1]), bits(outs[0][0][1]))
        np.testing.assert_array_equal(o[1], outs[0][1])


@pytest.mark.parametrize("unaligned", [False, True])
def test_ht_telemetry_totals(unaligned):
    # total error sum_t ||e_{t+1}||^2, total pairs sent and the running max of
    # |e'|, accumulated over an EF loop, against the oracle's residuals
    d, T = 1_000_003, 6
    gs = [synth.small_gradient(500 + t, d) for t in range(T)]
    lam = oracle.calibrate_lambda(gs[0], 0.005)
    st = HT(d, unaligned=unaligned)
    tel = efs.new_telemetry(DEV)
    e_ref = np.zeros(d, dtype=np.float32)
    err2, sent, maxbits = 0.0, 0, 0
    for t in range(T):
        efs.ht_compress_telemetry(to_dev(gs[t], unaligned), st.e, LR, lam, st.idx, st.val, st.ctr,
                                  tel)
        ri, rv, e_ref, rk = oracle.ht(gs[t], e_ref, LR, lam)
        assert efs.counter_value(st.ctr) == rk
        assert_bits_equal(st.e.cpu().numpy(), e_ref, "e' t=%d" % t)
        err2 += float(np.sum(e_ref.astype(np.float64) ** 2))
        sent += rk
        maxbits = max(maxbits, int(np.max(bits(e_ref) & np.uint32(0x7FFFFFFF))))
    got = efs.read_telemetry(tel)
    assert got["calls"] == T
    assert got["sent_total"] == sent
    assert got["max_abs_bits"] == maxbits
    assert got["max_abs"] < lam          # absolute compressor: every residual below lambda
    assert abs(got["err2_total"] - err2) <= 1e-9 * err2


def test_ht_telemetry_object_shared_by_calls_of_different_sizes():
    # one telemetry object for vectors of 1 tile, 40 tiles and 4000 tiles:
    # the calls run 1, 40 and hundreds of workgroups, so they fill different
    # sets of the 32 partial sums, whose total must still be every call's sum
    tel = efs.new_telemetry(DEV)
    err2, sent, maxbits, calls = 0.0, 0, 0, 0
    for d, seed in ((4093, 31), (4096 * 40, 32), (4096 * 4000 + 7, 33)):
        g = synth.small_gradient(seed, d)
        lam = oracle.calibrate_lambda(g, 0.01)
        st = HT(d)
        for t in range(2):
            gt = g if t == 0 else synth.small_gradient(seed + 100, d)
            efs.ht_compress_telemetry(to_dev(gt), st.e, LR, lam, st.idx, st.val, st.ctr, tel)
            e_prev = np.zeros(d, np.float32) if t == 0 else e_ref
            _, _, e_ref, rk = oracle.ht(gt, e_prev, LR, lam)
            err2 += float(np.sum(e_ref.astype(np.float64) ** 2))
            sent += rk
            maxbits = max(maxbits, int(np.max(bits(e_ref) & np.uint32(0x7FFFFFFF))))
            calls += 1
        assert_bits_equal(st.e.cpu().numpy(), e_ref, "e' d=%d" % d)
    got = efs.read_telemetry(tel)
    assert got["calls"] == calls and got["sent_total"] == sent
    assert got["max_abs_bits"] == maxbits
    assert abs(got["err2_total"] - err2) <= 1e-9 * err2
    parts = np.frombuffer(tel.cpu().numpy().tobytes()[:256], dtype="<f8")
    assert np.count_nonzero(parts) == 32  # the large call reaches every part


def test_ht_telemetry_empty_and_all_sent():
    st = HT(4096 * 3 + 1)
    tel = efs.new_telemetry(DEV)
    g = synth.small_gradient(9, st.d)
    efs.ht_compress_telemetry(to_dev(g), st.e, LR, 0.0, st.idx, st.val, st.ctr, tel)
    got = efs.read_telemetry(tel)
    assert got == {"err2_total": 0.0, "sent_total": float(st.d), "max_abs": 0.0,
                   "max_abs_bits": 0, "calls": 1}


# ---------------------------------------------------------------------------
# Top-k
# ---------------------------------------------------------------------------

TOPK_CASES = [(1, 1), (5, 3), (64, 64), (4097, 1), (4097, 4096), (12_289, 100),
              (100_003, 1000), (100_003, 50_001), (1_000_000, 1000), (1_000_000, 10_000)]


@pytest.mark.parametrize("unaligned", [False, True])
@pytest.mark.parametrize("d,k", TOPK_CASES)
def test_topk_matches_oracle(d, k, unaligned):
    say("topk parity d=%d k=%d unaligned=%s" % (d, k, unaligned))
    g = synth.small_gradient(60, d)
    e = synth.small_gradient(61, d, scale=1e-4)
    gi, gv, ge = topk_gpu(g, e, k, unaligned=unaligned)
    ri, rv, re = oracle.topk(g, e, LR, k)
    assert_payload_equal(gi, gv, ri, rv)
    assert_bits_equal(ge, re)


@pytest.mark.parametrize("d,k", [(10, 0), (100_000, 0), (100_000, 100_000), (4096, 4096)])
def test_topk_keep_none_or_all(d, k):
    g = synth.small_gradient(62, d)
    e = np.zeros(d, dtype=np.float32)
    gi, gv, ge = topk_gpu(g, e, k)
    ri, rv, re = oracle.topk(g, e, LR, k)
    assert_payload_equal(gi, gv, ri, rv)
    assert_bits_equal(ge, re)


@pytest.mark.parametrize("levels", [3, 41, 1001])
@pytest.mark.parametrize("k", [1, 777, 5000, 33_333])
def test_topk_ties_go_to_lower_index(levels, k):
    # quantised gradients: thousands of exact ties at the k-th magnitude
    d = 60_011
    rng = np.random.default_rng(levels * 7 + k)
    g = (rng.integers(-levels, levels + 1, size=d).astype(np.float32) * np.float32(1e-3))
    e = np.zeros(d, dtype=np.float32)
    gi, gv, ge = topk_gpu(g, e, k)
    ri, rv, re = oracle.topk(g, e, LR, k)
    assert_payload_equal(gi, gv, ri, rv, "levels=%d k=%d" % (levels, k))
    assert_bits_equal(ge, re)


def test_topk_all_equal_and_zero_vectors():
    d = 50_000
    for g in (np.full(d, 0.25, np.float32), np.zeros(d, np.float32),
              np.where(np.arange(d) % 2 == 0, np.float32(-0.0), np.float32(0.0)).astype(np.float32)):
        for k in (1, 12_345, d - 1):
            gi, gv, ge = topk_gpu(g, np.zeros(d, np.float32), k)
            ri, rv, re = oracle.topk(g, np.zeros(d, np.float32), LR, k)
            assert_payload_equal(gi, gv, ri, rv)
            assert_bits_equal(ge, re)


@pytest.mark.parametrize("unaligned", [False, True])
@pytest.mark.parametrize("case", ["many_ties", "many_zero_ties", "listed_zero_ties"])
def test_topk_radix_path_ties_below_larger_keys(case, unaligned):
    # Fresh workspace (radix path): larger keys elsewhere in the vector and
    # ties at the k-th magnitude split by index.  many_ties: ~40k ties at
    # 0.5 under ~10k larger keys (more ties than a list holds, so they are
    # counted per tile and ranked by a second read); many_zero_ties: ~60k
    # zeros tie at a zero threshold (the coordinates cleared for the larger
    # keys must not read as ties); listed_zero_ties: ~10k zeros, few enough
    # to be listed in the same read that sends the larger keys.
    d = 100_003
    rng = np.random.default_rng({"many_ties": 71, "many_zero_ties": 72, "listed_zero_ties": 73}[case])
    u = rng.random(d)
    small = (rng.standard_normal(d) * 1e-3).astype(np.float32)
    if case == "many_ties":
        g = np.where(u < 0.4, np.float32(0.5), np.where(u < 0.5, np.float32(1.0) + small, small))
        k = 30_000
    elif case == "many_zero_ties":
        g = np.where(u < 0.6, np.float32(0.0), np.float32(1.0) + small)
        k = 50_000
    else:
        g = np.where(u < 0.1, np.float32(0.0), np.float32(1.0) + small)
        k = 95_000
    g = g.astype(np.float32)
    e = np.zeros(d, dtype=np.float32)
    gi, gv, ge = topk_gpu(g, e, k, unaligned=unaligned)
    ri, rv, re = oracle.topk(g, e, LR, k)
    assert_payload_equal(gi, gv, ri, rv, case)
    assert_bits_equal(ge, re, case)


def test_topk_special_values():
    d = 9000
    g = synth.small_gradient(63, d)
    g[[5, 700, 4500]] = [np.nan, np.inf, -np.inf]
    e = np.zeros(d, dtype=np.float32)
    e[8] = np.frombuffer(np.uint32(3).tobytes(), dtype=np.float32)[0]
    for k in (1, 2, 3, 4, 100, d):
        gi, gv, ge = topk_gpu(g, e, k)
        ri, rv, re = oracle.topk(g, e, LR, k)
        assert_payload_equal(gi, gv, ri, rv, "k=%d" % k)
        assert_bits_equal(ge, re)


def test_topk_ef_loop_properties():
    # five EF iterations with e carried on the device, checked each step
    d, k = 2_000_003, 2000
    g0 = synth.small_gradient(70, d)
    e_dev = torch.zeros(d, dtype=torch.float32, device=DEV)
    ws = efs.new_topk_workspace(d, k, DEV)
    idx = torch.empty(k, dtype=torch.int32, device=DEV)
    val = torch.empty(k, dtype=torch.float32, device=DEV)
    e_host = np.zeros(d, dtype=np.float32)
    for t in range(5):
        g = synth.small_gradient(70 + t, d) if t else g0
        acc = oracle.ht(g, e_host, LR, np.inf)[2]
        efs.topk_compress(to_dev(g), e_dev, LR, k, idx, val, ws)
        e_host = e_dev.cpu().numpy()
        check_topk_properties(acc, k, idx.cpu().numpy(), val.cpu().numpy(), e_host)


class TopkState:
    """One Top-k EF trajectory on the device, with one workspace kept across
    calls (so later calls may take the bracket path)."""

    def __init__(self, d, kmax):
        self.d = d
        self.e = torch.zeros(d, dtype=torch.float32, device=DEV)
        self.ws = efs.new_topk_workspace(d, kmax, DEV)
        self.idx = torch.empty(kmax, dtype=torch.int32, device=DEV)
        self.val = torch.empty(kmax, dtype=torch.float32, device=DEV)

    def step(self, g_host, k, e_host):
        """One call from e_host; returns the device result."""
        self.e.copy_(torch.from_numpy(e_host))
        efs.topk_compress(to_dev(g_host), self.e, LR, k, self.idx[:k], self.val[:k], self.ws)
        return self.idx[:k].cpu().numpy(), self.val[:k].cpu().numpy(), self.e.cpu().numpy()

    def bracket(self):
        return efs.topk_took_bracket_path(self.ws)


def test_topk_workspace_reuse_matches_oracle():
    # A sequence of calls on one workspace: repeats of a distribution (the
    # bracket around the previous threshold holds), jumps in scale (it does
    # not), changes of k, ties split by index, and a call whose payload is
    # exactly the keys above the bracket.
    d = 300_007
    st = TopkState(d, 20_000)
    rng = np.random.default_rng(123)
    e = np.zeros(d, np.float32)
    calls = []   # (name, g, k, path expected: True bracket / False radix / None either)
    for t in range(4):
        calls.append(("gauss", (rng.standard_normal(d) * 1e-3).astype(np.float32), 3000,
                      False if t == 0 else True))
    calls.append(("scaled x50", (rng.standard_normal(d) * 5e-2).astype(np.float32), 3000, False))
    calls.append(("scaled back", (rng.standard_normal(d) * 1e-3).astype(np.float32), 3000, False))
    calls.append(("k up", (rng.standard_normal(d) * 1e-3).astype(np.float32), 20_000, None))
    calls.append(("k down", (rng.standard_normal(d) * 1e-3).astype(np.float32), 100, None))
    q = (rng.integers(-40, 41, size=d).astype(np.float32) * np.float32(1e-4))
    calls.append(("ties a", q, 7777, None))
    calls.append(("ties b", q[::-1].copy(), 7777, True))
    for name, g, k, path in calls:
        if name in ("gauss", "ties a", "ties b"):
            # fresh error: the same magnitude distribution (and exact ties for
            # the quantised vectors) in every call of the group
            e = np.zeros(d, np.float32)
        gi, gv, ge = st.step(g, k, e)
        ri, rv, re = oracle.topk(g, e, LR, k)
        assert_payload_equal(gi, gv, ri, rv, name)
        assert_bits_equal(ge, re, name)
        if path is not None:
            assert st.bracket() == path, name
        e = re
    # exactly k keys far above the previous threshold, the rest far below
    e = np.zeros(d, np.float32)
    g = np.full(d, 1e-6, np.float32)
    k = 500
    st.step(synth.small_gradient(5, d), k, e)        # sets a threshold near 3e-4
    g[rng.choice(d, k, replace=False)] = np.float32(1.0)
    gi, gv, ge = st.step(g, k, e)
    ri, rv, re = oracle.topk(g, e, LR, k)
    assert_payload_equal(gi, gv, ri, rv, "exactly k above")
    assert_bits_equal(ge, re, "exactly k above")
    assert st.bracket()


@pytest.mark.parametrize("levels", [81, 5])
def test_topk_bracket_path_splits_ties(levels):
    # the same quantised vector twice (fresh e): the second call takes the
    # bracket, and the k-th key is shared by thousands of coordinates of
    # which only the lowest indices are kept.  81 levels: fewer ties than
    # the bracket path ranks from a list; 5 levels: more (whole-vector ranks)
    d = 300_007
    st = TopkState(d, 20_000)
    rng = np.random.default_rng(140 + levels)
    half = levels // 2
    q = (rng.integers(-half, half + 1, size=d).astype(np.float32) * np.float32(1e-4))
    k = 7777 if levels > 10 else 150_001
    st.ws = efs.new_topk_workspace(d, k, DEV)
    st.idx = torch.empty(k, dtype=torch.int32, device=DEV)
    st.val = torch.empty(k, dtype=torch.float32, device=DEV)
    e = np.zeros(d, np.float32)
    for t in range(2):
        gi, gv, ge = st.step(q, k, e)
        ri, rv, re = oracle.topk(q, e, LR, k)
        assert_payload_equal(gi, gv, ri, rv, "levels %d call %d" % (levels, t))
        assert_bits_equal(ge, re, "levels %d call %d" % (levels, t))
    assert st.bracket()


@pytest.mark.parametrize("neg_zero", [False, True])
def test_topk_zero_threshold_with_many_ties_on_one_workspace(neg_zero):
    # fewer than k non-zero entries: the threshold key is that of zero and
    # ~200k zeros tie at it, far more than the bracket path ranks from a
    # list.  The second and third calls start from the first call's
    # threshold (0), so their bracket holds every zero; the ties must still
    # go to the lowest indices, none of them a coordinate already sent.
    d, k = 300_007, 150_000
    st = TopkState(d, k)
    rng = np.random.default_rng(2024 + neg_zero)
    e = np.zeros(d, np.float32)
    if neg_zero:
        # -0 + lr * -0 is -0: both signs of zero among the tied keys
        e[rng.random(d) < 0.5] = np.float32(-0.0)
    paths = []
    for t in range(3):
        g = np.zeros(d, np.float32)
        if neg_zero:
            g[rng.random(d) < 0.5] = np.float32(-0.0)
        nz = rng.choice(d, 100_000, replace=False)
        g[nz] = (rng.standard_normal(nz.size) * 1e-3).astype(np.float32)
        gi, gv, ge = st.step(g, k, e)
        ri, rv, re = oracle.topk(g, e, LR, k)
        assert np.unique(gi).size == k, "call %d: duplicate indices in the payload" % t
        assert_payload_equal(gi, gv, ri, rv, "zero threshold, call %d" % t)
        assert_bits_equal(ge, re, "zero threshold, call %d" % t)
        paths.append(st.bracket())
        e = re
    say("zero threshold calls, bracket path per call: %s" % paths)


def test_topk_bracket_with_many_candidates():
    # |p| uniform in [0.9, 1.1]: the bracket around the previous threshold
    # (the 90th percentile) holds ~40 % of the vector, so the bracket path
    # moves its candidates several per thread per chunk
    d, k = 1 << 20, 100_000
    st = TopkState(d, k)
    rng = np.random.default_rng(150)
    for t in range(2):
        g = (rng.uniform(9.0, 11.0, size=d) * rng.choice([-1.0, 1.0], size=d)).astype(np.float32)
        e = np.zeros(d, np.float32)
        gi, gv, ge = st.step(g, k, e)
        ri, rv, re = oracle.topk(g, e, LR, k)
        assert_payload_equal(gi, gv, ri, rv, "call %d" % t)
        assert_bits_equal(ge, re, "call %d" % t)
    assert st.bracket()


@pytest.mark.parametrize("seed", range(6))
def test_topk_randomised_ef_loops(seed):
    # random size and k, six EF steps on one workspace with scale jumps and
    # quantised steps: every step against the oracle, whichever path it takes
    rng = np.random.default_rng(950 + seed)
    d = int(rng.integers(10_000, 400_000))
    k = int(np.ceil(d * 10.0 ** rng.uniform(-3.5, -0.5)))
    st = TopkState(d, k)
    e = np.zeros(d, np.float32)
    paths = []
    for t in range(6):
        scale = np.float32(10.0 ** rng.choice([0.0, 0.0, 0.0, 1.5, -1.0]))
        g = (synth.small_gradient(960 + 10 * seed + t, d) * scale).astype(np.float32)
        if rng.random() < 0.3:
            g = (np.round(g / np.float32(2e-3)) * np.float32(2e-3)).astype(np.float32)
        gi, gv, ge = st.step(g, k, e)
        ri, rv, re = oracle.topk(g, e, LR, k)
        assert_payload_equal(gi, gv, ri, rv, "seed %d t=%d" % (seed, t))
        assert_bits_equal(ge, re, "seed %d t=%d e'" % (seed, t))
        paths.append(int(st.bracket()))
        e = re
    say("topk randomised seed=%d d=%d k=%d: bracket path per step %s" % (seed, d, k, paths))


def test_topk_workspace_contents_do_not_matter():
    d, k = 200_003, 1500
    g = synth.small_gradient(77, d)
    ri, rv, re = oracle.topk(g, np.zeros(d, np.float32), LR, k)
    for fill in (0x00, 0xFF, 0x54, None):
        ws = efs.new_topk_workspace(d, k, DEV)
        if fill is None:
            ws.copy_(torch.from_numpy(np.random.default_rng(9).integers(0, 256, ws.numel(),
                                                                          dtype=np.uint8)))
        else:
            ws.fill_(fill)
        e = torch.zeros(d, dtype=torch.float32, device=DEV)
        idx = torch.empty(k, dtype=torch.int32, device=DEV)
        val = torch.empty(k, dtype=torch.float32, device=DEV)
        efs.topk_compress(to_dev(g), e, LR, k, idx, val, ws)
        assert_payload_equal(idx.cpu().numpy(), val.cpu().numpy(), ri, rv, "fill %r" % fill)
        assert_bits_equal(e.cpu().numpy(), re, "fill %r" % fill)


def test_topk_ef_loop_matches_oracle_each_step():
    # the training-like case: e carried, one workspace, 12 iterations
    d, k = 500_009, 2500
    st = TopkState(d, k)
    e = np.zeros(d, np.float32)
    hits = 0
    for t in range(12):
        g = synth.small_gradient(300 + t, d)
        gi, gv, ge = st.step(g, k, e)
        ri, rv, e = oracle.topk(g, e, LR, k)
        assert_payload_equal(gi, gv, ri, rv, "t=%d" % t)
        assert_bits_equal(ge, e, "t=%d" % t)
        hits += st.bracket()
    say("bracket path taken in %d of 12 iterations" % hits)
    assert hits >= 1


# ---------------------------------------------------------------------------
# n-worker average
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("layout", efs.LAYOUTS)
@pytest.mark.parametrize("n", [1, 2, 3, 8, 40])
def test_accumulate_matches_oracle(n, layout):
    d = 400_009
    lam = np.float32(2.2e-4)
    payloads_dev, payloads_ref = [], []
    for w in range(n):
        g = synth.small_gradient(80 + w, d)
        st = HT(d, cap=d // 10)
        gi, gv, ge, gk = st.step(g, lam)
        assert gk <= st.cap
        payloads_dev.append((st.idx, st.val, st.ctr))
        payloads_ref.append((gi, gv))
    out = torch.empty(d, dtype=torch.float32, device=DEV)
    ws = efs.new_apply_workspace(payloads_dev, d, DEV, layout=layout)
    efs.sparse_accumulate(payloads_dev, d, out, ws)
    ref = oracle.accumulate(payloads_ref, d)
    assert_bits_equal(out.cpu().numpy(), ref)
    assert efs.sparse_status(ws) == 0


def test_accumulate_layouts_alternate_on_one_workspace():
    # the same memory used as bucketed (whole) and as packed (a shorter view)
    # in turn, with different payloads each call: both layouts keep the
    # counters and the control block in the same state between calls
    d, n = 300_007, 3
    lam = np.float32(3e-4)
    states = [HT(d, cap=d // 8) for _ in range(n)]
    p_dev = [(s.idx, s.val, s.ctr) for s in states]
    whole = efs.new_apply_workspace(p_dev, d, DEV, layout="bucketed")
    packed = whole[:efs.sparse_apply_workspace_bytes(n, d, sum(s.cap for s in states))]
    out = torch.empty(d, dtype=torch.float32, device=DEV)
    for t in range(6):
        ref_in = []
        for w, s in enumerate(states):
            gi, gv, _, _ = s.step(synth.small_gradient(700 + 10 * t + w, d), lam)
            ref_in.append((gi, gv))
        ws = whole if t % 3 != 1 else packed
        efs.sparse_accumulate(p_dev, d, out, ws)
        assert_bits_equal(out.cpu().numpy(), oracle.accumulate(ref_in, d), "call %d" % t)
        assert efs.sparse_status(whole) == 0


def test_accumulate_topk_payloads_and_tail():
    d = 4096 * 3 + 3
    ps_dev, ps_ref = [], []
    for w in range(3):
        g = synth.small_gradient(90 + w, d)
        gi, gv, _ = topk_gpu(g, np.zeros(d, np.float32), 500)
        ps_dev.append((to_dev(gi), to_dev(gv)))
        ps_ref.append((gi, gv))
    out = torch.empty(d, dtype=torch.float32, device=DEV)
    efs.sparse_accumulate(ps_dev, d, out, efs.new_apply_workspace(ps_dev, d, DEV))
    assert_bits_equal(out.cpu().numpy(), oracle.accumulate(ps_ref, d))


@pytest.mark.parametrize("layout", efs.LAYOUTS)
@pytest.mark.parametrize("n", [3, 8])
def test_accumulate_special_values(n, layout):
    # signed zeros, sums that cancel to zero, infinities, NaN and subnormals,
    # also at the ragged tail: the division by n leaves every zero as it is
    # and must divide everything else with one IEEE rounding
    d = 4096 * 2 + 3
    tiny = np.float32(1e-45)
    base = [(5, -0.0), (6, 0.0), (8, np.inf), (9, -np.inf), (10, np.nan),
            (11, tiny), (12, -3 * tiny), (d - 1, 2.5), (d - 2, -0.0)]
    ps_dev, ps_ref = [], []
    for w in range(n):
        pairs = list(base) + [(200 + w, float(w) - 1.25)]
        # workers 0 and 1 alone touch 7 and d - 3, with opposite values: the
        # sums there are +0
        if w == 0:
            pairs += [(7, 1.5), (d - 3, 7.0)]
        if w == 1:
            pairs = [(7, -1.5), (d - 3, -7.0), (100 + w, 1.0)]
        idx = np.array([i for i, _ in pairs], dtype=np.int32)
        val = np.array([v for _, v in pairs], dtype=np.float32)
        ps_dev.append((to_dev(idx), to_dev(val)))
        ps_ref.append((idx, val))
    out = torch.full((d,), 9.0, dtype=torch.float32, device=DEV)
    efs.sparse_accumulate(ps_dev, d, out, efs.new_apply_workspace(ps_dev, d, DEV, layout=layout))
    got = out.cpu().numpy()
    ref = oracle.accumulate(ps_ref, d)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert_bits_equal(got[~nan], ref[~nan])
    assert bits(got[7]) == 0 and bits(got[d - 3]) == 0  # cancelled sums are +0


@pytest.mark.parametrize("layout", efs.LAYOUTS)
def test_accumulate_reports_out_of_range_indices(layout):
    # indices outside [0, d) are skipped and the status word says so; the
    # next call on the same workspace with a clean payload reports 0 again
    d = 1000
    idx = np.array([3, -1, 999, 1000, 7], dtype=np.int32)
    val = np.array([1.0, 5.0, 2.0, 6.0, 3.0], dtype=np.float32)
    out = torch.empty(d, dtype=torch.float32, device=DEV)
    ps = [(to_dev(idx), to_dev(val)), (to_dev(idx[:1]), to_dev(val[:1]))]
    ws = efs.new_apply_workspace(ps, d, DEV, layout=layout)
    efs.sparse_accumulate(ps, d, out, ws)
    keep = (idx >= 0) & (idx < d)
    ref = oracle.accumulate([(idx[keep], val[keep]), (idx[:1], val[:1])], d)
    assert_bits_equal(out.cpu().numpy(), ref)
    assert efs.sparse_status(ws) == efs.SPARSE_BAD_INDEX
    clean = [(to_dev(idx[keep]), to_dev(val[keep])), ps[1]]
    efs.sparse_accumulate(clean, d, out, ws)
    assert_bits_equal(out.cpu().numpy(), ref)
    assert efs.sparse_status(ws) == 0


@pytest.mark.parametrize("layout", efs.LAYOUTS)
def test_accumulate_reports_a_truncated_hard_threshold_payload(layout):
    # a hard-threshold call whose k_t exceeds the payload capacity: the
    # average uses the cap pairs written and the status word reports the
    # truncation (the error of the dropped coordinates is already +0)
    d = 300_007
    g = synth.small_gradient(3, d)
    lam = oracle.calibrate_lambda(g, 0.05)
    full, short = HT(d), HT(d, cap=1000)
    gi, gv, _, gk = full.step(g, lam)
    si, sv, _, sk = short.step(g, lam)
    assert sk == gk > 1000 and si.size == 1000
    out = torch.empty(d, dtype=torch.float32, device=DEV)
    ps = [(full.idx, full.val, full.ctr), (short.idx, short.val, short.ctr)]
    ws = efs.new_apply_workspace(ps, d, DEV, layout=layout)
    efs.sparse_accumulate(ps, d, out, ws)
    assert efs.sparse_status(ws) == efs.SPARSE_TRUNCATED
    assert_bits_equal(out.cpu().numpy(), oracle.accumulate([(gi, gv), (si, sv)], d))
    efs.sparse_accumulate(ps[:1], d, out, ws)
    assert efs.sparse_status(ws) == 0


def test_copy_probe_copies():
    for n in (0, 3, 4096 * 5 + 2):
        src = torch.arange(n, dtype=torch.float32, device=DEV)
        dst = torch.zeros(n, dtype=torch.float32, device=DEV)
        efs.copy_probe(src, dst)
        assert torch.equal(src, dst)


@pytest.mark.parametrize("shape", [0, 4], ids=["persistent", "tile_per_workgroup"])
def test_stream_probes(shape):
    n = 4096 * 7 + 5
    x = torch.arange(n, dtype=torch.float32, device=DEV)
    y = torch.full((n,), 2.0, dtype=torch.float32, device=DEV)
    efs.stream_probe(x, y, 0 + shape)
    assert torch.equal(x, y)
    y.fill_(2.0)
    efs.stream_probe(x, y, 3 + shape)
    whole = 4096 * 7
    assert torch.equal(y[:whole], 2.0 + 0.5 * x[:whole])
    assert torch.all(y[whole:] == 2.0)
    efs.stream_probe(x, y, 2 + shape)
    assert torch.equal(y[:whole].view(-1, 4), torch.tensor([1.0, 2.0, 3.0, 4.0], device=DEV).expand(whole // 4, 4))
    efs.stream_probe(x, y, 1 + shape)
    torch.cuda.synchronize()


def test_sticky_last_error():
    lib = efs.load_library()
    g = torch.zeros(8, dtype=torch.float32, device=DEV)
    idx = torch.empty(8, dtype=torch.int32, device=DEV)
    val = torch.empty(8, dtype=torch.float32, device=DEV)
    ctr = efs.new_counter(DEV)
    lib.efs_last_error()                    # clear
    efs.ht_compress(g, g.clone(), 0.1, 1e-3, idx, val, ctr)
    assert lib.efs_last_error() == efs.EFS_OK
    with pytest.raises(efs.EfsError):
        efs.ht_compress(g, g.clone(), 0.1, -1.0, idx, val, ctr)   # lambda < 0
    efs.ht_compress(g, g.clone(), 0.1, 1e-3, idx, val, ctr)       # a good call after it
    assert lib.efs_last_error() == efs.EFS_EINVAL                # sticky until read
    assert lib.efs_last_error() == efs.EFS_OK
