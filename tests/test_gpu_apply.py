"""GPU parity of sparse_apply (exchange-and-average fused with the model
update: Algorithm 1's x <- x - avg and the momentum form of Algorithm 2,
Appendix C.6.2) against the CPU oracle, bit for bit, through the C ABI.

Payloads come from the library's own compressors (so their pair order is the
unspecified block order the kernels produce) or are written by hand to cover
shuffled, dense, empty and out-of-range cases.  Sizes span several
8192-coordinate ranges and a ragged tail.
"""
import numpy as np
import pytest

import oracle
from paper_2108_00951_amd import synth
from tests._checks import assert_bits_equal

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2108_00951_amd import binding as efs  # noqa: E402

LR = np.float32(0.1)
DEV = "cuda"
BETA, GAMMA = 0.9, 0.05


def say(*a):
    print(*a, flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def ht_payloads(d, n, lam, seed, cap=None):
    """n workers' hard-threshold payloads (device, with counters) and their
    canonical host copies."""
    cap = d // 8 if cap is None else cap
    p_dev, p_ref = [], []
    for w in range(n):
        g = synth.small_gradient(seed + w, d)
        e = torch.zeros(d, dtype=torch.float32, device=DEV)
        idx = torch.empty(cap, dtype=torch.int32, device=DEV)
        val = torch.empty(cap, dtype=torch.float32, device=DEV)
        ctr = efs.new_counter(DEV)
        efs.ht_compress(dev(g), e, LR, lam, idx, val, ctr)
        k = efs.counter_value(ctr)
        assert k <= cap
        p_dev.append((idx, val, ctr))
        p_ref.append((idx[:k].cpu().numpy(), val[:k].cpu().numpy()))
    return p_dev, p_ref


def host_state(d, seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(d).astype(np.float32)
    m = (rng.standard_normal(d) * 1e-3).astype(np.float32)
    # a few signed zeros and subnormals in both
    c = min(d, 4)
    x[:c] = np.array([-0.0, 0.0, 1e-45, -2e-39], np.float32)[:c]
    m[:c] = np.array([-0.0, 1e-44, 0.0, -3e-40], np.float32)[:c]
    return x, m


def run_apply(p_dev, d, mode, x_host, m_host=None, ws=None, layout="bucketed"):
    x = dev(x_host)
    m = dev(m_host) if m_host is not None else None
    if ws is None:
        ws = efs.new_apply_workspace(p_dev, d, DEV, layout=layout)
    efs.sparse_apply(p_dev, d, mode, x, ws, m=m, beta=BETA, gamma=GAMMA)
    return x.cpu().numpy(), (m.cpu().numpy() if m is not None else None)


def check_all_modes(p_dev, p_ref, d, seed, layout="bucketed"):
    x0, m0 = host_state(d, seed)
    say("  average (%s)" % layout)
    got, _ = run_apply(p_dev, d, efs.APPLY_AVERAGE, np.full(d, 7.0, np.float32), layout=layout)
    assert_bits_equal(got, oracle.accumulate(p_ref, d))
    say("  sgd")
    got, _ = run_apply(p_dev, d, efs.APPLY_SGD, x0, layout=layout)
    want, _ = oracle.update(p_ref, x0, 1)
    assert_bits_equal(got, want)
    say("  momentum")
    got_x, got_m = run_apply(p_dev, d, efs.APPLY_MOMENTUM, x0, m0, layout=layout)
    want_x, want_m = oracle.update(p_ref, x0, 2, m=m0, beta=BETA, gamma=GAMMA)
    assert_bits_equal(got_m, want_m)
    assert_bits_equal(got_x, want_x)


@pytest.mark.parametrize("layout", efs.LAYOUTS)
@pytest.mark.parametrize("n", [1, 2, 3, 8])
def test_apply_ht_payloads(n, layout):
    d = 400_009
    say("apply ht payloads n=%d d=%d" % (n, d))
    p_dev, p_ref = ht_payloads(d, n, np.float32(2.2e-4), 100 + 10 * n)
    check_all_modes(p_dev, p_ref, d, n, layout)


@pytest.mark.parametrize("layout", efs.LAYOUTS)
@pytest.mark.parametrize("d", [1, 5, 8192, 8192 * 2 + 5])
def test_apply_dense_payloads(d, layout):
    # lambda = 0: every worker sends every coordinate (the densest payload)
    say("apply dense payloads d=%d" % d)
    p_dev, p_ref = ht_payloads(d, 3, np.float32(0.0), 7, cap=d)
    assert all(p[0].size == d for p in p_ref)
    check_all_modes(p_dev, p_ref, d, 3, layout)


def test_apply_topk_payloads():
    d = 8192 * 5 + 123
    say("apply top-k payloads d=%d" % d)
    p_dev, p_ref = [], []
    for w in range(3):
        g = synth.small_gradient(300 + w, d)
        ws = efs.new_topk_workspace(d, 900)
        idx = torch.empty(900, dtype=torch.int32, device=DEV)
        val = torch.empty(900, dtype=torch.float32, device=DEV)
        efs.topk_compress(dev(g), torch.zeros(d, dtype=torch.float32, device=DEV), LR, 900,
                          idx, val, ws)
        p_dev.append((idx, val))
        p_ref.append((idx.cpu().numpy(), val.cpu().numpy()))
    check_all_modes(p_dev, p_ref, d, 4)


@pytest.mark.parametrize("layout", efs.LAYOUTS)
def test_apply_shuffled_overlapping_payloads(layout):
    # pairs in random order, heavy overlap between workers, values chosen so
    # the worker order of the sum matters
    d = 8192 * 4 + 77
    rng = np.random.default_rng(11)
    p_dev, p_ref = [], []
    for w in range(5):
        idx = rng.permutation(d)[: d // 3].astype(np.int32)
        val = (rng.standard_normal(idx.size) * 10.0 ** rng.integers(-6, 3, idx.size)).astype(np.float32)
        p_dev.append((dev(idx), dev(val)))
        p_ref.append((idx, val))
    say("apply shuffled payloads")
    check_all_modes(p_dev, p_ref, d, 5, layout)


def test_apply_worker_order_decides_rounding():
    # (1, 2^-24, 2^-24) at one coordinate averages to 0x3EAAAAAB only in
    # worker order
    d = 10
    ps = [(dev(np.array([4], np.int32)), dev(np.array([v], np.float32)))
          for v in (1.0, 2.0 ** -24, 2.0 ** -24)]
    got, _ = run_apply(ps, d, efs.APPLY_AVERAGE, np.zeros(d, np.float32))
    assert got.view(np.uint32)[4] == 0x3EAAAAAB


@pytest.mark.parametrize("layout", efs.LAYOUTS)
def test_apply_empty_payloads_and_counts(layout):
    d = 8192 * 2 + 9
    x0, m0 = host_state(d, 8)
    idx = torch.empty(16, dtype=torch.int32, device=DEV)
    val = torch.empty(16, dtype=torch.float32, device=DEV)
    ctr = efs.new_counter(DEV)  # count 0 with capacity 16
    empty = torch.empty(0, dtype=torch.int32, device=DEV)
    emptyv = torch.empty(0, dtype=torch.float32, device=DEV)
    p_dev = [(idx, val, ctr), (empty, emptyv)]
    got, _ = run_apply(p_dev, d, efs.APPLY_AVERAGE, np.full(d, 3.0, np.float32), layout=layout)
    assert np.all(got.view(np.uint32) == 0)
    got, _ = run_apply(p_dev, d, efs.APPLY_SGD, x0, layout=layout)
    assert_bits_equal(got, x0)
    got_x, got_m = run_apply(p_dev, d, efs.APPLY_MOMENTUM, x0, m0, layout=layout)
    none = (np.zeros(0, np.int32), np.zeros(0, np.float32))
    want_x, want_m = oracle.update([none, none], x0, 2, m=m0, beta=BETA, gamma=GAMMA)
    assert_bits_equal(got_m, want_m)
    assert_bits_equal(got_x, want_x)


@pytest.mark.parametrize("layout", efs.LAYOUTS)
def test_apply_ignores_out_of_range_indices(layout):
    d = 9000
    idx = np.array([3, -1, 8999, 9000, 8192, 2 ** 31 - 1, 7], dtype=np.int32)
    val = np.array([1.0, 5.0, 2.0, 6.0, 3.0, 4.0, 0.5], dtype=np.float32)
    keep = (idx >= 0) & (idx < d)
    p_dev = [(dev(idx), dev(val)), (dev(idx[:1]), dev(val[:1]))]
    p_ref = [(idx[keep], val[keep]), (idx[:1], val[:1])]
    check_all_modes(p_dev, p_ref, d, 9, layout)
    ws = efs.new_apply_workspace(p_dev, d, DEV, layout=layout)
    run_apply(p_dev, d, efs.APPLY_SGD, np.zeros(d, np.float32), ws=ws)
    assert efs.sparse_status(ws) == efs.SPARSE_BAD_INDEX


def test_apply_one_worker_signed_zeros():
    # one worker: x - (+0 + v), never x - v (they differ for x = -0, v = -0),
    # and out-of-range indices ignored
    d = 9000
    idx = np.array([0, 1, 2, 3, 4, -5, 9000, 8191, 8192], dtype=np.int32)
    val = np.array([-0.0, 0.0, -1e-45, 2e-39, -0.0, 1.0, 2.0, 3.5, -0.0], dtype=np.float32)
    keep = (idx >= 0) & (idx < d)
    x0, m0 = host_state(d, 21)
    x0[4] = np.float32(-0.0)
    x0[8192] = np.float32(-0.0)
    p_dev = [(dev(idx), dev(val))]
    p_ref = [(idx[keep], val[keep])]
    got, _ = run_apply(p_dev, d, efs.APPLY_SGD, x0)
    want, _ = oracle.update(p_ref, x0, 1)
    assert_bits_equal(got, want)
    assert got[4].view(np.uint32) == np.float32(-0.0).view(np.uint32)
    got, _ = run_apply(p_dev, d, efs.APPLY_AVERAGE, np.full(d, 7.0, np.float32))
    assert_bits_equal(got, oracle.accumulate(p_ref, d))
    got_x, got_m = run_apply(p_dev, d, efs.APPLY_MOMENTUM, x0, m0)
    want_x, want_m = oracle.update(p_ref, x0, 2, m=m0, beta=BETA, gamma=GAMMA)
    assert_bits_equal(got_m, want_m)
    assert_bits_equal(got_x, want_x)


@pytest.mark.parametrize("layout", efs.LAYOUTS)
def test_apply_count_larger_than_capacity(layout):
    # a counter above the capacity (an overflowed payload) uses caps[w] pairs
    d = 20_000
    rng = np.random.default_rng(12)
    idx = rng.permutation(d)[:500].astype(np.int32)
    val = rng.standard_normal(500).astype(np.float32)
    ctr = efs.new_counter(DEV)
    ctr[0] = 100_000
    p_dev = [(dev(idx), dev(val), ctr)]
    ws = efs.new_apply_workspace(p_dev, d, DEV, layout=layout)
    got, _ = run_apply(p_dev, d, efs.APPLY_AVERAGE, np.zeros(d, np.float32), ws=ws)
    assert_bits_equal(got, oracle.accumulate([(idx, val)], d))
    assert efs.sparse_status(ws) == efs.SPARSE_TRUNCATED


@pytest.mark.parametrize("layout", efs.LAYOUTS)
def test_apply_max_workers(layout):
    d = 8192 + 1000
    n = efs.MAX_WORKERS
    rng = np.random.default_rng(13)
    p_dev, p_ref = [], []
    for w in range(n):
        idx = rng.permutation(d)[:2000].astype(np.int32)
        val = rng.standard_normal(2000).astype(np.float32)
        p_dev.append((dev(idx), dev(val)))
        p_ref.append((idx, val))
    say("apply n=%d" % n)
    check_all_modes(p_dev, p_ref, d, 13, layout)


@pytest.mark.parametrize("layout", efs.LAYOUTS)
def test_apply_workspace_contents_do_not_matter_and_repeat(layout):
    d = 8192 * 3 + 1
    p_dev, p_ref = ht_payloads(d, 4, np.float32(2.2e-4), 40)
    x0, m0 = host_state(d, 14)
    want_x, want_m = oracle.update(p_ref, x0, 2, m=m0, beta=BETA, gamma=GAMMA)
    ws = efs.new_apply_workspace(p_dev, d, DEV, layout=layout)
    for fill in (0, 255, 0x5A, None):
        if fill is None:
            ws.copy_(torch.randint(0, 256, ws.shape, dtype=torch.uint8, device=DEV))
        else:
            ws.fill_(fill)
        got_x, got_m = run_apply(p_dev, d, efs.APPLY_MOMENTUM, x0, m0, ws=ws)
        assert_bits_equal(got_m, want_m)
        assert_bits_equal(got_x, want_x)


@pytest.mark.parametrize("layout", efs.LAYOUTS)
def test_apply_ef_momentum_loop(layout):
    # Algorithm 2 end to end for 4 steps: every worker compresses g + e with
    # the hard threshold (lr = 1: the learning rate is applied at the update),
    # the payloads are averaged and applied with momentum; x, m and each e
    # are compared with the oracle after every step
    d, n, T = 8192 * 6 + 321, 3, 4
    lam = np.float32(2e-3)
    x_ref, m_ref = host_state(d, 15)
    x, m = dev(x_ref), dev(m_ref)
    e_dev = [torch.zeros(d, dtype=torch.float32, device=DEV) for _ in range(n)]
    e_ref = [np.zeros(d, np.float32) for _ in range(n)]
    idx = [torch.empty(d, dtype=torch.int32, device=DEV) for _ in range(n)]
    val = [torch.empty(d, dtype=torch.float32, device=DEV) for _ in range(n)]
    ctr = [efs.new_counter(DEV) for _ in range(n)]
    p_dev = [(idx[w], val[w], ctr[w]) for w in range(n)]
    ws = efs.new_apply_workspace(p_dev, d, DEV, layout=layout)
    for t in range(T):
        say("  momentum loop step", t)
        p_ref = []
        for w in range(n):
            g = synth.small_gradient(500 + 10 * t + w, d)
            efs.ht_compress(dev(g), e_dev[w], 1.0, lam, idx[w], val[w], ctr[w])
            ri, rv, e_ref[w], _ = oracle.ht(g, e_ref[w], 1.0, lam)
            p_ref.append((ri, rv))
        efs.sparse_apply(p_dev, d, efs.APPLY_MOMENTUM, x, ws, m=m, beta=BETA, gamma=GAMMA)
        x_ref, m_ref = oracle.update(p_ref, x_ref, 2, m=m_ref, beta=BETA, gamma=GAMMA)
        for w in range(n):
            assert_bits_equal(e_dev[w].cpu().numpy(), e_ref[w])
        assert_bits_equal(m.cpu().numpy(), m_ref)
        assert_bits_equal(x.cpu().numpy(), x_ref)


@pytest.mark.parametrize("layout", efs.LAYOUTS)
def test_apply_many_ranges(layout):
    # more than 4096 ranges of 8192 coordinates: more (range, worker)
    # counters than one tile of the packed layout's scan (8192), pairs at
    # both ends and in the last range
    d = 4096 * 8192 + 8192 * 37 + 11
    rng = np.random.default_rng(16)
    p_dev, p_ref = [], []
    for w in range(3):
        idx = rng.choice(d, 200_000, replace=False).astype(np.int32)
        idx[:3] = [0, d - 1, 4096 * 8192 + w]
        val = rng.standard_normal(idx.size).astype(np.float32)
        p_dev.append((dev(idx), dev(val)))
        p_ref.append((idx, val))
    say("apply many ranges d=%d (%s)" % (d, layout))
    x0 = rng.standard_normal(d).astype(np.float32)
    got, _ = run_apply(p_dev, d, efs.APPLY_SGD, x0, layout=layout)
    want, _ = oracle.update(p_ref, x0, 1)
    assert_bits_equal(got, want)
    got, _ = run_apply(p_dev, d, efs.APPLY_AVERAGE, x0, layout=layout)
    assert_bits_equal(got, oracle.accumulate(p_ref, d))
