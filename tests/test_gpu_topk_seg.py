"""GPU parity of the layer-wise Top-k (topk_segmented_compress; Appendix
C.5: Top-k on each layer's tensor on its own) against the CPU oracle.

Within a segment the payload order is unspecified, so each segment's pairs
are compared after sorting by index; indices, values and the whole error
vector are compared bit for bit.  Layouts mix empty, tiny, 4096-aligned and
unaligned segments; budgets cover k = 0, k = size, k > size; values cover
ties at the threshold (quantised values, all-zero segments), special values,
and candidate sets larger than the final pass holds in LDS.
"""
import numpy as np
import pytest

import oracle
from paper_2108_00951_amd import synth
from tests._checks import assert_bits_equal, bits

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2108_00951_amd import binding as efs  # noqa: E402

LR = np.float32(0.1)
DEV = "cuda"


def say(*a):
    print(*a, flush=True)


def dev(a, unaligned=False):
    a = np.ascontiguousarray(a)
    if not unaligned:
        return torch.from_numpy(a).to(DEV)
    buf = torch.empty(a.size + 1, dtype=torch.from_numpy(a[:0]).dtype, device=DEV)
    v = buf[1:]
    v.copy_(torch.from_numpy(a))
    return v


def run_gpu(g, e, offsets, ks, lr=LR, unaligned=False, k_total=None, ws=None):
    """One call; returns (idx, val, e_next, workspace) on the host."""
    offsets = np.asarray(offsets, dtype=np.int64)
    ks = np.asarray(ks, dtype=np.int64)
    sizes = np.diff(offsets)
    total = int(np.minimum(np.maximum(ks, 0), np.maximum(sizes, 0)).sum())
    if k_total is None:
        k_total = total
    gd, ed = dev(g, unaligned), dev(e, unaligned)
    idx = torch.full((max(k_total, 1),), -7, dtype=torch.int32, device=DEV)[:k_total]
    val = torch.full((max(k_total, 1),), -7.0, dtype=torch.float32, device=DEV)[:k_total]
    if ws is None:
        ws = efs.new_topk_segmented_workspace(ks.size, k_total, DEV)
    efs.topk_segmented_compress(gd, ed, lr, dev(offsets), dev(ks), idx, val, ws)
    return idx.cpu().numpy(), val.cpu().numpy(), ed.cpu().numpy(), ws


def check(g, e, offsets, ks, lr=LR, unaligned=False, what=""):
    gi, gv, ge, ws = run_gpu(g, e, offsets, ks, lr, unaligned)
    assert efs.topk_segmented_status(ws) == 0
    ri, rv, re = oracle.topk_segmented(g, e, lr, offsets, ks)
    assert gi.size == ri.size, what
    # per segment: same region, same pairs after sorting by index
    offsets = np.asarray(offsets)
    pos = 0
    for s in range(len(ks)):
        n = int(min(max(int(ks[s]), 0), int(offsets[s + 1] - offsets[s])))
        seg_i, seg_v = gi[pos:pos + n], gv[pos:pos + n]
        order = np.argsort(seg_i, kind="stable")
        np.testing.assert_array_equal(seg_i[order], ri[pos:pos + n], "%s segment %d" % (what, s))
        assert_bits_equal(seg_v[order], rv[pos:pos + n], "%s segment %d values" % (what, s))
        pos += n
    assert_bits_equal(ge, re, "%s e'" % what)
    return gi, gv, ge


def random_layout(rng, d, nseg):
    cuts = np.sort(rng.integers(0, d + 1, size=nseg - 1))
    return np.concatenate([[0], cuts, [d]]).astype(np.int64)


@pytest.mark.parametrize("unaligned", [False, True])
def test_segmented_mixed_layout(unaligned):
    sizes = [0, 1, 64, 4096, 4097, 8192 * 3, 0, 70_001, 5, 4095, 250_000, 1]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    d = int(off[-1])
    ks = np.array([0, 1, 3, 40, 4097, 100, 2, 70, 9, 0, 2500, 1], dtype=np.int64)
    g = synth.small_gradient(401, d)
    e = (synth.small_gradient(402, d) * np.float32(0.1)).astype(np.float32)
    say("segmented mixed layout unaligned=%s d=%d" % (unaligned, d))
    check(g, e, off, ks, unaligned=unaligned, what="mixed")


@pytest.mark.parametrize("seed", range(4))
def test_segmented_random_layouts(seed):
    rng = np.random.default_rng(410 + seed)
    d = int(rng.integers(10_000, 400_000))
    nseg = int(rng.integers(1, 60))
    off = random_layout(rng, d, nseg)
    sizes = np.diff(off)
    ks = np.ceil(sizes * 10.0 ** rng.uniform(-3.5, -0.5, size=nseg)).astype(np.int64)
    ks[rng.random(nseg) < 0.1] = 0
    g = synth.small_gradient(420 + seed, d)
    e = np.zeros(d, np.float32)
    say("segmented random layout seed=%d d=%d nseg=%d" % (seed, d, nseg))
    check(g, e, off, ks, what="random %d" % seed)


@pytest.mark.parametrize("levels", [3, 17])
def test_segmented_ties_at_threshold(levels):
    # few distinct magnitudes: the k-th key is shared by many coordinates
    # and only the lowest indices among them are kept
    rng = np.random.default_rng(430 + levels)
    d = 300_000
    off = random_layout(rng, d, 9)
    sizes = np.diff(off)
    g = (rng.integers(-levels, levels + 1, size=d) * np.float32(0.125)).astype(np.float32)
    e = np.zeros(d, np.float32)
    ks = np.maximum(sizes // 7 + 3, 1)
    say("segmented ties levels=%d" % levels)
    check(g, e, off, ks, lr=np.float32(1.0), what="ties")


def test_segmented_zero_segments_take_lowest_indices():
    # all-zero segments with a partial budget: every key is 0, so the kept
    # set is the k lowest indices (and the candidate region cannot hold the
    # tie bin: the scan path)
    sizes = [100_000, 9, 50_000, 4096]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    d = int(off[-1])
    g = np.zeros(d, np.float32)
    g[100_000:100_009] = 1.0           # segment 1 is not all zero
    g[-1] = -0.0                       # -0 ties with +0
    e = np.zeros(d, np.float32)
    ks = np.array([10, 4, 1234, 4000], dtype=np.int64)
    say("segmented zero segments")
    gi, _, _ = check(g, e, off, ks, what="zeros")
    np.testing.assert_array_equal(np.sort(gi[:10]), np.arange(10))


def test_segmented_large_candidate_sets():
    # a budget of several thousand in a large segment: more candidates than
    # the final pass holds in LDS
    d = 2_000_000
    off = np.array([0, 37, 1_500_000, d], dtype=np.int64)
    ks = np.array([5, 6000, 3000], dtype=np.int64)
    g = synth.small_gradient(440, d)
    e = np.zeros(d, np.float32)
    say("segmented large candidate sets")
    check(g, e, off, ks, what="large")


def test_segmented_large_candidate_sets_many_layers():
    # 400 layers, so the final pass holds at most 3,840 candidates in LDS;
    # in the two large layers 10,000 and 5,000 distinct magnitudes share
    # the digit of the k-th key, so their lists are ranked from global memory
    d = 2_000_000
    small = 37 + 100 * np.arange(397, dtype=np.int64)
    off = np.concatenate([[0], small, [1_500_000, d]]).astype(np.int64)
    ks = np.full(off.size - 1, 2, dtype=np.int64)
    ks[-2:] = [6000, 3000]
    rng = np.random.default_rng(441)
    g = (synth.small_gradient(441, d) * np.float32(1e-3)).astype(np.float32)
    for lo, hi, n in [(off[-3], off[-2], 10_000), (off[-2], off[-1], 5_000)]:
        pos = rng.choice(np.arange(lo, hi), n, replace=False)
        mag = np.float32(1.0) + rng.random(n).astype(np.float32) * np.float32(0.02)
        g[pos] = np.where(rng.random(n) < 0.5, -mag, mag).astype(np.float32)
    e = np.zeros(d, np.float32)
    say("segmented large candidate sets among %d layers" % ks.size)
    check(g, e, off, ks, lr=np.float32(1.0), what="large, many layers")


def test_segmented_special_values():
    d = 5000
    off = np.array([0, 1000, 2500, d], dtype=np.int64)
    rng = np.random.default_rng(450)
    g = (rng.standard_normal(d) * 1e-3).astype(np.float32)
    g[[3, 1500, 4000]] = np.nan
    g[[7, 2600]] = np.inf
    g[[8, 2601]] = -np.inf
    g[[9, 10, 1501]] = np.float32(1e-41)
    g[11] = -0.0
    e = np.zeros(d, np.float32)
    ks = np.array([4, 2, 3], dtype=np.int64)
    say("segmented special values")
    check(g, e, off, ks, what="special")


def test_segmented_one_segment_matches_flat_topk():
    d = 1_000_003
    g = synth.small_gradient(460, d)
    e = np.zeros(d, np.float32)
    k = 1234
    gi, gv, ge, _ = run_gpu(g, e, [0, d], [k])
    ws = efs.new_topk_workspace(d, k)
    ed = dev(e)
    idx = torch.empty(k, dtype=torch.int32, device=DEV)
    val = torch.empty(k, dtype=torch.float32, device=DEV)
    efs.topk_compress(dev(g), ed, LR, k, idx, val, ws)
    fi = idx.cpu().numpy()
    np.testing.assert_array_equal(np.sort(gi), np.sort(fi))
    assert_bits_equal(ge, ed.cpu().numpy())


def test_segmented_ef_loop():
    # five EF steps with e carried, layer-wise budgets at 0.5 %
    rng = np.random.default_rng(470)
    d = 600_000
    off = random_layout(rng, d, 25)
    ks = synth.layerwise_k(off, 0.005)
    e_ref = np.zeros(d, np.float32)
    ed = torch.zeros(d, dtype=torch.float32, device=DEV)
    k_total = int(ks.sum())
    idx = torch.empty(k_total, dtype=torch.int32, device=DEV)
    val = torch.empty(k_total, dtype=torch.float32, device=DEV)
    ws = efs.new_topk_segmented_workspace(ks.size, k_total, DEV)
    ws.zero_()
    offd, kd = dev(off), dev(ks)
    hits = []
    for t in range(5):
        g = synth.small_gradient(480 + t, d)
        efs.topk_segmented_compress(dev(g), ed, LR, offd, kd, idx, val, ws)
        ri, rv, e_ref = oracle.topk_segmented(g, e_ref, LR, off, ks)
        gi = idx.cpu().numpy()
        pos = 0
        for s in range(ks.size):
            n = int(ks[s])
            np.testing.assert_array_equal(np.sort(gi[pos:pos + n]), ri[pos:pos + n])
            pos += n
        assert_bits_equal(ed.cpu().numpy(), e_ref, "e' t=%d" % t)
        hits.append(efs.topk_segmented_bracket_segments(ws))
        say("  segmented EF step %d ok (bracket in %d of %d segments)" % (t, hits[-1], ks.size))
    assert hits[0] == 0          # no hint on the first call
    assert sum(hits[1:]) > 0     # error feedback keeps thresholds close


@pytest.mark.parametrize("case", ["first_offset", "decreasing", "last_offset", "negative_k",
                                  "budget"])
def test_segmented_bad_layout_changes_nothing(case):
    d = 10_000
    off = np.array([0, 3000, 7000, d], dtype=np.int64)
    ks = np.array([10, 20, 30], dtype=np.int64)
    k_total = 60
    if case == "first_offset":
        off[0] = 5
    elif case == "decreasing":
        off[1] = 7500
    elif case == "last_offset":
        off[3] = d - 1
    elif case == "negative_k":
        ks[1] = -1
    else:
        k_total = 59
    g = synth.small_gradient(490, d)
    e = synth.small_gradient(491, d)
    gi, gv, ge, ws = run_gpu(g, e, off, ks, k_total=k_total)
    assert efs.topk_segmented_status(ws) == 1
    assert_bits_equal(ge, e)
    assert np.all(gi == -7)
    # the same workspace then serves a good call
    good_off, good_ks = np.array([0, 3000, 7000, d]), np.array([10, 20, 30])
    gi, gv, ge, _ = run_gpu(g, e, good_off, good_ks, k_total=k_total if case != "budget" else 60,
                            ws=ws if case != "budget" else None)
    assert efs.topk_segmented_status(ws) == (0 if case != "budget" else 1)
    ri, rv, re = oracle.topk_segmented(g, e, LR, good_off, good_ks)
    np.testing.assert_array_equal(np.sort(gi[:60]), np.sort(ri))
    assert_bits_equal(ge, re)


@pytest.mark.parametrize("case", ["first_offset", "decreasing_late", "last_offset",
                                  "negative_k_late", "budget"])
def test_segmented_bad_layout_of_many_layers_changes_nothing(case):
    # 3,000 layers: the layer tables are formed by one workgroup per 512
    # layers in two launches; a defect in a late chunk, at either end of the
    # offsets or in the totals still rejects the whole call
    nseg = 3000
    sizes = (4 + np.arange(nseg) % 7).astype(np.int64)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    d = int(off[-1])
    ks = np.ones(nseg, dtype=np.int64)
    k_total = nseg
    if case == "first_offset":
        off[0] = 1
    elif case == "decreasing_late":
        off[2900] = off[2899] - 1
    elif case == "last_offset":
        off[-1] = d - 1
    elif case == "negative_k_late":
        ks[2600] = -1
    else:
        k_total = nseg - 1
    g = synth.small_gradient(496, d)
    e = synth.small_gradient(497, d)
    gi, gv, ge, ws = run_gpu(g, e, off, ks, k_total=k_total)
    assert efs.topk_segmented_status(ws) == 1
    assert_bits_equal(ge, e)
    assert np.all(gi == -7)


@pytest.mark.parametrize("nseg", [2048, 2049, 2560])
def test_segmented_layer_count_at_the_table_launch_switch(nseg):
    # up to 2048 layers one workgroup forms the tables, above that one
    # workgroup per 512 layers; both must give the same call
    rng = np.random.default_rng(nseg)
    sizes = rng.integers(1, 3000, size=nseg).astype(np.int64)
    sizes[rng.choice(nseg, 8, replace=False)] = 20_000
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    d = int(off[-1])
    ks = synth.layerwise_k(off, 0.01)
    say("segmented layer count %d d=%d" % (nseg, d))
    check(synth.small_gradient(498, d), synth.small_gradient(499, d), off, ks,
          what="%d layers" % nseg)


def test_segmented_workspace_contents_do_not_matter():
    rng = np.random.default_rng(495)
    d = 200_000
    off = random_layout(rng, d, 12)
    ks = synth.layerwise_k(off, 0.01)
    g = synth.small_gradient(496, d)
    e = np.zeros(d, np.float32)
    ri, rv, re = oracle.topk_segmented(g, e, LR, off, ks)
    ws = efs.new_topk_segmented_workspace(ks.size, int(ks.sum()), DEV)
    for fill in (0, 255, 0x3C):
        ws.fill_(fill)
        gi, gv, ge, _ = run_gpu(g, e, off, ks, ws=ws)
        np.testing.assert_array_equal(np.sort(gi), np.sort(ri))
        assert_bits_equal(ge, re)


def _two_calls(gs, off, ks):
    """Calls on one zeroed workspace, e from zero each time; each call
    checked against the oracle.  Returns the bracket count of each call."""
    ws = efs.new_topk_segmented_workspace(len(ks), int(np.sum(ks)), DEV)
    ws.zero_()
    hits = []
    for g in gs:
        e = np.zeros(g.size, np.float32)
        gi, gv, ge, _ = run_gpu(g, e, off, ks, ws=ws)
        ri, rv, re = oracle.topk_segmented(g, e, LR, off, ks)
        np.testing.assert_array_equal(np.sort(gi), np.sort(ri))
        assert_bits_equal(np.sort(gv), np.sort(rv))
        assert_bits_equal(ge, re)
        hits.append(efs.topk_segmented_bracket_segments(ws))
    return hits


def test_segmented_bracket_exactly_k_above():
    # the first call puts the threshold at |p| = 1.0; on the second exactly k
    # keys (1.05) lie above the bracket around it and three more (1.0)
    # inside: the bracket is confirmed with nothing left to take from the
    # candidates
    rng = np.random.default_rng(660)
    d0, k0 = 3 * 4096, 10
    off = np.array([0, d0, d0 + 20_000], dtype=np.int64)
    ks = np.array([k0, 0], dtype=np.int64)
    tiny = lambda n: rng.uniform(-1e-2, 1e-2, size=n).astype(np.float32)
    pos = rng.choice(d0, 13, replace=False)
    g1 = np.concatenate([tiny(d0), synth.small_gradient(661, 20_000)])
    g1[pos[:10]] = np.float32(10.0)
    g2 = np.concatenate([tiny(d0), synth.small_gradient(662, 20_000)])
    g2[pos[:10]] = np.float32(-10.5)
    g2[pos[10:]] = np.float32(10.0)
    say("segmented bracket with exactly k pairs above it")
    hits = _two_calls([g1, g2], off, ks)
    assert hits == [0, 1]


def test_segmented_bracket_bin_too_large_falls_back():
    # 2,200 keys tied at the threshold share one bracket bin; with the
    # candidates they exceed the segment's candidate region (16 k + 4096), so
    # the bin cannot be listed and the radix path takes over
    rng = np.random.default_rng(670)
    d0, k0 = 2 * 4096, 10
    off = np.array([0, d0], dtype=np.int64)
    ks = np.array([k0], dtype=np.int64)
    g = rng.uniform(-1e-2, 1e-2, size=d0).astype(np.float32)
    pos = rng.choice(d0, 2205, replace=False)
    g[pos[:2200]] = np.float32(10.0)
    g[pos[2200:]] = np.float32(10.1)
    say("segmented bracket bin too large for the list")
    hits = _two_calls([g, g], off, ks)
    assert hits == [0, 0]


def test_segmented_bracket_bin_listed():
    # the same shape with 2,000 tied keys: the bin fits after the candidates,
    # is listed by pass 2 and ranked by index in the final pass
    rng = np.random.default_rng(680)
    d0, k0 = 2 * 4096, 10
    off = np.array([0, d0], dtype=np.int64)
    ks = np.array([k0], dtype=np.int64)
    g = rng.uniform(-1e-2, 1e-2, size=d0).astype(np.float32)
    pos = rng.choice(d0, 2005, replace=False)
    g[pos[:2000]] = np.float32(10.0)
    g[pos[2000:]] = np.float32(-10.1)
    say("segmented bracket bin listed")
    hits = _two_calls([g, g], off, ks)
    assert hits == [0, 1]


def test_segmented_bracket_from_another_scale_falls_back():
    # hints learned on one scale make a bracket that misses the next call's
    # thresholds (50x larger): the radix path takes over, results exact; the
    # call after that, on the same scale, selects from the bracket
    rng = np.random.default_rng(497)
    d = 300_000
    off = random_layout(rng, d, 10)
    ks = synth.layerwise_k(off, 0.01)
    ws = efs.new_topk_segmented_workspace(ks.size, int(ks.sum()), DEV)
    ws.zero_()   # no hints yet (a reused allocation could hold some)
    g1 = synth.small_gradient(498, d)
    g2 = (synth.small_gradient(499, d) * np.float32(50.0)).astype(np.float32)
    e = np.zeros(d, np.float32)
    hits = []
    for g in (g1, g2, g2):
        gi, gv, ge, _ = run_gpu(g, e, off, ks, ws=ws)
        ri, rv, re = oracle.topk_segmented(g, e, LR, off, ks)
        np.testing.assert_array_equal(np.sort(gi), np.sort(ri))
        assert_bits_equal(ge, re)
        hits.append(efs.topk_segmented_bracket_segments(ws))
    assert hits[0] == 0 and hits[1] == 0
    assert hits[2] == ks.size


def small_layer_layout(rng, nseg):
    """Mostly small layers (1 to 1100 elements, so that runs of them fit one
    4096-element block each and others straddle two), with empty layers and
    exact sizes 1, 64, 65, 1023, 1024, 1025 mixed in."""
    sizes = np.exp(rng.uniform(0.0, np.log(1100.0), size=nseg)).astype(np.int64)
    special = np.array([0, 1, 64, 65, 1023, 1024, 1025, 0], dtype=np.int64)
    pick = rng.random(nseg) < 0.15
    sizes[pick] = special[rng.integers(0, special.size, size=int(pick.sum()))]
    return np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)


@pytest.mark.parametrize("nseg,unaligned", [(700, False), (700, True), (5000, False)])
def test_segmented_small_layers_by_wave(nseg, unaligned):
    # one-tile layers of at most 1,024 elements with k <= 8 or k >= size are
    # selected a wave each, up to four at once; every k from 0 to 9 and k at
    # or past the size, ties among quantised values, two error-feedback calls
    # (above 4,096 layers the sweeps take longer slices)
    rng = np.random.default_rng(4600 + nseg + int(unaligned))
    off = small_layer_layout(rng, nseg)
    sizes = np.diff(off)
    d = int(off[-1])
    ks = rng.integers(0, 10, size=nseg).astype(np.int64)
    full = rng.random(nseg) < 0.08
    ks[full] = sizes[full] + rng.integers(0, 3, size=int(full.sum()))
    g = synth.small_gradient(4610 + nseg, d)
    g = (np.round(g / np.float32(2e-4)) * np.float32(2e-4)).astype(np.float32)  # ties
    e = np.zeros(d, np.float32)
    one_tile = np.array([(sz > 0) and (o // 4096 == (o + sz - 1) // 4096) for o, sz in zip(off[:-1], sizes)])
    wave = one_tile & (sizes <= 1024) & ((ks <= 8) | (ks >= sizes))
    say("segmented small layers nseg=%d unaligned=%s d=%d, %d by wave" % (nseg, unaligned, d, int(wave.sum())))
    assert wave.sum() > nseg // 2
    for step in range(2):
        _, _, e = check(g, e, off, ks, unaligned=unaligned, what="small layers step %d" % step)
        e = e.copy()


def test_segmented_bracket_small_bins_with_ties():
    # two- to four-tile layers on the bracket path whose bin of the k-th key
    # holds a few tied keys (ranked a wave per layer in the final pass,
    # ties to the lower index): g on a power-of-two grid and lr = 1 keep
    # p = e + g exact, so equal magnitudes stay equal from step to step
    rng = np.random.default_rng(4700)
    sizes = rng.integers(4500, 16000, size=400).astype(np.int64)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    d = int(off[-1])
    ks = np.ceil(sizes * 0.002).astype(np.int64)
    e = np.zeros(d, np.float32)
    ws = efs.new_topk_segmented_workspace(ks.size, int(ks.sum()), DEV)
    hits, split_ties = [], 0
    say("segmented bracket small bins with ties d=%d" % d)
    for t in range(5):
        g = (np.round(rng.standard_normal(d) * 8.0) * 2.0 ** -13).astype(np.float32)
        gi, gv, ge, _ = run_gpu(g, e, off, ks, lr=1.0, ws=ws)
        ri, rv, re = oracle.topk_segmented(g, e, 1.0, off, ks)
        pos = 0
        for s_ in range(ks.size):
            n = int(ks[s_])
            o = np.argsort(gi[pos:pos + n], kind="stable")
            np.testing.assert_array_equal(gi[pos:pos + n][o], ri[pos:pos + n], "step %d segment %d" % (t, s_))
            assert_bits_equal(gv[pos:pos + n][o], rv[pos:pos + n], "step %d segment %d values" % (t, s_))
            pos += n
        assert_bits_equal(ge, re, "step %d e'" % t)
        hits.append(efs.topk_segmented_bracket_segments(ws))
        if t > 0:
            # layers whose k-th magnitude is shared by kept and dropped
            # coordinates, at most 64 of them (a bracket bin here spans one
            # grid level, so the bin ranked in the final pass is the tie)
            p = (e + g).astype(np.float32)
            pos = 0
            for s_ in range(ks.size):
                n = int(ks[s_])
                mag = np.abs(p[off[s_]:off[s_ + 1]])
                kth = np.abs(rv[pos:pos + n]).min()
                tied = int(np.sum(mag == kth))
                kept = int(np.sum(np.abs(rv[pos:pos + n]) == kth))
                split_ties += int(kept < tied <= 64)
                pos += n
        e = re
    say("  bracket layers per step: %s, split ties %d" % (hits, split_ties))
    assert hits[0] == 0 and sum(hits[1:]) > 0
    assert split_ties > 0


@pytest.mark.parametrize("unaligned", [False, True])
def test_segmented_light_layers_miss_their_brackets(unaligned):
    # layers of two to four tiles starting anywhere in a block (the sizes
    # whose bracket path keeps no digit-1 histogram), error feedback carried:
    # the thresholds grow over the first steps and leave the brackets, settle
    # on one scale, then a 30x jump puts every threshold above its bracket,
    # a 100x drop follows and a quantised step ties many keys; a missed
    # layer's digit-1 histogram then comes from its elements.  Every step
    # against the oracle
    rng = np.random.default_rng(4242)
    sizes = rng.integers(4097, 3 * 4096 + 4000, size=60)
    sizes[::7] = rng.integers(1, 4000, size=sizes[::7].size)   # one-tile layers among them
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    d = int(off[-1])
    ks = synth.layerwise_k(off, 0.01)
    k_total = int(ks.sum())
    ws = efs.new_topk_segmented_workspace(ks.size, k_total, DEV)
    e = np.zeros(d, np.float32)
    scales = [1.0] * 8 + [30.0] * 3 + [0.01, 1.0]
    hits = []
    say("segmented light layers d=%d nseg=%d unaligned=%s" % (d, ks.size, unaligned))
    for t, sc in enumerate(scales):
        g = (synth.small_gradient(4300 + t, d) * np.float32(sc)).astype(np.float32)
        if t == len(scales) - 1:
            g = (np.round(g / np.float32(4e-4)) * np.float32(4e-4)).astype(np.float32)
        gi, gv, ge, _ = run_gpu(g, e, off, ks, k_total=k_total, ws=ws, unaligned=unaligned)
        assert efs.topk_segmented_status(ws) == 0
        ri, rv, re = oracle.topk_segmented(g, e, LR, off, ks)
        order = np.lexsort((gi, np.repeat(np.arange(ks.size), np.minimum(ks, sizes))))
        np.testing.assert_array_equal(gi[order], ri, "t=%d indices" % t)
        assert_bits_equal(gv[order], rv, "t=%d values" % t)
        assert_bits_equal(ge, re, "t=%d e'" % t)
        e = re
        hits.append(efs.topk_segmented_bracket_segments(ws))
        say("  step %d scale %g ok (bracket in %d layers)" % (t, sc, hits[-1]))
    multi = int(np.sum(sizes > 4096))
    assert min(hits[1:4]) < multi // 4   # growing thresholds: most brackets missed
    assert hits[7] > multi // 2          # settled on one scale: brackets hold
    assert hits[8] < multi // 4          # the jump: most brackets missed


@pytest.mark.parametrize("levels", [4, 1000])
def test_segmented_many_small_layers(levels):
    # hundreds of layers that fit in one 4096-element tile (selected inside
    # pass 1) mixed with a few large ones; few magnitudes -> ties at nearly
    # every threshold, split by index
    rng = np.random.default_rng(600 + levels)
    sizes = rng.integers(1, 4097, size=700)
    sizes[rng.choice(700, 5, replace=False)] = rng.integers(5000, 60000, size=5)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    d = int(off[-1])
    half = levels // 2
    g = (rng.integers(-half, half + 1, size=d) * np.float32(0.125)).astype(np.float32)
    e = np.zeros(d, np.float32)
    ks = np.ceil(sizes * rng.uniform(0.0, 1.2, size=sizes.size)).astype(np.int64)
    say("segmented many small layers levels=%d d=%d" % (levels, d))
    check(g, e, off, ks, lr=np.float32(1.0), what="small layers")


def test_segmented_thousands_of_layers_ef_loop():
    # 5,000 layers (the reset scans the layer table 512 layers at a time: ten
    # chunks), mostly within one tile, some spanning many; three EF steps
    rng = np.random.default_rng(990)
    sizes = np.exp(rng.uniform(np.log(1), np.log(2000), size=5000)).astype(np.int64)
    sizes[rng.choice(5000, 40, replace=False)] = rng.integers(8000, 40000, size=40)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    d = int(off[-1])
    ks = synth.layerwise_k(off, 0.01)
    k_total = int(ks.sum())
    e_ref = np.zeros(d, np.float32)
    ed = torch.zeros(d, dtype=torch.float32, device=DEV)
    idx = torch.empty(k_total, dtype=torch.int32, device=DEV)
    val = torch.empty(k_total, dtype=torch.float32, device=DEV)
    ws = efs.new_topk_segmented_workspace(ks.size, k_total, DEV)
    ws.zero_()
    offd, kd = dev(off), dev(ks)
    say("segmented thousands of layers d=%d nseg=%d k=%d" % (d, ks.size, k_total))
    for t in range(3):
        g = synth.small_gradient(995 + t, d)
        efs.topk_segmented_compress(dev(g), ed, LR, offd, kd, idx, val, ws)
        assert efs.topk_segmented_status(ws) == 0
        ri, rv, e_ref = oracle.topk_segmented(g, e_ref, LR, off, ks)
        gi, gv = idx.cpu().numpy(), val.cpu().numpy()
        # layer regions in order: sort each region by index, then compare
        order = np.lexsort((gi, np.repeat(np.arange(ks.size), ks)))
        np.testing.assert_array_equal(gi[order], ri, "t=%d indices" % t)
        assert_bits_equal(gv[order], rv, "t=%d values" % t)
        assert_bits_equal(ed.cpu().numpy(), e_ref, "e' t=%d" % t)
        say("  step %d ok (bracket in %d layers)" % (t, efs.topk_segmented_bracket_segments(ws)))


def test_segmented_twenty_thousand_layers_ef_steps():
    # 20,000 layers over 25.6e6 (log-uniform sizes from 1 to 10^4 before
    # scaling): more layers than two rounds of the tile-to-layer search
    # cover, so the sweeps take long slices; most layers lie in one tile and
    # the final pass runs with its small LDS buffer.  Four error-feedback
    # steps on one workspace (the later ones mostly from the brackets), each
    # against the oracle
    d, nseg = 25_600_000, 20_000
    sizes = synth.segment_sizes(7, nseg, d, lo=1.0, hi=1e4)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    ks = synth.layerwise_k(off, 0.001)
    k_total = int(ks.sum())
    e_ref = np.zeros(d, np.float32)
    ed = torch.zeros(d, dtype=torch.float32, device=DEV)
    idx = torch.empty(k_total, dtype=torch.int32, device=DEV)
    val = torch.empty(k_total, dtype=torch.float32, device=DEV)
    ws = efs.new_topk_segmented_workspace(nseg, k_total, DEV)
    offd, kd = dev(off), dev(ks)
    say("segmented 20,000 layers d=%d k=%d" % (d, k_total))
    for t in range(4):
        g = synth.small_gradient(2000 + t, d)
        efs.topk_segmented_compress(dev(g), ed, LR, offd, kd, idx, val, ws)
        assert efs.topk_segmented_status(ws) == 0
        ri, rv, e_ref = oracle.topk_segmented(g, e_ref, LR, off, ks)
        gi, gv = idx.cpu().numpy(), val.cpu().numpy()
        order = np.lexsort((gi, np.repeat(np.arange(nseg), ks)))
        np.testing.assert_array_equal(gi[order], ri, "t=%d indices" % t)
        assert_bits_equal(gv[order], rv, "t=%d values" % t)
        assert_bits_equal(ed.cpu().numpy(), e_ref, "e' t=%d" % t)
        say("  step %d ok (bracket in %d layers)" % (t, efs.topk_segmented_bracket_segments(ws)))
    assert efs.topk_segmented_bracket_segments(ws) >= 500  # 687 on this input


@pytest.mark.parametrize("seed", range(8))
def test_segmented_randomised_ef_loops(seed):
    # random layouts (empty, one-tile and multi-tile layers), random budgets,
    # six EF steps on one workspace with the gradient scale sometimes jumping
    # and some steps quantised (heavy ties): every step against the oracle,
    # whichever path each layer takes
    rng = np.random.default_rng(900 + seed)
    d = int(rng.integers(20_000, 300_000))
    nseg = int(rng.integers(1, 80))
    off = random_layout(rng, d, nseg)
    sizes = np.diff(off)
    ks = np.ceil(sizes * 10.0 ** rng.uniform(-3.0, -0.3, size=nseg)).astype(np.int64)
    ks[rng.random(nseg) < 0.1] = 0
    ks[rng.random(nseg) < 0.05] = 10 ** 9  # more than the layer holds: all kept
    k_total = int(np.minimum(ks, sizes).sum())
    ws = efs.new_topk_segmented_workspace(nseg, k_total, DEV)
    ws.zero_()
    e = np.zeros(d, np.float32)
    hits = []
    say("segmented randomised seed=%d d=%d nseg=%d" % (seed, d, nseg))
    for t in range(6):
        scale = np.float32(10.0 ** rng.choice([0.0, 0.0, 0.0, 1.5, -1.0]))
        g = (synth.small_gradient(910 + 10 * seed + t, d) * scale).astype(np.float32)
        if rng.random() < 0.3:
            g = (np.round(g / np.float32(2e-3)) * np.float32(2e-3)).astype(np.float32)
        gi, gv, ge, _ = run_gpu(g, e, off, ks, k_total=k_total, ws=ws)
        assert efs.topk_segmented_status(ws) == 0
        ri, rv, re = oracle.topk_segmented(g, e, LR, off, ks)
        pos = 0
        for s in range(nseg):
            n = int(min(ks[s], sizes[s]))
            o = np.argsort(gi[pos:pos + n], kind="stable")
            np.testing.assert_array_equal(gi[pos:pos + n][o], ri[pos:pos + n],
                                          "seed %d t=%d segment %d" % (seed, t, s))
            assert_bits_equal(gv[pos:pos + n][o], rv[pos:pos + n],
                              "seed %d t=%d segment %d" % (seed, t, s))
            pos += n
        assert_bits_equal(ge, re, "seed %d t=%d e'" % (seed, t))
        hits.append(efs.topk_segmented_bracket_segments(ws))
        e = re
    say("  bracket segments per step: %s" % hits)
