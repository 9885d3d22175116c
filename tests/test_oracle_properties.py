"""Randomised pins of the oracle against the definitions it implements
(hypothesis, derandomised), on small inputs with ties and special values.
Each property is stated from the paper, not from the oracle's code:

  * hard threshold (§4.2, S_lambda(x) = { i : |x_i| >= lambda }; Algorithm 1):
    the payload is exactly the coordinates of p = fl(e + fl(lr g)) with
    |p_i| >= lambda, in ascending order, with p_i's bits; e' is +0 there and
    p elsewhere;
  * Top-k (Lemma 2, ties to the lower index): exactly min(k, d) pairs; every
    kept key is at least every dropped key, and a dropped key equal to a kept
    one has the larger index; e' is +0 at the kept coordinates and p
    elsewhere;
  * Lemma 3: with lambda the K-th largest magnitude and no tie at it, the
    hard threshold and Top-K keep the same set;
  * layer-wise Top-k (App. C.5): each layer is the flat Top-k of that layer;
  * the average (Algorithm 1's exchange and average): the fp32 sum in worker
    order, then one division by n;
  * the multi-core build returns the same bits as the single-threaded one.
"""
import numpy as np
import pytest

hypothesis = pytest.importorskip("hypothesis")
from hypothesis import HealthCheck, given, settings  # noqa: E402
from hypothesis import strategies as st  # noqa: E402

import oracle  # noqa: E402
from tests._checks import bits  # noqa: E402

LR = np.float32(0.1)
SETTINGS = settings(max_examples=200, deadline=None, derandomize=True, database=None,
                    suppress_health_check=[HealthCheck.too_slow])
SPECIALS = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 1e-45, -3e-44,
                     np.finfo(np.float32).max], dtype=np.float32)


def draw(rng, d, family, n_special):
    if family == "gauss":
        x = rng.standard_normal(d) * 1e-3
    elif family == "ties":
        x = rng.choice(np.array([-2e-3, -1e-3, 0.0, 1e-3, 2e-3]), size=d)
    else:
        x = rng.standard_normal(d) * 10.0 ** rng.integers(-20, 20, size=d)
    x = x.astype(np.float32)
    if n_special and d:
        pos = rng.choice(d, min(d, n_special), replace=False)
        x[pos] = rng.choice(SPECIALS, size=pos.size)
    return x


def inputs(max_d=3000):
    return st.tuples(st.integers(0, 2 ** 32 - 1), st.integers(1, max_d),
                     st.sampled_from(["gauss", "ties", "spread"]), st.integers(0, 12))


def ef_p(g, e):
    # fl(e + fl(lr g)) element by element in fp32 (numpy rounds each op)
    with np.errstate(invalid="ignore", over="ignore"):
        return (e + (LR * g).astype(np.float32)).astype(np.float32)


def keys(p):
    return bits(np.abs(p))


@SETTINGS
@given(inputs(), st.sampled_from([0.0, 1e-4, 1e-3, np.inf]))
def test_hard_threshold_is_its_definition(inp, lam):
    seed, d, family, n_special = inp
    rng = np.random.default_rng(seed)
    g, e = draw(rng, d, family, n_special), draw(rng, d, family, n_special)
    lam = np.float32(lam)
    idx, val, e2, k = oracle.ht(g, e, LR, lam)
    p = ef_p(g, e)
    with np.errstate(invalid="ignore"):
        kept = np.abs(p) >= lam          # NaN compares false: never kept
    assert k == int(kept.sum())
    np.testing.assert_array_equal(idx, np.nonzero(kept)[0])
    np.testing.assert_array_equal(bits(val), bits(p[kept]))
    want = p.copy()
    want[kept] = np.float32(0.0)
    np.testing.assert_array_equal(bits(e2), bits(want))


@SETTINGS
@given(inputs(), st.floats(0.0, 1.0))
def test_topk_is_its_definition(inp, kfrac):
    seed, d, family, n_special = inp
    rng = np.random.default_rng(seed)
    g, e = draw(rng, d, family, n_special), draw(rng, d, family, n_special)
    k = int(round(kfrac * d))
    idx, val, e2 = oracle.topk(g, e, LR, k)
    p = ef_p(g, e)
    assert idx.size == min(k, d)
    kept = np.zeros(d, bool)
    kept[idx] = True
    assert int(kept.sum()) == idx.size          # distinct indices
    kk, dk = keys(p[kept]), keys(p[~kept])
    if kk.size and dk.size:
        assert kk.min() >= dk.max()
        tie = kk.min()
        if (dk == tie).any():
            assert np.nonzero(kept & (keys(p) == tie))[0].max() < \
                np.nonzero(~kept & (keys(p) == tie))[0].min()
    np.testing.assert_array_equal(bits(val), bits(p[idx]))
    want = p.copy()
    want[kept] = np.float32(0.0)
    np.testing.assert_array_equal(bits(e2), bits(want))


@SETTINGS
@given(inputs(), st.floats(0.001, 0.5))
def test_lemma3_threshold_at_kth_magnitude_equals_topk(inp, kfrac):
    seed, d, family, _ = inp
    rng = np.random.default_rng(seed)
    g = draw(rng, d, family, 0)
    e = np.zeros(d, np.float32)
    K = max(1, int(round(kfrac * d)))
    p = ef_p(g, e)
    a = np.sort(np.abs(p))[::-1]
    lam = a[K - 1]
    if K < d and a[K] == lam:
        return   # a tie at the K-th magnitude: Lemma 3 assumes none
    hi, hv, _, _ = oracle.ht(g, e, LR, lam)
    ti, tv, _ = oracle.topk(g, e, LR, K)
    np.testing.assert_array_equal(np.sort(ti), hi)


@SETTINGS
@given(inputs(), st.integers(1, 12), st.floats(0.0, 0.6))
def test_layerwise_topk_is_flat_topk_per_layer(inp, nseg, kfrac):
    seed, d, family, n_special = inp
    rng = np.random.default_rng(seed)
    g, e = draw(rng, d, family, n_special), draw(rng, d, family, n_special)
    cuts = np.sort(rng.integers(0, d + 1, size=nseg - 1))
    off = np.concatenate([[0], cuts, [d]]).astype(np.int64)
    ks = np.round(kfrac * np.diff(off)).astype(np.int64)
    idx, val, e2 = oracle.topk_segmented(g, e, LR, off, ks)
    pos = 0
    for s in range(nseg):
        lo, hi = int(off[s]), int(off[s + 1])
        fi, fv, fe = oracle.topk(g[lo:hi], e[lo:hi], LR, int(ks[s]))
        n = fi.size
        np.testing.assert_array_equal(idx[pos:pos + n], fi + lo)
        np.testing.assert_array_equal(bits(val[pos:pos + n]), bits(fv))
        np.testing.assert_array_equal(bits(e2[lo:hi]), bits(fe))
        pos += n
    assert pos == idx.size


@SETTINGS
@given(inputs(2000), st.integers(1, 6))
def test_average_is_in_order_sum_then_division(inp, n):
    seed, d, family, n_special = inp
    rng = np.random.default_rng(seed)
    payloads = []
    acc = np.zeros(d, np.float32)
    with np.errstate(invalid="ignore", over="ignore"):
        for w in range(n):
            c = int(rng.integers(0, d + 1))
            i = rng.choice(d, c, replace=False).astype(np.int32)
            v = draw(rng, c, family, n_special) if c else np.zeros(0, np.float32)
            payloads.append((i, v))
            acc[i] = (acc[i] + v).astype(np.float32)   # worker w after workers < w
        want = acc if n == 1 else (acc / np.float32(n)).astype(np.float32)
    got = oracle.accumulate(payloads, d)
    nan = np.isnan(want)
    np.testing.assert_array_equal(np.isnan(got), nan)
    np.testing.assert_array_equal(bits(got[~nan]), bits(want[~nan]))


@SETTINGS
@given(inputs(), st.floats(0.0, 1.0), st.sampled_from([0.0, 1e-3, np.inf]))
def test_multicore_oracle_returns_the_same_bits(inp, kfrac, lam):
    seed, d, family, n_special = inp
    rng = np.random.default_rng(seed)
    g, e = draw(rng, d, family, n_special), draw(rng, d, family, n_special)
    a = oracle.ht(g, e, LR, np.float32(lam))
    b = oracle.ht(g, e, LR, np.float32(lam), mt=True)
    assert a[3] == b[3]
    for x, y in zip(a[:3], b[:3]):
        np.testing.assert_array_equal(np.asarray(x).view(np.uint32), np.asarray(y).view(np.uint32))
    k = int(round(kfrac * d))
    a = oracle.topk(g, e, LR, k)
    b = oracle.topk(g, e, LR, k, mt=True)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(np.asarray(x).view(np.uint32), np.asarray(y).view(np.uint32))
