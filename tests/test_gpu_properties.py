"""Randomised parity of every entry point against the oracle (hypothesis,
derandomised so that a run is repeatable).  Each example draws a size
(ragged, 1 to 20,000 elements, so tiles, layers and ranges end anywhere), an
input family (Gaussian, a few repeated magnitudes so that ties decide
Top-k, wide exponent spread, or sparse with exact zeros), special values
planted at random positions (±0, ±inf, NaN, subnormals, the largest
finite float), and the call's parameters; the device result must equal the
oracle's bit for bit (NaN compared by position: which NaN payload an
operation returns is not part of the method).

Hard threshold: Algorithm 1 with §4.2's S_lambda; Top-k and layer-wise
Top-k: Lemma 2 with ties to the lower index, App. C.5; the average:
Algorithm 1's exchange-and-average in worker order (both workspace
layouts), and the model update of App. C.6.2."""
import numpy as np
import pytest

hypothesis = pytest.importorskip("hypothesis")
from hypothesis import HealthCheck, given, settings  # noqa: E402
from hypothesis import strategies as st  # noqa: E402

import oracle  # noqa: E402
from paper_2108_00951_amd import synth  # noqa: E402
from tests._checks import bits, canonical  # noqa: E402

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2108_00951_amd import binding as efs  # noqa: E402

DEV = "cuda"
LR = synth.LR
SETTINGS = settings(max_examples=150, deadline=None, derandomize=True, database=None,
                    suppress_health_check=[HealthCheck.too_slow])
FAMILIES = ["gauss", "ties", "spread", "sparse"]
SPECIALS = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 1e-45, -3e-44, 1e-39,
                     np.finfo(np.float32).max, -np.finfo(np.float32).max], dtype=np.float32)


def draw(rng, d, family, n_special):
    if family == "gauss":
        x = rng.standard_normal(d) * 1e-3
    elif family == "ties":
        x = rng.choice(np.array([-3e-3, -1e-3, 0.0, 1e-3, 2e-3, 3e-3]), size=d)
    elif family == "spread":
        x = rng.standard_normal(d) * 10.0 ** rng.integers(-30, 30, size=d)
    else:
        x = np.where(rng.random(d) < 0.1, rng.standard_normal(d), 0.0)
    x = x.astype(np.float32)
    if n_special and d:
        pos = rng.choice(d, min(d, n_special), replace=False)
        x[pos] = rng.choice(SPECIALS, size=pos.size)
    return x


def same_floats(a, b, what):
    a = np.asarray(a, np.float32)
    b = np.asarray(b, np.float32)
    assert a.shape == b.shape, what
    na, nb = np.isnan(a), np.isnan(b)
    np.testing.assert_array_equal(na, nb, err_msg=what + ": NaN positions")
    np.testing.assert_array_equal(bits(a[~na]), bits(b[~nb]), err_msg=what)


def dev(a, unaligned=False):
    a = np.ascontiguousarray(a)
    if not unaligned:
        return torch.from_numpy(a).to(DEV)
    buf = torch.empty(a.size + 1, dtype=torch.from_numpy(a[:0]).dtype, device=DEV)
    v = buf[1:]
    v.copy_(torch.from_numpy(a))
    return v


def inputs():
    return st.tuples(st.integers(0, 2 ** 32 - 1), st.integers(1, 20_000),
                     st.sampled_from(FAMILIES), st.integers(0, 40))


@SETTINGS
@given(inputs(), st.sampled_from(["zero", "quantile", "inf", "tiny"]), st.booleans())
def test_property_hard_threshold(inp, lam_kind, unaligned):
    seed, d, family, n_special = inp
    rng = np.random.default_rng(seed)
    g, e = draw(rng, d, family, n_special), draw(rng, d, family, n_special // 2)
    finite = np.abs(g[np.isfinite(g)])
    lam = {"zero": 0.0, "inf": np.inf, "tiny": 1e-44,
           "quantile": float(np.quantile(finite, 0.9)) * float(LR) if finite.size else 1.0}[lam_kind]
    lam = np.float32(lam)
    idx = torch.empty(d, dtype=torch.int32, device=DEV)
    val = torch.empty(d, dtype=torch.float32, device=DEV)
    ctr = efs.new_counter(DEV)
    ed = dev(e, unaligned)
    efs.ht_compress(dev(g, unaligned), ed, LR, lam, idx, val, ctr)
    k = efs.counter_value(ctr)
    ri, rv, re, rk = oracle.ht(g, e, LR, lam)
    assert k == rk
    gi, gv = canonical(idx[:k].cpu().numpy(), val[:k].cpu().numpy())
    np.testing.assert_array_equal(gi, ri)
    same_floats(gv, rv, "payload values")
    same_floats(ed.cpu().numpy(), re, "e'")


@SETTINGS
@given(inputs(), st.floats(0.0, 1.0), st.booleans())
def test_property_topk_two_calls(inp, kfrac, unaligned):
    # two error-feedback calls on one workspace: the second may select from
    # the first call's bracket
    seed, d, family, n_special = inp
    rng = np.random.default_rng(seed)
    k = int(round(kfrac * d))
    e = draw(rng, d, family, n_special // 2)
    ed = dev(e, unaligned)
    ws = efs.new_topk_workspace(d, k, DEV)
    idx = torch.empty(max(k, 1), dtype=torch.int32, device=DEV)[:k]
    val = torch.empty(max(k, 1), dtype=torch.float32, device=DEV)[:k]
    for t in range(2):
        g = draw(rng, d, family, n_special)
        efs.topk_compress(dev(g, unaligned), ed, LR, k, idx, val, ws)
        ri, rv, e = oracle.topk(g, e, LR, k)
        gi, gv = canonical(idx.cpu().numpy(), val.cpu().numpy())
        np.testing.assert_array_equal(gi, ri, err_msg="call %d indices" % t)
        same_floats(gv, rv, "call %d values" % t)
        same_floats(ed.cpu().numpy(), e, "call %d e'" % t)


@SETTINGS
@given(inputs(), st.integers(1, 24), st.floats(0.0, 0.5))
def test_property_layerwise_topk(inp, nseg, kfrac):
    seed, d, family, n_special = inp
    rng = np.random.default_rng(seed)
    cuts = np.sort(rng.integers(0, d + 1, size=nseg - 1))
    off = np.concatenate([[0], cuts, [d]]).astype(np.int64)
    sizes = np.diff(off)
    ks = np.minimum(sizes, np.round(kfrac * sizes + rng.integers(0, 3, size=nseg))).astype(np.int64)
    k_total = int(ks.sum())
    e = draw(rng, d, family, n_special // 2)
    ed = dev(e)
    ws = efs.new_topk_segmented_workspace(nseg, k_total, DEV)
    idx = torch.empty(max(k_total, 1), dtype=torch.int32, device=DEV)[:k_total]
    val = torch.empty(max(k_total, 1), dtype=torch.float32, device=DEV)[:k_total]
    offd, kd = dev(off), dev(ks)
    for t in range(2):
        g = draw(rng, d, family, n_special)
        efs.topk_segmented_compress(dev(g), ed, LR, offd, kd, idx, val, ws)
        assert efs.topk_segmented_status(ws) == 0
        ri, rv, e = oracle.topk_segmented(g, e, LR, off, ks)
        gi, gv = idx.cpu().numpy(), val.cpu().numpy()
        pos = 0
        for s in range(nseg):
            n = int(ks[s])
            si, sv = canonical(gi[pos:pos + n], gv[pos:pos + n])
            np.testing.assert_array_equal(si, ri[pos:pos + n], err_msg="call %d layer %d" % (t, s))
            same_floats(sv, rv[pos:pos + n], "call %d layer %d values" % (t, s))
            pos += n
        same_floats(ed.cpu().numpy(), e, "call %d e'" % t)


@SETTINGS
@given(inputs(), st.integers(1, 6), st.sampled_from(efs.LAYOUTS),
       st.sampled_from(["average", "sgd", "momentum"]))
def test_property_average_and_update(inp, n, layout, mode):
    seed, d, family, n_special = inp
    rng = np.random.default_rng(seed)
    p_dev, p_ref = [], []
    for w in range(n):
        c = int(rng.integers(0, d + 1))
        i = np.sort(rng.choice(d, c, replace=False)) if c else np.zeros(0, np.int64)
        rng.shuffle(i)   # the pair order of a payload is open
        i = i.astype(np.int32)
        v = draw(rng, c, family, n_special // 4) if c else np.zeros(0, np.float32)
        p_dev.append((dev(i), dev(v)))
        p_ref.append((i, v))
    ws = efs.new_apply_workspace(p_dev, d, DEV, layout=layout)
    x0 = draw(rng, d, "gauss", n_special // 4)
    m0 = (rng.standard_normal(d) * 1e-3).astype(np.float32)
    x, m = dev(x0), dev(m0)
    code = {"average": efs.APPLY_AVERAGE, "sgd": efs.APPLY_SGD, "momentum": efs.APPLY_MOMENTUM}[mode]
    efs.sparse_apply(p_dev, d, code, x, ws, m=m if mode == "momentum" else None,
                     beta=0.9, gamma=0.05)
    assert efs.sparse_status(ws) == 0
    if mode == "average":
        same_floats(x.cpu().numpy(), oracle.accumulate(p_ref, d), "average")
    elif mode == "sgd":
        want, _ = oracle.update(p_ref, x0, 1)
        same_floats(x.cpu().numpy(), want, "x after sgd")
    else:
        want_x, want_m = oracle.update(p_ref, x0, 2, m=m0, beta=0.9, gamma=0.05)
        same_floats(m.cpu().numpy(), want_m, "m")
        same_floats(x.cpu().numpy(), want_x, "x after momentum")
