"""Comparison helpers shared by the GPU parity tests (no method arithmetic
beyond reading bit patterns; expected values always come from the oracle)."""
import numpy as np


def bits(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


def canonical(idx, val):
    """Payload pairs sorted by index (the ABI leaves the pair order open)."""
    idx = np.asarray(idx)
    order = np.argsort(idx, kind="stable")
    return idx[order], np.asarray(val)[order]


def assert_payload_equal(gidx, gval, ridx, rval, what=""):
    gi, gv = canonical(gidx, gval)
    assert gi.size == ridx.size, "%s: %d pairs vs oracle %d" % (what, gi.size, ridx.size)
    np.testing.assert_array_equal(gi, ridx, err_msg=what + " indices")
    np.testing.assert_array_equal(bits(gv), bits(rval), err_msg=what + " values")


def assert_bits_equal(a, b, what=""):
    ab, bb = bits(a), bits(b)
    if not np.array_equal(ab, bb):
        bad = np.nonzero(ab != bb)[0]
        raise AssertionError("%s: %d of %d elements differ; first at %d: %r vs %r"
                             % (what, bad.size, ab.size, bad[0], a[bad[0]], b[bad[0]]))


def check_topk_properties(acc, k, idx, val, e_next):
    """The Top-k payload is unique given acc: exactly the k first coordinates
    under (|p| bit pattern descending, index ascending).  Checks that
    (idx, val, e_next) is that set, at any size, in O(d)."""
    d = acc.size
    idx, val = canonical(idx, val)
    assert idx.size == k
    if k:
        assert idx[0] >= 0 and idx[-1] < d
        assert np.all(np.diff(idx) > 0), "duplicate indices"
    ab = bits(acc)
    np.testing.assert_array_equal(bits(val), ab[idx], err_msg="payload values")
    kept = np.zeros(d, dtype=bool)
    kept[idx] = True
    eb = bits(e_next)
    assert np.all(eb[kept] == 0), "e' not +0 at kept coordinates"
    np.testing.assert_array_equal(eb[~kept], ab[~kept], err_msg="e' at dropped coordinates")
    if 0 < k < d:
        key = ab & np.uint32(0x7FFFFFFF)
        T = key[idx].min()
        above = key > T
        assert np.all(kept[above]), "a larger magnitude was dropped"
        assert not np.any(kept[key < T]), "a smaller magnitude was kept"
        tied = np.nonzero(key == T)[0]
        m = k - int(np.count_nonzero(above))
        np.testing.assert_array_equal(np.nonzero(kept & (key == T))[0], tied[:m],
                                      err_msg="ties not resolved to the lower index")


def check_topk_chunked(d, k, idx, val, acc_fn, e_next_fn, chunk=1 << 26, log=None):
    """check_topk_properties for vectors too large to hold several copies of:
    acc_fn(lo, hi) and e_next_fn(lo, hi) return float32 slices [lo, hi)."""
    idx, val = canonical(idx, val)
    assert idx.size == k
    if k == 0:
        return
    assert idx[0] >= 0 and idx[-1] < d and np.all(np.diff(idx) > 0)
    key_kept = bits(val) & np.uint32(0x7FFFFFFF)
    T = key_kept.min()
    above = 0
    tie_flags = []
    for lo in range(0, d, chunk):
        hi = min(d, lo + chunk)
        acc = acc_fn(lo, hi)
        en = e_next_fn(lo, hi)
        a, b = np.searchsorted(idx, [lo, hi])
        ki = idx[a:b] - lo
        kept = np.zeros(hi - lo, dtype=bool)
        kept[ki] = True
        ab = bits(acc)
        np.testing.assert_array_equal(bits(val[a:b]), ab[ki], err_msg="values at %d" % lo)
        eb = bits(en)
        assert np.all(eb[kept] == 0), "e' not +0 at kept coordinates near %d" % lo
        np.testing.assert_array_equal(eb[~kept], ab[~kept], err_msg="e' near %d" % lo)
        key = ab & np.uint32(0x7FFFFFFF)
        gt = key > T
        assert np.all(kept[gt]), "a larger magnitude was dropped near %d" % lo
        assert not np.any(kept[key < T]), "a smaller magnitude was kept near %d" % lo
        above += int(np.count_nonzero(gt))
        tie_flags.append(kept[key == T])
        if log is not None:
            log("  checked [%d, %d)" % (lo, hi))
    flags = np.concatenate(tie_flags)
    m = k - above
    assert 1 <= m <= flags.size
    assert np.all(flags[:m]) and not np.any(flags[m:]), "ties not resolved to the lower index"
