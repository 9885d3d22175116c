"""CPU oracle for the error-feedback sparsification step (TEST INFRASTRUCTURE).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  It is a thin ctypes wrapper over ``oracle.c`` (plain,
scalar C: the definitions of Algorithm 1's accumulate / compress / error
update with the hard-threshold and Top-k sparsifiers, and the
exchange-and-average step).  It shares no code with the HIP library.

All functions take and return numpy arrays on the host.  With ``mt=True``
they run the multi-core variant (``oracle_mt.c``, OpenMP over contiguous
index chunks), which returns the same bits as the single-threaded
definitions.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_LIB_MT_PATH = os.path.join(_HERE, "liboracle_mt.so")
_lib = None
_lib_mt = None

_f32p = ctypes.POINTER(ctypes.c_float)
_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)


def _declare(lib):
    lib.orc_ht.argtypes = [_f32p, _f32p, ctypes.c_int64, ctypes.c_float, ctypes.c_float,
                           _i32p, _f32p, ctypes.c_int64, _i64p]
    lib.orc_ht.restype = None
    lib.orc_topk.argtypes = [_f32p, _f32p, ctypes.c_int64, ctypes.c_float, ctypes.c_int64,
                             _i32p, _f32p]
    lib.orc_topk.restype = ctypes.c_int
    lib.orc_accumulate.argtypes = [ctypes.POINTER(_i32p), ctypes.POINTER(_f32p), _i64p,
                                   ctypes.c_int32, ctypes.c_int64, _f32p]
    lib.orc_accumulate.restype = ctypes.c_int
    lib.orc_update.argtypes = [ctypes.POINTER(_i32p), ctypes.POINTER(_f32p), _i64p,
                               ctypes.c_int32, ctypes.c_int64, ctypes.c_int, _f32p, _f32p,
                               ctypes.c_float, ctypes.c_float]
    lib.orc_update.restype = ctypes.c_int
    lib.orc_topk_segmented.argtypes = [_f32p, _f32p, ctypes.c_int64, ctypes.c_float,
                                       ctypes.c_int32, _i64p, _i64p, _i32p, _f32p]
    lib.orc_topk_segmented.restype = ctypes.c_int64
    return lib


def _load(mt=False):
    """The single-threaded library, or with mt the multi-core one."""
    global _lib, _lib_mt
    if (_lib_mt if mt else _lib) is not None:
        return _lib_mt if mt else _lib
    if not (os.path.exists(_LIB_PATH) and os.path.exists(_LIB_MT_PATH)):
        from . import build as _b
        _b.build()
    if not mt:
        _lib = _declare(ctypes.CDLL(_LIB_PATH))
        return _lib
    lib = _declare(ctypes.CDLL(_LIB_MT_PATH))
    lib.orc_ht_mt.argtypes = lib.orc_ht.argtypes
    lib.orc_ht_mt.restype = None
    lib.orc_topk_mt.argtypes = lib.orc_topk.argtypes
    lib.orc_topk_mt.restype = ctypes.c_int
    lib.orc_topk_segmented_mt.argtypes = lib.orc_topk_segmented.argtypes
    lib.orc_topk_segmented_mt.restype = ctypes.c_int64
    lib.orc_accumulate_mt.argtypes = lib.orc_accumulate.argtypes
    lib.orc_accumulate_mt.restype = ctypes.c_int
    lib.orc_mt_threads.argtypes = []
    lib.orc_mt_threads.restype = ctypes.c_int
    _lib_mt = lib
    return lib


def mt_threads():
    """Threads the multi-core variant uses (OpenMP's maximum)."""
    return int(_load(mt=True).orc_mt_threads())


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _ptr(a, t):
    return a.ctypes.data_as(t)


def ht(g, e, lr, lam, cap=None, mt=False):
    """Hard-threshold EF step (Algorithm 1 with C_lambda, section 4.2).

    Returns (idx int32[k], val float32[k], e_next float32[d], k) with the
    payload in ascending index order.  ``e`` is not modified.
    """
    lib = _load(mt)
    fn = lib.orc_ht_mt if mt else lib.orc_ht
    g = _f32(g)
    e_next = np.array(e, dtype=np.float32, copy=True)
    d = g.size
    assert e_next.size == d
    if cap is None:
        cap = d
    idx = np.empty(max(cap, 1), dtype=np.int32)
    val = np.empty(max(cap, 1), dtype=np.float32)
    count = ctypes.c_int64(0)
    fn(_ptr(g, _f32p), _ptr(e_next, _f32p), d, ctypes.c_float(lr), ctypes.c_float(lam),
       _ptr(idx, _i32p), _ptr(val, _f32p), cap, ctypes.byref(count))
    k = count.value
    n = min(k, cap)
    return idx[:n].copy(), val[:n].copy(), e_next, k


def topk(g, e, lr, k, mt=False):
    """Top-k EF step (Algorithm 1 with Top-k; Lemma 2).

    Returns (idx int32[min(k,d)], val float32[...], e_next float32[d]) with
    the payload in ascending index order.  ``e`` is not modified.
    """
    lib = _load(mt)
    fn = lib.orc_topk_mt if mt else lib.orc_topk
    g = _f32(g)
    e_next = np.array(e, dtype=np.float32, copy=True)
    d = g.size
    assert e_next.size == d
    kk = max(0, min(int(k), d))
    idx = np.empty(max(kk, 1), dtype=np.int32)
    val = np.empty(max(kk, 1), dtype=np.float32)
    rc = fn(_ptr(g, _f32p), _ptr(e_next, _f32p), d, ctypes.c_float(lr), kk,
            _ptr(idx, _i32p), _ptr(val, _f32p))
    if rc != 0:
        raise MemoryError("oracle top-k scratch allocation failed")
    return idx[:kk].copy(), val[:kk].copy(), e_next


def accumulate(payloads, d, mt=False):
    """Exchange-and-average step: (sum_w decompress(payload_w)) / n.

    ``payloads`` is a sequence of (idx, val) pairs, summed in that order.
    """
    lib = _load(mt)
    fn = lib.orc_accumulate_mt if mt else lib.orc_accumulate
    n = len(payloads)
    idxs = [np.ascontiguousarray(p[0], dtype=np.int32) for p in payloads]
    vals = [_f32(p[1]) for p in payloads]
    for i, v in zip(idxs, vals):
        assert i.size == v.size
    idx_arr = (_i32p * max(n, 1))(*[_ptr(i, _i32p) for i in idxs])
    val_arr = (_f32p * max(n, 1))(*[_ptr(v, _f32p) for v in vals])
    counts = np.array([i.size for i in idxs] or [0], dtype=np.int64)
    out = np.empty(d, dtype=np.float32)
    rc = fn(idx_arr, val_arr, _ptr(counts, _i64p), n, d, _ptr(out, _f32p))
    if rc != 0:
        raise ValueError("payload index outside [0, d)")
    return out


def update(payloads, x, mode, m=None, beta=0.0, gamma=0.0):
    """Model update after averaging the payloads: mode 1 x - avg (Algorithm 1),
    mode 2 the momentum form of Algorithm 2.  Returns (x_new, m_new); the
    inputs are not modified."""
    lib = _load()
    n = len(payloads)
    idxs = [np.ascontiguousarray(p[0], dtype=np.int32) for p in payloads]
    vals = [_f32(p[1]) for p in payloads]
    idx_arr = (_i32p * max(n, 1))(*[_ptr(i, _i32p) for i in idxs])
    val_arr = (_f32p * max(n, 1))(*[_ptr(v, _f32p) for v in vals])
    counts = np.array([i.size for i in idxs] or [0], dtype=np.int64)
    x_new = np.array(x, dtype=np.float32, copy=True)
    d = x_new.size
    m_new = (np.zeros(d, dtype=np.float32) if m is None
             else np.array(m, dtype=np.float32, copy=True))
    rc = lib.orc_update(idx_arr, val_arr, _ptr(counts, _i64p), n, d, int(mode),
                        _ptr(x_new, _f32p), _ptr(m_new, _f32p), ctypes.c_float(beta),
                        ctypes.c_float(gamma))
    if rc != 0:
        raise ValueError("bad payload index or mode")
    return x_new, m_new


def topk_segmented(g, e, lr, offsets, ks, mt=False):
    """Layer-wise Top-k (Appendix C.5): Top-k with k = ks[s] on each segment
    [offsets[s], offsets[s+1]).  Returns (idx, val, e_next): segment by
    segment, ascending index order within each, global indices."""
    lib = _load(mt)
    fn = lib.orc_topk_segmented_mt if mt else lib.orc_topk_segmented
    g = _f32(g)
    e_next = np.array(e, dtype=np.float32, copy=True)
    d = g.size
    off = np.ascontiguousarray(offsets, dtype=np.int64)
    k = np.ascontiguousarray(ks, dtype=np.int64)
    nseg = k.size
    assert off.size == nseg + 1
    total = int(np.minimum(np.maximum(k, 0), np.diff(off)).sum()) if nseg else 0
    idx = np.empty(max(total, 1), dtype=np.int32)
    val = np.empty(max(total, 1), dtype=np.float32)
    n = fn(_ptr(g, _f32p), _ptr(e_next, _f32p), d, ctypes.c_float(lr), nseg,
           _ptr(off, _i64p), _ptr(k, _i64p), _ptr(idx, _i32p), _ptr(val, _f32p))
    if n < 0:
        raise ValueError("bad segment layout")
    return idx[:n].copy(), val[:n].copy(), e_next


def calibrate_lambda(g0, density, lr=np.float32(0.1)):
    """Threshold giving the requested density at the first iteration.

    With e_0 = 0 the first compressed vector is a = fl(lr * g_0).  For
    K = round(density * d) (at least 1, at most d) the threshold is the K-th
    largest |a|, the upper end of the interval (A_(K+1), A_(K)] of Lemma 3,
    so the first iteration keeps exactly K coordinates when that magnitude
    is not tied (more when it is).  numpy's float32 product rounds like the
    fp32 multiply of the step.
    """
    a = np.abs(np.float32(lr) * np.asarray(g0, dtype=np.float32))
    d = a.size
    K = min(max(int(round(density * d)), 1), d)
    return np.float32(np.partition(a, d - K)[d - K])
