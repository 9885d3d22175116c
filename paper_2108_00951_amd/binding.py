"""ctypes binding of libefsparse.so (argument marshalling only).

Every function takes torch tensors that live on a ROCm device, passes their
raw pointers and the current HIP stream to the C ABI declared in
include/efsparse.h, and raises EfsError on a non-OK status.  No arithmetic
of the method happens here; when the shared library is missing the import
of a function fails loudly instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libefsparse.so")

EFS_OK, EFS_EINVAL, EFS_ESPACE, EFS_EHIP = 0, 1, 2, 3
COUNTER_WORDS = 4
MAX_WORKERS = 64

_lib = None


class EfsError(RuntimeError):
    """A non-OK status from libefsparse."""

    def __init__(self, status: int, message: str):
        super().__init__("efsparse status %d: %s" % (status, message))
        self.status = status


def load_library(path: str = LIB_PATH):
    """Load libefsparse.so once and declare the C signatures.

    torch is imported first so that the library binds to the HIP runtime
    torch already loaded (one runtime per process, shared streams).
    """
    global _lib
    if _lib is not None:
        return _lib
    import torch  # noqa: F401  (binds the HIP runtime before the library loads)
    if not os.path.exists(path):
        raise ImportError("libefsparse.so not built at %s; run python -m paper_2108_00951_amd.build"
                          % path)
    lib = ctypes.CDLL(path)
    declare(lib)
    _lib = lib
    return lib


def declare(lib):
    """Attach argtypes/restype of every exported function to a CDLL."""
    vp, i64, f32, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_float, ctypes.c_int32
    lib.ht_compress.argtypes = [vp, vp, i64, f32, f32, vp, vp, i64, vp, vp]
    lib.ht_compress.restype = ctypes.c_int
    lib.ht_compress_telemetry.argtypes = [vp, vp, i64, f32, f32, vp, vp, i64, vp, vp, vp]
    lib.ht_compress_telemetry.restype = ctypes.c_int
    lib.topk_workspace_bytes.argtypes = [i64, i64]
    lib.topk_workspace_bytes.restype = ctypes.c_size_t
    lib.topk_path_flag_offset.argtypes = []
    lib.topk_path_flag_offset.restype = ctypes.c_size_t
    lib.topk_compress.argtypes = [vp, vp, i64, f32, i64, vp, vp, vp, ctypes.c_size_t, vp]
    lib.topk_compress.restype = ctypes.c_int
    lib.sparse_accumulate.argtypes = [ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp),
                                      ctypes.POINTER(i64), i32, i64, vp, vp, ctypes.c_size_t, vp]
    lib.sparse_accumulate.restype = ctypes.c_int
    lib.sparse_accumulate_workspace_bytes.argtypes = [i32, i64, i64]
    lib.sparse_accumulate_workspace_bytes.restype = ctypes.c_size_t
    lib.sparse_bucket_workspace_bytes.argtypes = [i32, i64]
    lib.sparse_bucket_workspace_bytes.restype = ctypes.c_size_t
    lib.sparse_status_offset.argtypes = []
    lib.sparse_status_offset.restype = ctypes.c_size_t
    lib.topk_segmented_workspace_bytes.argtypes = [i32, i64]
    lib.topk_segmented_workspace_bytes.restype = ctypes.c_size_t
    lib.topk_segmented_status_offset.argtypes = []
    lib.topk_segmented_status_offset.restype = ctypes.c_size_t
    lib.topk_segmented_bracket_offset.argtypes = []
    lib.topk_segmented_bracket_offset.restype = ctypes.c_size_t
    lib.topk_segmented_compress.argtypes = [vp, vp, i64, f32, i32, vp, vp, i64, vp, vp, vp,
                                            ctypes.c_size_t, vp]
    lib.topk_segmented_compress.restype = ctypes.c_int
    lib.sparse_accumulate_static.argtypes = [ctypes.POINTER(vp), ctypes.POINTER(vp),
                                             ctypes.POINTER(vp), ctypes.POINTER(i64), i32, i64,
                                             vp, vp]
    lib.sparse_accumulate_static.restype = ctypes.c_int
    lib.sparse_apply_workspace_bytes.argtypes = [i32, i64, i64]
    lib.sparse_apply_workspace_bytes.restype = ctypes.c_size_t
    lib.sparse_apply.argtypes = [ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp),
                                 ctypes.POINTER(i64), i32, i64, ctypes.c_int, vp, vp, f32, f32, vp,
                                 ctypes.c_size_t, vp]
    lib.sparse_apply.restype = ctypes.c_int
    lib.efs_copy_probe.argtypes = [vp, vp, i64, vp]
    lib.efs_copy_probe.restype = ctypes.c_int
    lib.efs_stream_probe.argtypes = [vp, vp, i64, ctypes.c_int, vp]
    lib.efs_stream_probe.restype = ctypes.c_int
    lib.efs_status_string.argtypes = [ctypes.c_int]
    lib.efs_status_string.restype = ctypes.c_char_p
    lib.efs_last_error_message.argtypes = []
    lib.efs_last_error_message.restype = ctypes.c_char_p
    lib.efs_last_error.argtypes = []
    lib.efs_last_error.restype = ctypes.c_int
    return lib


def _check(lib, rc: int):
    if rc != EFS_OK:
        raise EfsError(rc, lib.efs_last_error_message().decode())


def _stream_handle(stream) -> int:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(getattr(stream, "cuda_stream", stream))


def _ptr(t) -> Optional[int]:
    return t.data_ptr() if t is not None and t.numel() > 0 else None


def _require(t, dtype, name):
    import torch
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if t.device.type != "cuda":
        raise TypeError("%s must be a device tensor" % name)
    if not t.is_contiguous():
        raise TypeError("%s must be contiguous" % name)
    return torch


def new_counter(device="cuda"):
    """A zero-filled counter object (EFS_COUNTER_WORDS int32 words)."""
    import torch
    return torch.zeros(COUNTER_WORDS, dtype=torch.int32, device=device)


def counter_value(counter) -> int:
    """k_t from a counter object (synchronises with the device)."""
    return int(counter[0].item()) & 0xFFFFFFFF


def ht_compress(g, e, lr: float, lam: float, idx, val, counter, stream=None) -> None:
    """Hard-threshold EF step; see ht_compress in include/efsparse.h."""
    import torch
    lib = load_library()
    _require(g, torch.float32, "g")
    _require(e, torch.float32, "e")
    _require(idx, torch.int32, "idx")
    _require(val, torch.float32, "val")
    _require(counter, torch.int32, "counter")
    if g.numel() != e.numel() or idx.numel() != val.numel() or counter.numel() < COUNTER_WORDS:
        raise ValueError("size mismatch among g, e, idx, val, counter")
    rc = lib.ht_compress(_ptr(g), _ptr(e), g.numel(), float(lr), float(lam), _ptr(idx), _ptr(val),
                         idx.numel(), counter.data_ptr(), _stream_handle(stream))
    _check(lib, rc)


TELEMETRY_BYTES = 288


def new_telemetry(device="cuda"):
    """A zero-filled telemetry object (see EFS_TELEMETRY_BYTES)."""
    import torch
    return torch.zeros(TELEMETRY_BYTES, dtype=torch.uint8, device=device)


def read_telemetry(tel) -> dict:
    """Decode a telemetry object (synchronises with the device)."""
    import numpy as np
    raw = tel.cpu().numpy().tobytes()
    parts = np.frombuffer(raw[:256], dtype="<f8")
    err2 = 0.0
    for x in parts:  # the total error is the sum of the 32 parts
        err2 += float(x)
    (sent,) = np.frombuffer(raw[256:264], dtype="<f8")
    max_bits, calls = np.frombuffer(raw[264:272], dtype="<u4")
    return {"err2_total": float(err2), "sent_total": float(sent),
            "max_abs": float(np.array([max_bits], dtype=np.uint32).view(np.float32)[0]),
            "max_abs_bits": int(max_bits), "calls": int(calls)}


def ht_compress_telemetry(g, e, lr: float, lam: float, idx, val, counter, telemetry,
                          stream=None) -> None:
    """ht_compress plus telemetry; see ht_compress_telemetry in include/efsparse.h."""
    import torch
    lib = load_library()
    _require(g, torch.float32, "g")
    _require(e, torch.float32, "e")
    _require(idx, torch.int32, "idx")
    _require(val, torch.float32, "val")
    _require(counter, torch.int32, "counter")
    _require(telemetry, torch.uint8, "telemetry")
    if g.numel() != e.numel() or idx.numel() != val.numel() or counter.numel() < COUNTER_WORDS \
            or telemetry.numel() < TELEMETRY_BYTES:
        raise ValueError("size mismatch among g, e, idx, val, counter, telemetry")
    rc = lib.ht_compress_telemetry(_ptr(g), _ptr(e), g.numel(), float(lr), float(lam), _ptr(idx),
                                   _ptr(val), idx.numel(), counter.data_ptr(), telemetry.data_ptr(),
                                   _stream_handle(stream))
    _check(lib, rc)


def topk_workspace_bytes(d: int, k: int) -> int:
    return int(load_library().topk_workspace_bytes(int(d), int(k)))


def new_topk_workspace(d: int, k: int, device="cuda"):
    import torch
    return torch.empty(max(topk_workspace_bytes(d, k), 1), dtype=torch.uint8, device=device)


def topk_took_bracket_path(workspace) -> bool:
    """True if the last completed topk_compress on this workspace selected
    from the candidate set around the previous threshold (synchronises)."""
    off = int(load_library().topk_path_flag_offset())
    return bool(int(workspace[off:off + 4].cpu().numpy().view("<u4")[0]))


def topk_compress(g, e, lr: float, k: int, idx, val, workspace, stream=None) -> None:
    """Top-k EF step; see topk_compress in include/efsparse.h."""
    import torch
    lib = load_library()
    _require(g, torch.float32, "g")
    _require(e, torch.float32, "e")
    _require(idx, torch.int32, "idx")
    _require(val, torch.float32, "val")
    _require(workspace, torch.uint8, "workspace")
    if g.numel() != e.numel() or idx.numel() < k or val.numel() < k:
        raise ValueError("size mismatch among g, e, idx, val and k")
    rc = lib.topk_compress(_ptr(g), _ptr(e), g.numel(), float(lr), int(k), _ptr(idx), _ptr(val),
                           _ptr(workspace), workspace.numel(), _stream_handle(stream))
    _check(lib, rc)


def topk_segmented_workspace_bytes(nseg: int, k_total: int) -> int:
    return int(load_library().topk_segmented_workspace_bytes(int(nseg), int(k_total)))


def new_topk_segmented_workspace(nseg: int, k_total: int, device="cuda"):
    import torch
    return torch.empty(max(topk_segmented_workspace_bytes(nseg, k_total), 16), dtype=torch.uint8,
                       device=device)


def topk_segmented_status(workspace) -> int:
    """0 if the last completed topk_segmented_compress on this workspace
    accepted the layout, 1 if it rejected it (synchronises)."""
    off = int(load_library().topk_segmented_status_offset())
    return int(workspace[off:off + 4].cpu().numpy().view("<u4")[0])


def topk_segmented_bracket_segments(workspace) -> int:
    """Segments of the last completed topk_segmented_compress on this
    workspace that selected from the bracket around the previous threshold
    (synchronises)."""
    off = int(load_library().topk_segmented_bracket_offset())
    return int(workspace[off:off + 4].cpu().numpy().view("<u4")[0])


def topk_segmented_compress(g, e, lr: float, offsets, k, idx, val, workspace, stream=None) -> None:
    """Layer-wise Top-k EF step; see topk_segmented_compress in include/efsparse.h.
    offsets: int64 device tensor [nseg + 1]; k: int64 device tensor [nseg];
    the payload capacity k_total is idx.numel()."""
    import torch
    lib = load_library()
    _require(g, torch.float32, "g")
    _require(e, torch.float32, "e")
    _require(offsets, torch.int64, "offsets")
    _require(k, torch.int64, "k")
    _require(idx, torch.int32, "idx")
    _require(val, torch.float32, "val")
    _require(workspace, torch.uint8, "workspace")
    if g.numel() != e.numel() or idx.numel() != val.numel() or offsets.numel() != k.numel() + 1:
        raise ValueError("size mismatch among g, e, idx, val, offsets and k")
    rc = lib.topk_segmented_compress(_ptr(g), _ptr(e), g.numel(), float(lr), k.numel(),
                                     offsets.data_ptr(), k.data_ptr(), idx.numel(), _ptr(idx),
                                     _ptr(val), _ptr(workspace), workspace.numel(),
                                     _stream_handle(stream))
    _check(lib, rc)


def _payload_arrays(payloads: Sequence[Tuple]):
    """Host arrays of device pointers and capacities for n payloads, each
    (idx, val, counter_or_None); without a counter the whole idx/val tensor
    is the payload."""
    import torch
    n = len(payloads)
    vp = ctypes.c_void_p
    idx_arr = (vp * max(n, 1))()
    val_arr = (vp * max(n, 1))()
    cnt_arr = (vp * max(n, 1))()
    caps = (ctypes.c_int64 * max(n, 1))()
    for w, p in enumerate(payloads):
        idx, val = p[0], p[1]
        cnt = p[2] if len(p) > 2 else None
        _require(idx, torch.int32, "idx[%d]" % w)
        _require(val, torch.float32, "val[%d]" % w)
        if idx.numel() != val.numel():
            raise ValueError("payload %d: idx and val differ in length" % w)
        if cnt is not None:
            _require(cnt, torch.int32, "counter[%d]" % w)
        idx_arr[w] = _ptr(idx)
        val_arr[w] = _ptr(val)
        cnt_arr[w] = cnt.data_ptr() if cnt is not None else None
        caps[w] = idx.numel()
    return idx_arr, val_arr, cnt_arr, caps


def sparse_accumulate(payloads: Sequence[Tuple], d: int, out, workspace, stream=None) -> None:
    """Average of n payloads into out; see sparse_accumulate in include/efsparse.h.

    payloads: sequence of (idx, val, counter_or_None); workspace from
    new_apply_workspace (the average and the fused update share its layout).
    """
    prepare_sparse_accumulate(payloads, d, out, workspace, stream)()


SPARSE_TRUNCATED, SPARSE_BAD_INDEX = 1, 2


def sparse_status(workspace) -> int:
    """EFS_SPARSE_* bits of the last completed sparse_accumulate / sparse_apply
    on this workspace (synchronises)."""
    off = int(load_library().sparse_status_offset())
    return int(workspace[off:off + 4].cpu().numpy().view("<u4")[0])


APPLY_AVERAGE, APPLY_SGD, APPLY_MOMENTUM = 0, 1, 2


def sparse_apply_workspace_bytes(n_workers: int, d: int, total_cap: int) -> int:
    return int(load_library().sparse_apply_workspace_bytes(int(n_workers), int(d), int(total_cap)))


def sparse_bucket_workspace_bytes(n_workers: int, d: int) -> int:
    return int(load_library().sparse_bucket_workspace_bytes(int(n_workers), int(d)))


LAYOUTS = ("bucketed", "packed")


def new_apply_workspace(payloads: Sequence[Tuple], d: int, device="cuda", layout="bucketed"):
    """A workspace for sparse_accumulate or sparse_apply over payloads of
    these capacities, in the given layout: "bucketed" (two launches, about
    8 n d bytes) or "packed" (four launches, about 8 bytes per payload
    slot).  A call takes the bucketed layout whenever the workspace holds
    it, so a packed workspace at least that large is used as bucketed."""
    import torch
    if layout not in LAYOUTS:
        raise ValueError("layout must be one of %s" % (LAYOUTS,))
    if layout == "bucketed":
        nbytes = sparse_bucket_workspace_bytes(len(payloads), d)
    else:
        total = sum(int(p[0].numel()) for p in payloads)
        nbytes = sparse_apply_workspace_bytes(len(payloads), d, total)
    return torch.empty(max(nbytes, 16), dtype=torch.uint8, device=device)


def prepare_sparse_apply(payloads: Sequence[Tuple], d: int, mode: int, x, workspace, m=None,
                         beta: float = 0.0, gamma: float = 0.0, stream=None):
    """Marshal the arguments of sparse_apply once and return a callable that
    issues the call with them (for loops that repeat the same call on the
    same buffers: the per-call cost is then one C call).  The stream is fixed
    here too: `stream`, else the current stream at this call."""
    import torch
    lib = load_library()
    _require(x, torch.float32, "x")
    _require(workspace, torch.uint8, "workspace")
    if x.numel() != d:
        raise ValueError("x must have d elements")
    if m is not None:
        _require(m, torch.float32, "m")
        if m.numel() != d:
            raise ValueError("m must have d elements")
    idx_arr, val_arr, cnt_arr, caps = _payload_arrays(payloads)
    args = (idx_arr, val_arr, cnt_arr, caps, len(payloads), int(d), int(mode), _ptr(x), _ptr(m),
            float(beta), float(gamma), _ptr(workspace), workspace.numel(), _stream_handle(stream))
    fn = lib.sparse_apply

    def call():
        _check(lib, fn(*args))
    return call


def sparse_apply(payloads: Sequence[Tuple], d: int, mode: int, x, workspace, m=None,
                 beta: float = 0.0, gamma: float = 0.0, stream=None) -> None:
    """Average of n payloads fused with the model update; see sparse_apply in
    include/efsparse.h.  payloads as for sparse_accumulate."""
    prepare_sparse_apply(payloads, d, mode, x, workspace, m, beta, gamma, stream)()


def prepare_sparse_accumulate(payloads: Sequence[Tuple], d: int, out, workspace, stream=None):
    """sparse_accumulate with its arguments marshalled once (see
    prepare_sparse_apply)."""
    import torch
    lib = load_library()
    _require(out, torch.float32, "out")
    _require(workspace, torch.uint8, "workspace")
    if out.numel() != d:
        raise ValueError("out must have d elements")
    idx_arr, val_arr, cnt_arr, caps = _payload_arrays(payloads)
    args = (idx_arr, val_arr, cnt_arr, caps, len(payloads), int(d), _ptr(out), _ptr(workspace),
            workspace.numel(), _stream_handle(stream))
    fn = lib.sparse_accumulate

    def call():
        _check(lib, fn(*args))
    return call


STATIC_SCRATCH_BYTES = 64 << 20


def sparse_accumulate_static(payloads: Sequence[Tuple], d: int, out, stream=None) -> None:
    """sparse_accumulate with the library's per-device scratch in place of a
    workspace (no allocation by the call); see sparse_accumulate_static in
    include/efsparse.h."""
    import torch
    lib = load_library()
    _require(out, torch.float32, "out")
    if out.numel() != d:
        raise ValueError("out must have d elements")
    idx_arr, val_arr, cnt_arr, caps = _payload_arrays(payloads)
    _check(lib, lib.sparse_accumulate_static(idx_arr, val_arr, cnt_arr, caps, len(payloads), int(d),
                                             _ptr(out), _stream_handle(stream)))


def copy_probe(src, dst, stream=None) -> None:
    """Streaming copy used as the bandwidth ceiling in measurements."""
    import torch
    lib = load_library()
    _require(src, torch.float32, "src")
    _require(dst, torch.float32, "dst")
    if src.numel() != dst.numel():
        raise ValueError("src and dst differ in length")
    _check(lib, lib.efs_copy_probe(_ptr(src), _ptr(dst), src.numel(), _stream_handle(stream)))


def stream_probe(x, y, mode: int, stream=None) -> None:
    """Bandwidth probe: 0 copy, 1 read, 2 write, 3 two reads + one write;
    plus 4, one workgroup per 4096-element tile instead of the persistent grid."""
    import torch
    lib = load_library()
    _require(x, torch.float32, "x")
    _require(y, torch.float32, "y")
    if int(mode) & 3 != 1 and x.numel() != y.numel():
        raise ValueError("x and y differ in length")
    _check(lib, lib.efs_stream_probe(_ptr(x), _ptr(y), x.numel(), int(mode), _stream_handle(stream)))
