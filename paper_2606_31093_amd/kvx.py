"""Python binding of libkvx (include/kvx.h): argument marshalling only.

Every step of the copy runs in the library's HIP kernels.  PyTorch supplies
device memory and the stream: tensors are passed as raw pointers and the
kernels run on ``torch.cuda.current_stream()`` unless a stream is given.
The functions keep the C names: ``kvx_transfer``, ``kvx_transfer_slice``,
``kvx_transfer_layered``, ``kvx_transfer_planned``,
``kvx_transfer_layered_planned``, ``kvx_gather``, ``kvx_scatter``,
``kvx_gather_slice``, ``kvx_scatter_slice`` and ``kvx_page_hashes``.  A
missing or unloadable library raises; there is no fallback path.

Pool and buffer shapes are duck-typed: a pool shape has integer attributes
``L C H D T N e`` and a ``layout`` name; a buffer shape has ``L C H D e``
and ``cap`` (elements).  ``paper_2606_31093_amd.workloads.PoolSpec`` and
``BufSpec`` fit.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build_lib

LAYOUTS = {"LPCTHD": 0, "LPCHTD": 1, "PLCTHD": 2, "PLCHTD": 3}

DERR_SRC_PAGE = 1
DERR_DST_PAGE = 2
DERR_PT_RANGE = 4
DERR_BAD_REQ = 8
DERR_STALLED = 16
DERR_BAD_PLAN = 32

STATUS = {0: "KVX_OK", -1: "KVX_ERR_NULL", -2: "KVX_ERR_SHAPE", -3: "KVX_ERR_ALIGN",
          -4: "KVX_ERR_LAYOUT", -5: "KVX_ERR_RANGE", -6: "KVX_ERR_HIP"}

REQ_DTYPE = np.dtype([("src_pt_off", "<i8"), ("dst_pt_off", "<i8"), ("buf_off", "<i8"),
                      ("src_start", "<i4"), ("dst_start", "<i4"), ("n_tokens", "<i4"),
                      ("reserved", "<i4")])


HASH_REQ_DTYPE = np.dtype([("payload_off", "<i8"), ("out_off", "<i8"), ("seed", "<u8"),
                           ("n_positions", "<i4"), ("reserved", "<i4")])


class Pool(ctypes.Structure):
    _fields_ = [("base", ctypes.c_void_p), ("num_layers", ctypes.c_int32),
                ("num_kv", ctypes.c_int32), ("num_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("page_tokens", ctypes.c_int32),
                ("num_pages", ctypes.c_int32), ("elem_bytes", ctypes.c_int32),
                ("layout", ctypes.c_int32)]


class Buf(ctypes.Structure):
    _fields_ = [("base", ctypes.c_void_p), ("num_layers", ctypes.c_int32),
                ("num_kv", ctypes.c_int32), ("num_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("elem_bytes", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("capacity_elems", ctypes.c_int64)]


class Slice(ctypes.Structure):
    _fields_ = [(k, ctypes.c_int32) for k in (
        "src_layer0", "dst_layer0", "num_layers", "src_kv0", "dst_kv0", "num_kv",
        "src_head0", "dst_head0", "num_heads", "reserved")]


def slice_desc(sl) -> Slice:
    """A kvx_slice from (src_layer0, dst_layer0, num_layers, src_kv0, dst_kv0,
    num_kv, src_head0, dst_head0, num_heads)."""
    if isinstance(sl, Slice):
        return sl
    vals = [int(x) for x in sl]
    if len(vals) != 9:
        raise ValueError("a slice has nine fields")
    return Slice(*vals, 0)


class KvxError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


_LIB = None


def library_path() -> str:
    return os.environ.get("KVX_LIBRARY", build_lib.LIBRARY)


def lib() -> ctypes.CDLL:
    """The loaded libkvx.so.  Raises if it is missing: build it with
    ``python -m paper_2606_31093_amd.build_lib`` (or ``__graft_entry__.build()``)."""
    global _LIB
    if _LIB is None:
        _LIB = load(library_path())
    return _LIB


def load(path: str) -> ctypes.CDLL:
    """Load a build of the library at ``path`` and declare its entry points'
    argument types (``lib()`` does this once for the default build)."""
    if not os.path.exists(path):
        raise RuntimeError(f"libkvx is not built ({path} missing); run "
                           "python -m paper_2606_31093_amd.build_lib")
    # PyTorch ships its own HIP runtime.  Loaded first, it is the one
    # libkvx binds to (same soname), so the library and torch share one
    # runtime: the one that owns the tensors and streams passed in.
    # Loading libkvx first would bring a second HIP and HSA runtime into
    # the process, and one of them then finds no device.
    import torch  # noqa: F401
    L = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    pp, bp = ctypes.POINTER(Pool), ctypes.POINTER(Buf)
    L.kvx_transfer.argtypes = [pp, pp, vp, i64, vp, i64, vp, i32, vp, vp]
    L.kvx_transfer_slice.argtypes = [pp, pp, ctypes.POINTER(Slice), vp, i64, vp, i64, vp, i32,
                                     vp, vp]
    L.kvx_transfer_layered.argtypes = [pp, pp, ctypes.POINTER(Slice), vp, i64, vp, i64, vp,
                                       i32, i32, ctypes.POINTER(vp), i32, vp, vp]
    L.kvx_gather.argtypes = [pp, bp, vp, i64, vp, i32, vp, vp]
    L.kvx_scatter.argtypes = [bp, pp, vp, i64, vp, i32, vp, vp]
    sp = ctypes.POINTER(Slice)
    L.kvx_gather_slice.argtypes = [pp, bp, sp, vp, i64, vp, i32, vp, vp]
    L.kvx_scatter_slice.argtypes = [bp, pp, sp, vp, i64, vp, i32, vp, vp]
    for f in (L.kvx_transfer, L.kvx_transfer_slice, L.kvx_transfer_layered, L.kvx_gather,
              L.kvx_scatter, L.kvx_gather_slice, L.kvx_scatter_slice):
        f.restype = ctypes.c_int
    L.kvx_transfer_planned.argtypes = [pp, pp, ctypes.POINTER(Slice), vp, i64, vp, i64, vp, i32,
                                       vp, i64, i64, vp, vp]
    L.kvx_transfer_planned.restype = ctypes.c_int
    L.kvx_transfer_layered_planned.argtypes = [pp, pp, ctypes.POINTER(Slice), vp, i64, vp, i64, vp,
                                               i32, i32, ctypes.POINTER(vp), i32, vp, i64, i64, vp, vp]
    L.kvx_transfer_layered_planned.restype = ctypes.c_int
    L.kvx_plan_pages.argtypes = [vp, i32, i32, i32, vp, vp]
    L.kvx_plan_pages.restype = ctypes.c_int64
    L.kvx_plan_fill.argtypes = [vp, i32, i32, i32, i64, vp]
    L.kvx_plan_fill.restype = ctypes.c_int
    L.kvx_page_hashes.argtypes = [vp, i64, i32, i32, vp, i32, vp, i64, vp, vp]
    L.kvx_page_hashes.restype = ctypes.c_int
    L.kvx_pool_bytes.argtypes = [pp]
    L.kvx_pool_bytes.restype = ctypes.c_int64
    L.kvx_strerror.argtypes = [ctypes.c_int]
    L.kvx_strerror.restype = ctypes.c_char_p
    L.kvx_last_error.argtypes = []
    L.kvx_last_error.restype = ctypes.c_char_p
    L.kvx_abi_version.argtypes = []
    L.kvx_abi_version.restype = ctypes.c_int
    L.kvx_set_launch_choice.argtypes = [ctypes.c_int]
    L.kvx_set_launch_choice.restype = ctypes.c_int
    L.kvx_launch_choice.argtypes = []
    L.kvx_launch_choice.restype = ctypes.c_int
    L.kvx_last_launch.argtypes = []
    L.kvx_last_launch.restype = ctypes.c_int
    return L


# ---------------------------------------------------------------------------
# descriptors
# ---------------------------------------------------------------------------

def _ptr(x) -> int | None:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def pool_desc(spec, data=None) -> Pool:
    """A kvx_pool for a pool shape; ``data`` is a tensor (or raw address)."""
    return Pool(_ptr(data), spec.L, spec.C, spec.H, spec.D, spec.T, spec.N, spec.e,
                LAYOUTS[spec.layout] if isinstance(spec.layout, str) else int(spec.layout))


def buf_desc(spec, data=None) -> Buf:
    return Buf(_ptr(data), spec.L, spec.C, spec.H, spec.D, spec.e, 0, spec.cap)


def pack_reqs(rows) -> np.ndarray:
    """(n, 6) int64 rows ``src_pt_off, dst_pt_off, buf_off, src_start,
    dst_start, n_tokens`` -> kvx_req records (numpy structured array)."""
    rows = np.asarray(rows, dtype=np.int64).reshape(-1, 6)
    out = np.zeros(len(rows), dtype=REQ_DTYPE)
    for i, name in enumerate(("src_pt_off", "dst_pt_off", "buf_off")):
        out[name] = rows[:, i]
    for i, name in ((3, "src_start"), (4, "dst_start"), (5, "n_tokens")):
        col = rows[:, i]
        if ((col < -2**31) | (col >= 2**31)).any():
            raise ValueError(f"{name} does not fit int32")
        out[name] = col
    return out


def _records(rows) -> np.ndarray:
    """kvx_req records: ``rows`` itself if it already is a record array,
    else pack_reqs(rows)."""
    if isinstance(rows, np.ndarray) and rows.dtype == REQ_DTYPE:
        return rows
    return pack_reqs(rows)


def device_reqs(rows, device="cuda"):
    """kvx_req records as a device tensor (bytes)."""
    import torch
    recs = pack_reqs(rows)
    t = torch.from_numpy(recs.view(np.uint8).copy())
    return t.to(device)


def device_table(pt, device="cuda"):
    import torch
    a = np.ascontiguousarray(np.asarray(pt if pt is not None else [], dtype=np.int32))
    return torch.from_numpy(a).to(device)


def pool_bytes(spec) -> int:
    return int(lib().kvx_pool_bytes(ctypes.byref(pool_desc(spec, 0))))


# ---------------------------------------------------------------------------
# entry points
# ---------------------------------------------------------------------------

def _stream(stream) -> int | None:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(status: int) -> None:
    if status != 0:
        raise KvxError(status, lib().kvx_last_error().decode())


def _n_reqs(reqs) -> int:
    nbytes = reqs.numel() * reqs.element_size()
    if nbytes % REQ_DTYPE.itemsize:
        raise ValueError("reqs must hold whole 40-byte kvx_req records")
    if not reqs.is_contiguous():
        raise ValueError("reqs must be contiguous")
    return nbytes // REQ_DTYPE.itemsize


def _len(t) -> int:
    return 0 if t is None else t.numel()


def _table(t, name: str):
    """A page table: a contiguous tensor of 32-bit entries (or None)."""
    if t is not None and not isinstance(t, int):
        if t.element_size() != 4 or t.is_floating_point() or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous int32 tensor (got {t.dtype})")
    return t


def _err_word(t):
    """The optional device error word: one 32-bit integer."""
    if t is not None and not isinstance(t, int):
        if t.element_size() != 4 or t.is_floating_point() or t.numel() < 1:
            raise ValueError(f"dev_err must be a 32-bit integer tensor (got {t.dtype})")
    return t


def _need(t, nbytes: int, name: str) -> None:
    """A tensor argument must hold at least the bytes its descriptor names."""
    if t is None or isinstance(t, int):
        return
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{name} holds {have} bytes, its descriptor needs {nbytes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _pool_nbytes(spec) -> int:
    return spec.L * spec.C * spec.H * spec.D * spec.T * spec.N * spec.e


def kvx_transfer(src, src_spec, dst, dst_spec, src_pt, dst_pt, reqs, dev_err=None,
                 stream=None) -> None:
    """Pool -> pool (see kvx_transfer in include/kvx.h).  ``src_pt`` /
    ``dst_pt`` are int32 device tensors, ``reqs`` a device tensor from
    ``device_reqs``, ``dev_err`` an optional int32/uint32 device word."""
    _need(src, _pool_nbytes(src_spec), "src")
    _need(dst, _pool_nbytes(dst_spec), "dst")
    S, D = pool_desc(src_spec, src), pool_desc(dst_spec, dst)
    _table(src_pt, "src_pt"), _table(dst_pt, "dst_pt"), _err_word(dev_err)
    _check(lib().kvx_transfer(ctypes.byref(S), ctypes.byref(D), _ptr(src_pt), _len(src_pt),
                              _ptr(dst_pt), _len(dst_pt), _ptr(reqs), _n_reqs(reqs),
                              _ptr(dev_err), _stream(stream)))


def kvx_transfer_slice(src, src_spec, dst, dst_spec, sl, src_pt, dst_pt, reqs, dev_err=None,
                       stream=None) -> None:
    """Slice of a pool -> slice of another pool (see kvx_transfer_slice in
    include/kvx.h).  ``sl`` is a ``Slice`` or the nine range fields."""
    _need(src, _pool_nbytes(src_spec), "src")
    _need(dst, _pool_nbytes(dst_spec), "dst")
    S, D, X = pool_desc(src_spec, src), pool_desc(dst_spec, dst), slice_desc(sl)
    _table(src_pt, "src_pt"), _table(dst_pt, "dst_pt"), _err_word(dev_err)
    _check(lib().kvx_transfer_slice(ctypes.byref(S), ctypes.byref(D), ctypes.byref(X),
                                    _ptr(src_pt), _len(src_pt), _ptr(dst_pt), _len(dst_pt),
                                    _ptr(reqs), _n_reqs(reqs), _ptr(dev_err), _stream(stream)))


def kvx_transfer_planned(src, src_spec, dst, dst_spec, src_pt, dst_pt, reqs, plan, plan_pages,
                         plan_tokens, sl=None, dev_err=None, stream=None, library=None) -> None:
    """Pool -> pool with a plan (see kvx_transfer_planned in
    include/kvx.h): ``plan`` a device tensor holding the plan, and
    ``plan_pages``, ``plan_tokens`` its totals, as ``device_plan`` returns.  ``sl`` is an optional
    slice (nine range fields or a ``Slice``); ``library`` a build loaded with
    ``load`` (default: ``lib()``)."""
    _need(src, _pool_nbytes(src_spec), "src")
    _need(dst, _pool_nbytes(dst_spec), "dst")
    S, D = pool_desc(src_spec, src), pool_desc(dst_spec, dst)
    X = ctypes.byref(slice_desc(sl)) if sl is not None else None
    _table(src_pt, "src_pt"), _table(dst_pt, "dst_pt"), _err_word(dev_err)
    n = _n_reqs(reqs)
    if plan is not None and not isinstance(plan, int):
        if not plan.is_contiguous() or plan.numel() * plan.element_size() < plan_bytes(n, plan_pages):
            raise ValueError("plan must be a contiguous tensor of KVX_PLAN_BYTES(n_reqs, plan_pages) "
                             "bytes")
    L = library or lib()
    status = L.kvx_transfer_planned(ctypes.byref(S), ctypes.byref(D), X, _ptr(src_pt), _len(src_pt),
                                    _ptr(dst_pt), _len(dst_pt), _ptr(reqs), n, _ptr(plan),
                                    int(plan_pages), int(plan_tokens), _ptr(dev_err),
                                    _stream(stream))
    if status != 0:
        raise KvxError(status, L.kvx_last_error().decode())


def plan_pages(rows, page_tokens: int, side: int = 1):
    """kvx_plan_pages on a host copy of the (n, 6) rows: the exclusive prefix
    of pages per record (numpy int64, n + 1 entries), the total of pages and
    the tokens of the well-formed records, for side 0 (source) or 1
    (destination) of a pool with ``page_tokens`` tokens per page.  ``rows``
    may also be a kvx_req record array."""
    recs = _records(rows)
    prefix = np.zeros(len(recs) + 1, np.int64)
    tokens = ctypes.c_int64(0)
    n = int(lib().kvx_plan_pages(recs.ctypes.data if len(recs) else None, len(recs), int(page_tokens),
                                 int(side), prefix.ctypes.data, ctypes.byref(tokens)))
    if n < 0:
        raise KvxError(-5, lib().kvx_last_error().decode())
    return prefix, n, tokens.value


def plan_bytes(n_reqs: int, plan_pages: int) -> int:
    """KVX_PLAN_BYTES: the prefix (n_reqs + 1 int64) and the 32-byte slots."""
    return (int(n_reqs) + 1) * 8 + int(plan_pages) * 32


def host_plan(rows, src_page_tokens: int, dst_page_tokens: int):
    """kvx_plan_fill for the (n, 6) rows (or a kvx_req record array): the
    plan as a host int64 array (the prefix, then four words per slot), its
    pages and its tokens."""
    recs = _records(rows)
    _, pages, tokens = plan_pages(recs, dst_page_tokens, 1)
    buf = np.zeros(plan_bytes(len(recs), pages) // 8, np.int64)
    st = lib().kvx_plan_fill(recs.ctypes.data if len(recs) else None, len(recs), int(src_page_tokens),
                             int(dst_page_tokens), pages, buf.ctypes.data)
    if st != 0:
        raise KvxError(st, lib().kvx_last_error().decode())
    return buf, pages, tokens


def plan_slots(buf, n_reqs: int):
    """The slots of a host plan as an (pages, 8) int32 array (a view):
    dst_idx, src_idx, dst_slot, n_tokens, src_slot, req and two reserved."""
    return buf[n_reqs + 1:].view(np.int32).reshape(-1, 8)


def device_plan(rows, src_page_tokens: int, dst_page_tokens: int, device="cuda"):
    """The plan of ``rows`` on the device: (tensor, pages, tokens), the
    arguments of kvx_transfer_planned after the records."""
    import torch
    buf, pages, tokens = host_plan(rows, src_page_tokens, dst_page_tokens)
    return torch.from_numpy(buf).to(device), pages, tokens


def _event_handles(events, st, stream):
    """hipEvent_t handles of ``events`` (torch.cuda.Event objects or raw
    handles) as a ctypes array, and their count."""
    import torch
    handles = []
    for ev in events:
        if isinstance(ev, int):
            handles.append(ev)
            continue
        if not ev.cuda_event:          # torch creates the HIP event on first record
            ev.record(torch.cuda.ExternalStream(st) if stream is not None else None)
        handles.append(ev.cuda_event)
    return (ctypes.c_void_p * max(1, len(handles)))(*handles), len(handles)


def kvx_transfer_layered(src, src_spec, dst, dst_spec, src_pt, dst_pt, reqs, layers_per_group,
                         events, sl=None, dev_err=None, stream=None) -> None:
    """Layer-pipelined pool -> pool (see kvx_transfer_layered in
    include/kvx.h).  ``events`` are ``torch.cuda.Event`` objects (or raw
    hipEvent_t handles), one per layer group; the library records events[g]
    on the stream once group g has been copied."""
    _need(src, _pool_nbytes(src_spec), "src")
    _need(dst, _pool_nbytes(dst_spec), "dst")
    _table(src_pt, "src_pt"), _table(dst_pt, "dst_pt"), _err_word(dev_err)
    st = _stream(stream)
    arr, n_ev = _event_handles(events, st, stream)
    S, D = pool_desc(src_spec, src), pool_desc(dst_spec, dst)
    X = None if sl is None else ctypes.byref(slice_desc(sl))
    _check(lib().kvx_transfer_layered(ctypes.byref(S), ctypes.byref(D), X, _ptr(src_pt),
                                      _len(src_pt), _ptr(dst_pt), _len(dst_pt), _ptr(reqs),
                                      _n_reqs(reqs), int(layers_per_group), arr, n_ev,
                                      _ptr(dev_err), st))


def kvx_transfer_layered_planned(src, src_spec, dst, dst_spec, src_pt, dst_pt, reqs, layers_per_group,
                                 events, plan, plan_pages, plan_tokens, sl=None, dev_err=None,
                                 stream=None, library=None) -> None:
    """kvx_transfer_layered with a plan (see kvx_transfer_layered_planned
    in include/kvx.h); the plan as ``device_plan`` returns it."""
    _need(src, _pool_nbytes(src_spec), "src")
    _need(dst, _pool_nbytes(dst_spec), "dst")
    _table(src_pt, "src_pt"), _table(dst_pt, "dst_pt"), _err_word(dev_err)
    n = _n_reqs(reqs)
    if plan is not None and not isinstance(plan, int):
        if not plan.is_contiguous() or plan.numel() * plan.element_size() < plan_bytes(n, plan_pages):
            raise ValueError("plan must be a contiguous tensor of KVX_PLAN_BYTES(n_reqs, plan_pages) "
                             "bytes")
    st = _stream(stream)
    arr, n_ev = _event_handles(events, st, stream)
    S, D = pool_desc(src_spec, src), pool_desc(dst_spec, dst)
    X = None if sl is None else ctypes.byref(slice_desc(sl))
    L = library or lib()
    status = L.kvx_transfer_layered_planned(ctypes.byref(S), ctypes.byref(D), X, _ptr(src_pt),
                                            _len(src_pt), _ptr(dst_pt), _len(dst_pt), _ptr(reqs), n,
                                            int(layers_per_group), arr, n_ev, _ptr(plan),
                                            int(plan_pages), int(plan_tokens), _ptr(dev_err), st)
    if status != 0:
        raise KvxError(status, L.kvx_last_error().decode())


def kvx_gather(src, src_spec, dst, buf_spec, src_pt, reqs, dev_err=None, stream=None) -> None:
    """Pool -> flat buffer (see kvx_gather in include/kvx.h)."""
    _need(src, _pool_nbytes(src_spec), "src")
    _need(dst, buf_spec.cap * buf_spec.e, "dst")
    S, B = pool_desc(src_spec, src), buf_desc(buf_spec, dst)
    _table(src_pt, "src_pt"), _err_word(dev_err)
    _check(lib().kvx_gather(ctypes.byref(S), ctypes.byref(B), _ptr(src_pt), _len(src_pt),
                            _ptr(reqs), _n_reqs(reqs), _ptr(dev_err), _stream(stream)))


def kvx_scatter(src, buf_spec, dst, dst_spec, dst_pt, reqs, dev_err=None, stream=None) -> None:
    """Flat buffer -> pool (see kvx_scatter in include/kvx.h)."""
    _need(src, buf_spec.cap * buf_spec.e, "src")
    _need(dst, _pool_nbytes(dst_spec), "dst")
    B, D = buf_desc(buf_spec, src), pool_desc(dst_spec, dst)
    _table(dst_pt, "dst_pt"), _err_word(dev_err)
    _check(lib().kvx_scatter(ctypes.byref(B), ctypes.byref(D), _ptr(dst_pt), _len(dst_pt),
                             _ptr(reqs), _n_reqs(reqs), _ptr(dev_err), _stream(stream)))


def kvx_gather_slice(src, src_spec, dst, buf_spec, sl, src_pt, reqs, dev_err=None,
                     stream=None) -> None:
    """Slice of a pool -> flat buffer holding exactly the slice (see
    kvx_gather_slice in include/kvx.h).  ``sl`` is a ``Slice`` or the nine
    range fields."""
    _need(src, _pool_nbytes(src_spec), "src")
    _need(dst, buf_spec.cap * buf_spec.e, "dst")
    S, B, X = pool_desc(src_spec, src), buf_desc(buf_spec, dst), slice_desc(sl)
    _table(src_pt, "src_pt"), _err_word(dev_err)
    _check(lib().kvx_gather_slice(ctypes.byref(S), ctypes.byref(B), ctypes.byref(X), _ptr(src_pt),
                                  _len(src_pt), _ptr(reqs), _n_reqs(reqs), _ptr(dev_err),
                                  _stream(stream)))


def kvx_scatter_slice(src, buf_spec, dst, dst_spec, sl, dst_pt, reqs, dev_err=None,
                      stream=None) -> None:
    """Flat buffer holding exactly a slice -> that slice of a pool (see
    kvx_scatter_slice in include/kvx.h)."""
    _need(src, buf_spec.cap * buf_spec.e, "src")
    _need(dst, _pool_nbytes(dst_spec), "dst")
    B, D, X = buf_desc(buf_spec, src), pool_desc(dst_spec, dst), slice_desc(sl)
    _table(dst_pt, "dst_pt"), _err_word(dev_err)
    _check(lib().kvx_scatter_slice(ctypes.byref(B), ctypes.byref(D), ctypes.byref(X), _ptr(dst_pt),
                                   _len(dst_pt), _ptr(reqs), _n_reqs(reqs), _ptr(dev_err),
                                   _stream(stream)))


def pack_hash_reqs(rows) -> np.ndarray:
    """(payload_off, out_off, seed, n_positions) rows -> kvx_hash_req records."""
    rows = list(rows)
    out = np.zeros(len(rows), dtype=HASH_REQ_DTYPE)
    for i, (po, oo, seed, n) in enumerate(rows):
        out[i] = (int(po), int(oo), int(seed) & 0xFFFFFFFFFFFFFFFF, int(n), 0)
    return out


def device_hash_reqs(rows, device="cuda"):
    import torch
    return torch.from_numpy(pack_hash_reqs(rows).view(np.uint8).copy()).to(device)


def kvx_page_hashes(payload, rec_bytes, page_tokens, reqs, out, dev_err, stream=None,
                    library=None) -> None:
    """Chained page hashes (see kvx_page_hashes in include/kvx.h).  ``payload``
    is a device tensor of records of ``rec_bytes`` bytes, ``reqs`` a device
    tensor from ``device_hash_reqs``, ``out`` a 64-bit device tensor (one
    word per page) and ``dev_err`` the device error word the call requires.
    ``library`` is a build loaded with ``load`` (default: ``lib()``)."""
    nbytes = payload.numel() * payload.element_size()
    if nbytes % rec_bytes:
        raise ValueError("payload is not a whole number of records")
    if out.element_size() != 8 or not out.is_contiguous() or not payload.is_contiguous():
        raise ValueError("out must be a contiguous 64-bit tensor; payload contiguous")
    _err_word(dev_err)
    rb = reqs.numel() * reqs.element_size()
    if rb % HASH_REQ_DTYPE.itemsize:
        raise ValueError("reqs must hold whole 32-byte kvx_hash_req records")
    if not reqs.is_contiguous():
        raise ValueError("reqs must be contiguous")
    L = library or lib()
    status = L.kvx_page_hashes(_ptr(payload), nbytes // rec_bytes, int(rec_bytes),
                               int(page_tokens), _ptr(reqs), rb // HASH_REQ_DTYPE.itemsize,
                               _ptr(out), out.numel(), _ptr(dev_err), _stream(stream))
    if status != 0:
        raise KvxError(status, L.kvx_last_error().decode())


def kvx_strerror(status: int) -> str:
    return lib().kvx_strerror(status).decode()


def kvx_last_error() -> str:
    return lib().kvx_last_error().decode()


def kvx_abi_version() -> int:
    return int(lib().kvx_abi_version())


# Launch choice of planned transfers and launch kinds (include/kvx.h).
CHOOSE_MEASURED, CHOOSE_SWEEP, CHOOSE_GRID = 0, 1, 2
LAUNCH_NONE, LAUNCH_GRID, LAUNCH_SWEEP = 0, 1, 2
LAUNCH_NAMES = {LAUNCH_NONE: "none", LAUNCH_GRID: "grid", LAUNCH_SWEEP: "sweep"}


def kvx_set_launch_choice(mode: int, library=None) -> None:
    """How planned transfers that can sweep pick their launch: CHOOSE_MEASURED,
    CHOOSE_SWEEP or CHOOSE_GRID (process-wide; forgets earlier measurements)."""
    L = library or lib()
    status = L.kvx_set_launch_choice(int(mode))
    if status != 0:
        raise KvxError(status, L.kvx_last_error().decode())


def kvx_launch_choice(library=None) -> int:
    return int((library or lib()).kvx_launch_choice())


def kvx_last_launch(library=None) -> int:
    """LAUNCH_NONE, LAUNCH_GRID or LAUNCH_SWEEP: the kind of the last kernel
    this thread's last copy call enqueued."""
    return int((library or lib()).kvx_last_launch())
