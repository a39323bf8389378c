"""CPU oracle for the paged KV-cache gather / scatter / transfer path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this module; the product path
(the HIP library and its binding) never does.

The arithmetic lives in ``kvx_oracle.c`` (plain C, one element at a time, in
the order request -> token -> layer -> kv -> head -> dim).  This module only
compiles it with gcc, loads it with ctypes and marshals numpy arrays.  What it
computes is stated in the C file's header: Omni-Flow Sec. 4.1.1 (layer x page
x slice addressing), Sec. 4.1.2 (conversion between the paged layout and the
flat serialization), Sec. 4.1.4 (partial pages keep their other slots) and
Sec. 5.2 (slot-to-page translation through a page table); slices of a pool
(layer, kv and head ranges, Sec. 4.1.1 views) copied pool to pool or through
a flat buffer; and the chained page hashes of Sec. 5.1 (FNV-1a 64 page
digests chained page by page).

Inputs are duck-typed: a pool shape is any object with integer attributes
``L C H D T N e`` and a ``layout`` name (``"LPCTHD"``, ``"LPCHTD"``,
``"PLCTHD"`` or ``"PLCHTD"``); a buffer shape has ``L C H D e`` and ``cap``
(elements).  Request records are an ``(n, 6)`` int64 array with columns
``src_pt_off, dst_pt_off, buf_off, src_start, dst_start, n_tokens``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(HERE, "kvx_oracle.c")
LIBRARY = os.path.join(HERE, "libkvx_oracle.so")

LAYOUT_CODES = {"LPCTHD": 0, "LPCHTD": 1, "PLCTHD": 2, "PLCHTD": 3}

ERR_SRC_PAGE = 1
ERR_DST_PAGE = 2
ERR_PT_RANGE = 4
ERR_BAD_REQ = 8


class _Pool(ctypes.Structure):
    _fields_ = [(k, ctypes.c_int64) for k in ("L", "C", "H", "D", "T", "N", "e", "layout")]


class _Buf(ctypes.Structure):
    _fields_ = [(k, ctypes.c_int64) for k in ("L", "C", "H", "D", "e", "cap")]


def build(source: str = SOURCE, output: str = LIBRARY) -> str:
    """Compile the oracle with gcc (plain -O2, no vector intrinsics)."""
    tmp = f"{output}.tmp{os.getpid()}"
    cmd = ["gcc", "-O2", "-std=c99", "-Wall", "-Werror", "-shared", "-fPIC",
           "-o", tmp, source]
    subprocess.run(cmd, check=True)
    os.replace(tmp, output)        # atomic: concurrent test workers may build too
    return output


def pool_elems(p) -> int:
    return p.L * p.C * p.H * p.D * p.T * p.N


def _pool(p) -> _Pool:
    if p.layout not in LAYOUT_CODES:
        raise ValueError(f"unknown layout {p.layout!r}")
    return _Pool(p.L, p.C, p.H, p.D, p.T, p.N, p.e, LAYOUT_CODES[p.layout])


def _buf(b) -> _Buf:
    return _Buf(b.L, b.C, b.H, b.D, b.e, b.cap)


def _bytes(a: np.ndarray, nbytes: int, name: str, writable: bool = False) -> np.ndarray:
    if not (isinstance(a, np.ndarray) and a.flags.c_contiguous):
        raise TypeError(f"{name} must be a C-contiguous numpy array")
    if writable and not a.flags.writeable:
        raise ValueError(f"{name} must be writable")
    if a.nbytes != nbytes:
        raise ValueError(f"{name} holds {a.nbytes} bytes, expected {nbytes}")
    return a


def _i32(a) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.int32)
    return a if a.size else np.zeros(1, np.int32)


def _reqs(a) -> tuple[np.ndarray, int]:
    a = np.ascontiguousarray(a, dtype=np.int64).reshape(-1, 6)
    return (a if len(a) else np.zeros((1, 6), np.int64)), len(a)


def _same_elements(a, b):
    for k in ("L", "C", "H", "D", "e"):
        if getattr(a, k) != getattr(b, k):
            raise ValueError(f"element shapes differ in {k}: {getattr(a, k)} vs {getattr(b, k)}")


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


class Oracle:
    """One loaded copy of the oracle library (the tests load planted-mistake
    builds of the same source through this class too)."""

    def __init__(self, path: str = LIBRARY):
        if not os.path.exists(path):
            raise FileNotFoundError(f"{path} is not built; call oracle.kvx_oracle.build()")
        lib = ctypes.CDLL(path)
        vp, i64, u32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint32
        pp, bp = ctypes.POINTER(_Pool), ctypes.POINTER(_Buf)
        lib.ora_transfer.argtypes = [vp, pp, vp, pp, vp, i64, vp, i64, vp, i64]
        lib.ora_transfer.restype = u32
        lib.ora_gather.argtypes = [vp, pp, vp, bp, vp, i64, vp, i64]
        lib.ora_gather.restype = u32
        lib.ora_scatter.argtypes = [vp, bp, vp, pp, vp, i64, vp, i64]
        lib.ora_scatter.restype = u32
        lib.ora_transfer_slice.argtypes = [vp, pp, vp, pp, vp, vp, i64, vp, i64, vp, i64]
        lib.ora_transfer_slice.restype = u32
        lib.ora_gather_slice.argtypes = [vp, pp, vp, bp, vp, vp, i64, vp, i64]
        lib.ora_gather_slice.restype = u32
        lib.ora_scatter_slice.argtypes = [vp, bp, vp, pp, vp, vp, i64, vp, i64]
        lib.ora_scatter_slice.restype = u32
        lib.ora_fnv1a64.argtypes = [vp, i64, ctypes.c_uint64]
        lib.ora_fnv1a64.restype = ctypes.c_uint64
        lib.ora_page_hashes.argtypes = [vp, i64, i64, i64, vp, i64, vp, i64]
        lib.ora_page_hashes.restype = u32
        self.lib = lib

    def transfer(self, src: np.ndarray, src_shape, dst: np.ndarray, dst_shape,
                 src_pt, dst_pt, reqs) -> int:
        """Pool -> pool.  ``dst`` is updated in place; returns the error bits."""
        _same_elements(src_shape, dst_shape)
        _bytes(src, pool_elems(src_shape) * src_shape.e, "src")
        _bytes(dst, pool_elems(dst_shape) * dst_shape.e, "dst", writable=True)
        sp, dp = _i32(src_pt), _i32(dst_pt)
        rq, nr = _reqs(reqs)
        S, D = _pool(src_shape), _pool(dst_shape)
        return int(self.lib.ora_transfer(
            _ptr(src), ctypes.byref(S), _ptr(dst), ctypes.byref(D),
            _ptr(sp), np.asarray(src_pt).size, _ptr(dp), np.asarray(dst_pt).size,
            _ptr(rq), nr))

    def gather(self, src: np.ndarray, src_shape, dst: np.ndarray, buf_shape,
               src_pt, reqs) -> int:
        """Pool -> flat buffer.  ``dst`` is updated in place."""
        _same_elements(src_shape, buf_shape)
        _bytes(src, pool_elems(src_shape) * src_shape.e, "src")
        _bytes(dst, buf_shape.cap * buf_shape.e, "dst", writable=True)
        sp = _i32(src_pt)
        rq, nr = _reqs(reqs)
        S, B = _pool(src_shape), _buf(buf_shape)
        return int(self.lib.ora_gather(
            _ptr(src), ctypes.byref(S), _ptr(dst), ctypes.byref(B),
            _ptr(sp), np.asarray(src_pt).size, _ptr(rq), nr))

    def scatter(self, src: np.ndarray, buf_shape, dst: np.ndarray, dst_shape,
                dst_pt, reqs) -> int:
        """Flat buffer -> pool.  ``dst`` is updated in place."""
        _same_elements(buf_shape, dst_shape)
        _bytes(src, buf_shape.cap * buf_shape.e, "src")
        _bytes(dst, pool_elems(dst_shape) * dst_shape.e, "dst", writable=True)
        dp = _i32(dst_pt)
        rq, nr = _reqs(reqs)
        B, D = _buf(buf_shape), _pool(dst_shape)
        return int(self.lib.ora_scatter(
            _ptr(src), ctypes.byref(B), _ptr(dst), ctypes.byref(D),
            _ptr(dp), np.asarray(dst_pt).size, _ptr(rq), nr))


    @staticmethod
    def _buffer_slice(sl, pool_shape, buf_shape, pool_fields, buf_fields) -> np.ndarray:
        """Check a slice against a pool and a buffer that holds exactly the
        slice: the pool range inside the pool, the buffer offsets zero and
        the buffer's L, C, H equal to the slice counts."""
        sl = [int(x) for x in sl]
        if len(sl) != 9:
            raise ValueError("a slice has nine fields")
        for k, (po, bo, cnt) in zip("LCH", (sl[0:3], sl[3:6], sl[6:9])):
            p_off = po if pool_fields == 0 else bo
            b_off = bo if pool_fields == 0 else po
            if cnt < 0 or p_off < 0 or p_off + cnt > getattr(pool_shape, k):
                raise ValueError(f"slice range {k} does not fit the pool")
            if b_off != 0 or getattr(buf_shape, k) != cnt:
                raise ValueError(f"the buffer must hold exactly the slice in {k}")
        for k in ("D", "e"):
            if getattr(pool_shape, k) != getattr(buf_shape, k):
                raise ValueError(f"element shapes differ in {k}")
        return np.asarray(sl, dtype=np.int64)

    def gather_slice(self, src: np.ndarray, src_shape, dst: np.ndarray, buf_shape, sl,
                     src_pt, reqs) -> int:
        """Slice of a pool -> flat buffer holding exactly the slice (see
        ora_gather_slice).  ``dst`` is updated in place."""
        slc = self._buffer_slice(sl, src_shape, buf_shape, 0, 1)
        _bytes(src, pool_elems(src_shape) * src_shape.e, "src")
        _bytes(dst, buf_shape.cap * buf_shape.e, "dst", writable=True)
        sp = _i32(src_pt)
        rq, nr = _reqs(reqs)
        S, B = _pool(src_shape), _buf(buf_shape)
        return int(self.lib.ora_gather_slice(
            _ptr(src), ctypes.byref(S), _ptr(dst), ctypes.byref(B), _ptr(slc),
            _ptr(sp), np.asarray(src_pt).size, _ptr(rq), nr))

    def scatter_slice(self, src: np.ndarray, buf_shape, dst: np.ndarray, dst_shape, sl,
                      dst_pt, reqs) -> int:
        """Flat buffer holding exactly the slice -> slice of a pool (see
        ora_scatter_slice).  ``dst`` is updated in place."""
        slc = self._buffer_slice(sl, dst_shape, buf_shape, 1, 0)
        _bytes(src, buf_shape.cap * buf_shape.e, "src")
        _bytes(dst, pool_elems(dst_shape) * dst_shape.e, "dst", writable=True)
        dp = _i32(dst_pt)
        rq, nr = _reqs(reqs)
        B, D = _buf(buf_shape), _pool(dst_shape)
        return int(self.lib.ora_scatter_slice(
            _ptr(src), ctypes.byref(B), _ptr(dst), ctypes.byref(D), _ptr(slc),
            _ptr(dp), np.asarray(dst_pt).size, _ptr(rq), nr))

    def transfer_slice(self, src: np.ndarray, src_shape, dst: np.ndarray, dst_shape, sl,
                       src_pt, dst_pt, reqs) -> int:
        """Slice of a pool -> slice of another pool.  ``sl`` is (src_layer0,
        dst_layer0, n_layers, src_kv0, dst_kv0, n_kv, src_head0, dst_head0,
        n_heads); each range must lie inside both pools."""
        sl = [int(x) for x in sl]
        if len(sl) != 9:
            raise ValueError("a slice has nine fields")
        for (o_s, o_d, cnt), ks in ((sl[0:3], "L"), (sl[3:6], "C"), (sl[6:9], "H")):
            if cnt < 0 or o_s < 0 or o_d < 0 or o_s + cnt > getattr(src_shape, ks) \
                    or o_d + cnt > getattr(dst_shape, ks):
                raise ValueError(f"slice range {ks} does not fit the pools")
        for k in ("D", "e"):
            if getattr(src_shape, k) != getattr(dst_shape, k):
                raise ValueError(f"element shapes differ in {k}")
        _bytes(src, pool_elems(src_shape) * src_shape.e, "src")
        _bytes(dst, pool_elems(dst_shape) * dst_shape.e, "dst", writable=True)
        sp, dp = _i32(src_pt), _i32(dst_pt)
        rq, nr = _reqs(reqs)
        S, D = _pool(src_shape), _pool(dst_shape)
        slc = np.asarray(sl, dtype=np.int64)
        return int(self.lib.ora_transfer_slice(
            _ptr(src), ctypes.byref(S), _ptr(dst), ctypes.byref(D), _ptr(slc),
            _ptr(sp), np.asarray(src_pt).size, _ptr(dp), np.asarray(dst_pt).size,
            _ptr(rq), nr))

    def fnv1a64(self, data: bytes, h: int = 0xcbf29ce484222325) -> int:
        """FNV-1a 64 of ``data`` continued from state ``h``."""
        buf = np.frombuffer(bytes(data), dtype=np.uint8) if data else np.zeros(1, np.uint8)
        return int(self.lib.ora_fnv1a64(_ptr(buf), len(data), h))

    def page_hashes(self, payload: np.ndarray, rec_bytes: int, T: int, hreqs, out: np.ndarray) -> int:
        """Chained page hashes (see ora_page_hashes).  ``payload`` holds
        records of ``rec_bytes`` bytes; ``hreqs`` rows are (payload_off,
        out_off, seed, n_positions); ``out`` (uint64) is updated in place."""
        if payload.nbytes % rec_bytes:
            raise ValueError("payload is not a whole number of records")
        p = np.ascontiguousarray(payload).view(np.uint8).reshape(-1)
        if out.dtype != np.uint64 or not out.flags.c_contiguous:
            raise TypeError("out must be a contiguous uint64 array")
        rows = np.ascontiguousarray(
            np.asarray([[int(a), int(b), int(c) - (1 << 64) if int(c) >= 1 << 63 else int(c), int(d)]
                        for a, b, c, d in hreqs], dtype=np.int64).reshape(-1, 4))
        rq = rows if len(rows) else np.zeros((1, 4), np.int64)
        return int(self.lib.ora_page_hashes(_ptr(p if p.size else np.zeros(1, np.uint8)),
                                            p.size // rec_bytes, rec_bytes, T, _ptr(rq), len(rows),
                                            _ptr(out if out.size else np.zeros(1, np.uint64)),
                                            out.size))


_DEFAULT: Oracle | None = None


def default() -> Oracle:
    """The oracle built from ``kvx_oracle.c``; compiled on first use if absent."""
    global _DEFAULT
    if _DEFAULT is None:
        if not os.path.exists(LIBRARY):
            build()
        _DEFAULT = Oracle(LIBRARY)
    return _DEFAULT


def transfer(*a, **k) -> int:
    return default().transfer(*a, **k)


def gather(*a, **k) -> int:
    return default().gather(*a, **k)


def scatter(*a, **k) -> int:
    return default().scatter(*a, **k)


def transfer_slice(*a, **k) -> int:
    return default().transfer_slice(*a, **k)


def page_hashes(*a, **k) -> int:
    return default().page_hashes(*a, **k)
