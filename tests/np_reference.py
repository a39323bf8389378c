"""An independent statement of the copy through numpy indexing.

Used only to pin the C oracle: a pool is viewed as a 6-D numpy array with
axes (layer, page, kv, slot, head, dim) purely through ``reshape`` and
``transpose`` of its memory order, and the copy is one advanced-indexing
assignment per request.  None of the oracle's hand-written offset arithmetic
appears here, so a dropped term, a wrong stride or a transposed axis in the
oracle shows up as a mismatch.  Valid inputs only (no error cases).
"""
from __future__ import annotations

import numpy as np

_DT = {1: np.uint8, 2: np.dtype("<u2"), 4: np.dtype("<u4"), 8: np.dtype("<u8")}


def elems(a: np.ndarray, e: int) -> np.ndarray:
    return a.view(_DT[e])


def canon(a: np.ndarray, s) -> np.ndarray:
    """View a pool's bytes as [layer][page][kv][slot][head][dim]."""
    x = elems(a, s.e)
    L, N, C, T, H, D = s.L, s.N, s.C, s.T, s.H, s.D
    if s.layout == "LPCTHD":
        return x.reshape(L, N, C, T, H, D)
    if s.layout == "LPCHTD":
        return x.reshape(L, N, C, H, T, D).transpose(0, 1, 2, 4, 3, 5)
    if s.layout == "PLCTHD":
        return x.reshape(N, L, C, T, H, D).transpose(1, 0, 2, 3, 4, 5)
    if s.layout == "PLCHTD":
        return x.reshape(N, L, C, H, T, D).transpose(1, 0, 2, 4, 3, 5)
    raise ValueError(s.layout)


def block(a: np.ndarray, b, off: int, n: int) -> np.ndarray:
    """A request's block [layer][kv][token][head][dim] in a flat buffer."""
    x = elems(a, b.e)
    return x[off: off + b.L * b.C * n * b.H * b.D].reshape(b.L, b.C, n, b.H, b.D)


def _where(pt, off, start, n, T):
    q = start + np.arange(n)
    return pt[off + q // T], q % T


def transfer(src, S, dst, Dp, src_pt, dst_pt, reqs) -> None:
    Vs, Vd = canon(src, S), canon(dst, Dp)
    for so, do, _bo, s0, d0, n in np.asarray(reqs, dtype=np.int64).reshape(-1, 6):
        if n == 0:
            continue
        sp, ss = _where(np.asarray(src_pt), so, s0, n, S.T)
        dp, ds = _where(np.asarray(dst_pt), do, d0, n, Dp.T)
        Vd[:, dp, :, ds, :, :] = Vs[:, sp, :, ss, :, :]


def gather(src, S, dst, B, src_pt, reqs) -> None:
    Vs = canon(src, S)
    for so, _do, bo, s0, _d0, n in np.asarray(reqs, dtype=np.int64).reshape(-1, 6):
        if n == 0:
            continue
        sp, ss = _where(np.asarray(src_pt), so, s0, n, S.T)
        block(dst, B, bo, n)[...] = np.moveaxis(Vs[:, sp, :, ss, :, :], 0, 2)


def scatter(src, B, dst, Dp, dst_pt, reqs) -> None:
    Vd = canon(dst, Dp)
    for _so, do, bo, _s0, d0, n in np.asarray(reqs, dtype=np.int64).reshape(-1, 6):
        if n == 0:
            continue
        dp, ds = _where(np.asarray(dst_pt), do, d0, n, Dp.T)
        Vd[:, dp, :, ds, :, :] = np.moveaxis(block(src, B, bo, n), 2, 0)


def transfer_slice(src, S, dst, Dp, sl, src_pt, dst_pt, reqs) -> None:
    """Slice copy: layers, kv components and heads are numpy slices of the
    6-D views, each offset on its own side."""
    sl0, dl0, nl, sc0, dc0, nc, sh0, dh0, nh = [int(x) for x in sl]
    Vs, Vd = canon(src, S), canon(dst, Dp)
    for so, do, _bo, s0, d0, n in np.asarray(reqs, dtype=np.int64).reshape(-1, 6):
        if n == 0:
            continue
        sp, ss = _where(np.asarray(src_pt), so, s0, n, S.T)
        dp, ds = _where(np.asarray(dst_pt), do, d0, n, Dp.T)
        Vd[dl0:dl0 + nl, dp, dc0:dc0 + nc, ds, dh0:dh0 + nh, :] = \
            Vs[sl0:sl0 + nl, sp, sc0:sc0 + nc, ss, sh0:sh0 + nh, :]


def gather_slice(src, S, dst, B, sl, src_pt, reqs) -> None:
    """Slice of a pool -> buffer blocks [nl][nc][n][nh][D]: numpy slices of
    the 6-D source view at the slice's source offsets."""
    sl0, _dl0, nl, sc0, _dc0, nc, sh0, _dh0, nh = [int(x) for x in sl]
    Vs = canon(src, S)
    for so, _do, bo, s0, _d0, n in np.asarray(reqs, dtype=np.int64).reshape(-1, 6):
        if n == 0:
            continue
        sp, ss = _where(np.asarray(src_pt), so, s0, n, S.T)
        block(dst, B, bo, n)[...] = np.moveaxis(
            Vs[sl0:sl0 + nl, sp, sc0:sc0 + nc, ss, sh0:sh0 + nh, :], 0, 2)


def scatter_slice(src, B, dst, Dp, sl, dst_pt, reqs) -> None:
    """Buffer blocks [nl][nc][n][nh][D] -> slice of a pool at the slice's
    destination offsets."""
    _sl0, dl0, nl, _sc0, dc0, nc, _sh0, dh0, nh = [int(x) for x in sl]
    Vd = canon(dst, Dp)
    for _so, do, bo, _s0, d0, n in np.asarray(reqs, dtype=np.int64).reshape(-1, 6):
        if n == 0:
            continue
        dp, ds = _where(np.asarray(dst_pt), do, d0, n, Dp.T)
        Vd[dl0:dl0 + nl, dp, dc0:dc0 + nc, ds, dh0:dh0 + nh, :] = \
            np.moveaxis(block(src, B, bo, n), 2, 0)
