"""Pins for the CPU oracle: checks against facts fixed by the paper's model of
the copy and by plain mathematics, not against the oracle itself.

Each ``pin_*`` function takes an ``oracle.kvx_oracle.Oracle`` and raises
``AssertionError`` on a mismatch.  ``tests/test_oracle.py`` runs them on the
real oracle; ``tests/test_oracle_mutants.py`` runs them (through this file's
``__main__``) on builds with a planted mistake and expects a failure.

The pins:
  * worked examples whose expected rows are written out by hand;
  * the numpy-indexing statement of the copy (``np_reference``) for every
    layout pair, page-size pair, shifted and partial ranges, shared source
    pages and every element width;
  * special cases that reduce to library routines: identity page tables give
    a byte-for-byte copy or an ``np.transpose`` between layouts;
  * invariants: gather -> scatter -> gather returns the buffer; every written
    element decodes (flat-index codes) to exactly one source element at the
    same (layer, kv, head, dim) and the same request-relative token; nothing
    outside the requested positions changes and the source is never written;
  * the documented error rules, case by case.
"""
from __future__ import annotations

import itertools
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
for p in (ROOT, HERE):
    if p not in sys.path:
        sys.path.insert(0, p)

import np_reference as npr  # noqa: E402
from paper_2606_31093_amd.workloads import (  # noqa: E402
    LAYOUTS, BufSpec, PoolSpec, tiny, normal_bf16_bytes, prefill_bytes, random_bytes)

ERR_SRC_PAGE, ERR_DST_PAGE, ERR_PT_RANGE, ERR_BAD_REQ = 1, 2, 4, 8


def _req(so=0, do=0, bo=0, s0=0, d0=0, n=0):
    return [so, do, bo, s0, d0, n]


def _pool_bytes(spec, seed):
    return random_bytes(spec.nbytes, seed)


def _same(a, b, what):
    if not np.array_equal(a, b):
        bad = np.nonzero(a != b)[0]
        raise AssertionError(f"{what}: {len(bad)} bytes differ, first at {bad[:5]}")


# ---------------------------------------------------------------------------
# worked examples written out by hand
# ---------------------------------------------------------------------------

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden_rows(name: str) -> list:
    """Tab-separated rows of a fixture under tests/golden (comments skipped)."""
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                rows.append(line.rstrip("\n").split("\t"))
    return rows


def _check_golden_example(example: str, dst: np.ndarray) -> None:
    rows = [r for r in _golden_rows("layout_hand_examples.txt") if r[0] == example]
    assert rows, example
    for _, start, count, value in rows:
        a, n = int(start), int(count)
        assert (dst[a:a + n] == int(value)).all(), (example, a, n, value, dst[a:a + n])


def pin_hand_example(O):
    """One head of 8 bf16 per row.  Source: 4 pages x 2 tokens, page p slot s
    holds the row filled with 10p + s.  Request: source table [3, 1], start
    1, 3 tokens, into destination table [1] (4-token pages) at start 0.
    Positions 1, 2, 3 live at (page 3, slot 1), (page 1, slot 0),
    (page 1, slot 1): destination page 1 must read rows 31, 10, 11 and keep
    its last slot; page 0 is untouched."""
    S = PoolSpec(L=1, C=1, H=1, D=8, T=2, N=4, e=2, layout="LPCTHD")
    Dp = PoolSpec(L=1, C=1, H=1, D=8, T=4, N=2, e=2, layout="LPCTHD")
    src = np.zeros((4, 2, 8), dtype="<u2")
    for p in range(4):
        for s in range(2):
            src[p, s, :] = 10 * p + s
    dst = np.full((2, 4, 8), 999, dtype="<u2")
    err = O.transfer(src.reshape(-1).view(np.uint8), S, dst.reshape(-1).view(np.uint8), Dp,
                     [3, 1], [1], [_req(s0=1, d0=0, n=3)])
    assert err == 0, err
    _check_golden_example("lpcthd", dst.reshape(-1))


def pin_hand_example_plchtd(O):
    """Two layers, K and V, two heads, 8-element rows; source LPCTHD with
    2-token pages, destination PLCHTD with 4-token pages.  The source row of
    (layer l, kv c, page p, slot s, head h) is filled with 1000l + 100c +
    10h + 4p + s.  A request moves positions 0..2 from table [2, 0] to
    table [1] at start 1.  In PLCHTD [page][layer][kv][head][token][dim]
    with L=2, C=2, H=2, T=4, D=8 the row (page 1, layer 1, kv 0, head 1,
    slot 3) starts at element ((((1*2+1)*2+0)*2+1)*4+3)*8 = 440 and must
    hold position 2 = (source page 0, slot 0): 1000 + 0 + 10 + 0 + 0 = 1010.
    Row (page 1, layer 0, kv 1, head 0, slot 1) at element
    ((((1*2+0)*2+1)*2+0)*4+1)*8 = 328 holds position 0 = (page 2, slot 0):
    0 + 100 + 0 + 8 + 0 = 108.  Slot 0 of destination page 1 is untouched."""
    S = PoolSpec(L=2, C=2, H=2, D=8, T=2, N=3, e=2, layout="LPCTHD")
    Dp = PoolSpec(L=2, C=2, H=2, D=8, T=4, N=2, e=2, layout="PLCHTD")
    src = np.zeros((2, 3, 2, 2, 2, 8), dtype="<u2")      # [l][p][c][s][h][d]
    for l, p, c, s, h in itertools.product(range(2), range(3), range(2), range(2), range(2)):
        src[l, p, c, s, h, :] = 1000 * l + 100 * c + 10 * h + 4 * p + s
    dst = np.full(Dp.elems, 7, dtype="<u2")
    err = O.transfer(src.reshape(-1).view(np.uint8), S, dst.view(np.uint8), Dp,
                     [2, 0], [1], [_req(s0=0, d0=1, n=3)])
    assert err == 0, err
    _check_golden_example("plchtd", dst)


# ---------------------------------------------------------------------------
# numpy-indexing statement of the copy
# ---------------------------------------------------------------------------

def _transfer_case(O, ls, ld, Ts, Td, seed, e=2, D=8, L=2, C=2, H=3):
    rng = np.random.default_rng(seed)
    Ns, Nd = 64 // Ts * 4 + 8, 64 // Td * 4 + 8
    S = PoolSpec(L, C, H, D, T=Ts, N=Ns, e=e, layout=ls)
    Dp = PoolSpec(L, C, H, D, T=Td, N=Nd, e=e, layout=ld)
    src = _pool_bytes(S, seed)
    dst = prefill_bytes(Dp.nbytes, 3)
    sperm, dperm = rng.permutation(Ns).astype(np.int32), rng.permutation(Nd).astype(np.int32)
    # (src_start, dst_start, n, index of a request whose source pages it shares)
    spec = [
        (Ts // 2 + 1, Td - 1, 3 * Ts + 1, None),   # both starts mid-page, ragged end
        (0, 1, 2 * Ts - 1, 0),                     # shares request 0's source pages
        (Ts - 1, 2 * Td - 1, 1, None),             # one token
        (0, 0, 0, None),                           # empty
        (0, 0, min(Td, 2 * Ts), None),             # page-aligned
    ]
    src_pt, dst_pt, reqs, src_offs = [], [], [], []
    for s0, d0, n, share in spec:
        ks, kd = -(-(s0 + n) // Ts), -(-(d0 + n) // Td)
        so = src_offs[share] if share is not None else len(src_pt)
        if share is None:
            src_pt.extend(sperm[len(src_pt): len(src_pt) + ks])
        src_offs.append(so)
        reqs.append(_req(so=so, do=len(dst_pt), s0=s0, d0=d0, n=n))
        dst_pt.extend(dperm[len(dst_pt): len(dst_pt) + kd])
    src_pt, dst_pt = np.asarray(src_pt, np.int32), np.asarray(dst_pt, np.int32)
    exp = dst.copy()
    npr.transfer(src, S, exp, Dp, src_pt, dst_pt, reqs)
    got = dst.copy()
    src_before = src.copy()
    err = O.transfer(src, S, got, Dp, src_pt, dst_pt, reqs)
    assert err == 0, f"{ls}->{ld} T {Ts}->{Td}: error bits {err}"
    _same(got, exp, f"transfer {ls}->{ld} T {Ts}->{Td} e={e}")
    _same(src, src_before, "source modified")


def pin_numpy_transfer(O):
    pairs = [(16, 64), (32, 8), (4, 4), (1, 16), (8, 1)]
    for i, (ls, ld) in enumerate(itertools.product(LAYOUTS, LAYOUTS)):
        for j, (Ts, Td) in enumerate(pairs):
            _transfer_case(O, ls, ld, Ts, Td, seed=100 * i + j)


def pin_numpy_transfer_widths(O):
    """Element widths 1, 2, 4 and 8 bytes (rows of 16 to 64 bytes)."""
    for e, D in ((1, 16), (2, 8), (4, 4), (8, 2), (8, 8), (1, 48)):
        _transfer_case(O, "LPCTHD", "PLCHTD", 4, 8, seed=7 + e + D, e=e, D=D)
        _transfer_case(O, "LPCHTD", "PLCTHD", 8, 4, seed=9 + e + D, e=e, D=D, C=1, H=1)


def _gather_scatter_case(O, layout, T, e, D, seed):
    rng = np.random.default_rng(seed)
    L, C, H, N = 3, 2, 2, 24
    S = PoolSpec(L, C, H, D, T=T, N=N, e=e, layout=layout)
    ns = [5 * T // 2 + 1, 0, 1, 2 * T]
    starts = [T // 2 + 1, 0, T - 1, 0]
    blocks, off = [], 0
    align = 16 // e
    for n in ns:
        blocks.append(off)
        off += -(-(L * C * n * H * D) // align) * align + align    # gaps between blocks
    B = BufSpec(L, C, H, D, e, cap=off)
    perm = rng.permutation(N).astype(np.int32)
    pt, pos, reqs = [], 0, []
    for n, s0, bo in zip(ns, starts, blocks):
        k = -(-(s0 + n) // T)
        reqs.append(_req(so=pos, bo=bo, s0=s0, n=n))
        pt.extend(perm[pos: pos + k])
        pos += k
    pt = np.asarray(pt, np.int32)
    src = _pool_bytes(S, seed)
    buf0 = prefill_bytes(B.nbytes + (-B.nbytes) % 8, 4)[: B.nbytes].copy()
    exp, got = buf0.copy(), buf0.copy()
    npr.gather(src, S, exp, B, pt, reqs)
    assert O.gather(src, S, got, B, pt, reqs) == 0
    _same(got, exp, f"gather {layout} T={T} e={e}")
    # scatter the gathered blocks into a different page set (the source start
    # becomes the destination start)
    sreqs = [[0, r[0], r[2], 0, r[3], r[5]] for r in reqs]
    dperm = rng.permutation(N).astype(np.int32)[: len(pt)]
    pool0 = prefill_bytes(S.nbytes, 5)
    exp2, got2 = pool0.copy(), pool0.copy()
    npr.scatter(exp, B, exp2, S, dperm, sreqs)
    assert O.scatter(got, B, got2, S, dperm, sreqs) == 0
    _same(got2, exp2, f"scatter {layout} T={T} e={e}")


def pin_numpy_gather_scatter(O):
    for i, layout in enumerate(LAYOUTS):
        for T, e, D in ((16, 2, 64), (4, 2, 8), (8, 1, 16), (2, 4, 12), (1, 8, 2)):
            _gather_scatter_case(O, layout, T, e, D, seed=50 + 10 * i + T)


# ---------------------------------------------------------------------------
# special cases that reduce to library routines
# ---------------------------------------------------------------------------

_NATURAL = {"LPCTHD": "LNCTHD", "LPCHTD": "LNCHTD", "PLCTHD": "NLCTHD", "PLCHTD": "NLCHTD"}


def pin_identity_tables(O):
    """Identity page tables, one request over the whole pool: equal layouts
    give a byte-for-byte copy, different layouts give np.transpose between
    their axis orders."""
    L, C, H, D, T, N = 2, 2, 3, 8, 4, 5
    dims = dict(L=L, N=N, C=C, T=T, H=H, D=D)
    for ls, ld in itertools.product(LAYOUTS, LAYOUTS):
        S = PoolSpec(L, C, H, D, T=T, N=N, e=2, layout=ls)
        Dp = PoolSpec(L, C, H, D, T=T, N=N, e=2, layout=ld)
        src = normal_bf16_bytes(S.nbytes, 11)
        dst = prefill_bytes(Dp.nbytes, 6)
        ident = np.arange(N, dtype=np.int32)
        assert O.transfer(src, S, dst, Dp, ident, ident, [_req(n=N * T)]) == 0
        a_src = _NATURAL[ls]
        a_dst = _NATURAL[ld]
        x = src.view("<u2").reshape([dims[k] for k in a_src])
        want = np.transpose(x, [a_src.index(k) for k in a_dst]).reshape(-1)
        if ls == ld:
            _same(dst, src, f"memcpy {ls}")
        _same(dst.view("<u2"), want, f"transpose {ls}->{ld}")


def pin_roundtrip(O):
    """gather(A) -> buffer -> scatter(B) -> gather(B) returns the buffer, for
    pools of different page size and layout."""
    L, C, H, D = 2, 2, 2, 16
    A = PoolSpec(L, C, H, D, T=8, N=20, e=2, layout="PLCTHD")
    Bp = PoolSpec(L, C, H, D, T=16, N=12, e=2, layout="LPCHTD")
    rng = np.random.default_rng(5)
    ns = [37, 16, 5]
    blocks = np.cumsum([0] + [L * C * n * H * D for n in ns])
    buf = BufSpec(L, C, H, D, 2, cap=int(blocks[-1]))
    apt = rng.permutation(A.N).astype(np.int32)
    bpt = rng.permutation(Bp.N).astype(np.int32)
    areqs, breqs, ao, bo = [], [], 0, 0
    for n, b in zip(ns, blocks):
        areqs.append(_req(so=ao, bo=int(b), s0=3, n=n))
        breqs.append(_req(do=bo, bo=int(b), d0=0, n=n))
        ao += -(-(n + 3) // A.T)
        bo += -(-n // Bp.T)
    a = normal_bf16_bytes(A.nbytes, 21)
    b = prefill_bytes(Bp.nbytes, 7)
    buf1 = np.zeros(buf.nbytes, np.uint8)
    buf2 = np.ones(buf.nbytes, np.uint8)
    assert O.gather(a, A, buf1, buf, apt, areqs) == 0
    assert O.scatter(buf1, buf, b, Bp, bpt, breqs) == 0
    g2 = [[r[1], 0, r[2], r[4], 0, r[5]] for r in breqs]
    assert O.gather(b, Bp, buf2, buf, bpt, g2) == 0
    _same(buf2, buf1, "gather/scatter/gather round trip")
    # pool -> pool -> pool: A -> B -> fresh A' at the same positions
    b2 = prefill_bytes(Bp.nbytes, 8)
    treqs = [[ar[0], br[1], 0, 3, 0, n] for ar, br, n in zip(areqs, breqs, ns)]
    assert O.transfer(a, A, b2, Bp, apt, bpt, treqs) == 0
    a2 = prefill_bytes(A.nbytes, 9)
    back = [[br[1], ar[0], 0, 0, 3, n] for ar, br, n in zip(areqs, breqs, ns)]
    assert O.transfer(b2, Bp, a2, A, bpt, apt, back) == 0
    buf3 = np.zeros(buf.nbytes, np.uint8)
    assert O.gather(a2, A, buf3, buf, apt, areqs) == 0
    _same(buf3, buf1, "transfer there and back")


# ---------------------------------------------------------------------------
# bijection and untouched bytes, with flat-index codes
# ---------------------------------------------------------------------------

def _coords(flat, spec):
    """(layer, page, kv, slot, head, dim) of flat element indices, via
    np.unravel_index over the layout's axis order."""
    order = _NATURAL[spec.layout]
    dims = dict(L=spec.L, N=spec.N, C=spec.C, T=spec.T, H=spec.H, D=spec.D)
    u = np.unravel_index(flat, [dims[k] for k in order])
    got = dict(zip(order, u))
    return got["L"], got["N"], got["C"], got["T"], got["H"], got["D"]


def _bijection_case(O, ls, ld, Ts, Td, seed):
    rng = np.random.default_rng(seed)
    L, C, H, D = 2, 2, 2, 4
    S = PoolSpec(L, C, H, D, T=Ts, N=48 // Ts, e=4, layout=ls)
    Dp = PoolSpec(L, C, H, D, T=Td, N=48 // Td, e=4, layout=ld)
    SENT = np.uint32(0xFFFFFFFF)
    src = np.arange(S.elems, dtype="<u4")
    dst = np.full(Dp.elems, SENT, dtype="<u4")
    sperm = rng.permutation(S.N).astype(np.int32)
    dperm = rng.permutation(Dp.N).astype(np.int32)
    # two requests; starts chosen so page phases differ between the sides
    ns, s0s, d0s = [13, 7], [Ts // 2 + 1, 0], [1, Td - 1 if Td > 1 else 0]
    src_pt, dst_pt, reqs, so, do = [], [], [], 0, 0
    for n, s0, d0 in zip(ns, s0s, d0s):
        ks, kd = -(-(s0 + n) // Ts), -(-(d0 + n) // Td)
        reqs.append(_req(so=so, do=do, s0=s0, d0=d0, n=n))
        src_pt.extend(sperm[so: so + ks])
        dst_pt.extend(dperm[do: do + kd])
        so, do = so + ks, do + kd
    src_pt, dst_pt = np.asarray(src_pt, np.int32), np.asarray(dst_pt, np.int32)
    src_before = src.copy()
    assert O.transfer(src.view(np.uint8), S, dst.view(np.uint8), Dp, src_pt, dst_pt, reqs) == 0
    _same(src.view(np.uint8), src_before.view(np.uint8), "source modified")
    written = np.nonzero(dst != SENT)[0]
    assert len(written) == sum(ns) * L * C * H * D, (len(written), sum(ns))
    codes = dst[written].astype(np.int64)
    assert len(np.unique(codes)) == len(codes), "a source element landed twice"
    sl, sp, sc, ss, sh, sd = _coords(codes, S)
    dl, dp, dc, ds, dh, dd = _coords(written, Dp)
    assert (sl == dl).all() and (sc == dc).all() and (sh == dh).all() and (sd == dd).all()
    # request-relative token of each side, through the inverse page tables
    def rel(pages, slots, pt, T, which):
        req = np.full(len(pages), -1)
        tok = np.full(len(pages), -1)
        for r, row in enumerate(reqs):
            off, start, n = row[which], row[3 + which], row[5]
            k = -(-(start + n) // T)
            for j in range(k):
                m = pages == pt[off + j]
                q = j * T + slots[m]
                ok = (q >= start) & (q < start + n)
                idx = np.nonzero(m)[0][ok]
                req[idx], tok[idx] = r, (q - start)[ok]
        return req, tok
    rs, ts = rel(sp, ss, src_pt, Ts, 0)
    rd, td = rel(dp, ds, dst_pt, Td, 1)
    assert (rs >= 0).all() and (rd >= 0).all(), "element outside every request"
    assert (rs == rd).all() and (ts == td).all(), "element landed at the wrong token"


def pin_bijection(O):
    for i, (ls, ld) in enumerate(itertools.product(LAYOUTS, LAYOUTS)):
        for Ts, Td in ((4, 8), (8, 4), (2, 2), (3, 16)):
            _bijection_case(O, ls, ld, Ts, Td, seed=300 + 7 * i + Ts)


# ---------------------------------------------------------------------------
# documented error rules
# ---------------------------------------------------------------------------

def pin_errors(O):
    L, C, H, D, T = 1, 2, 1, 8, 4
    S = PoolSpec(L, C, H, D, T=T, N=4, e=2, layout="LPCTHD")
    Dp = PoolSpec(L, C, H, D, T=T, N=4, e=2, layout="LPCTHD")
    src = random_bytes(S.nbytes, 1)
    base = prefill_bytes(Dp.nbytes, 2)

    def run(src_pt, dst_pt, reqs):
        d = base.copy()
        return O.transfer(src, S, d, Dp, src_pt, dst_pt, reqs), d

    def tok_rows(d, page):      # bytes of one destination page (all slots)
        return d.reshape(L, Dp.N, C, T, H * D * 2)[:, page]

    good = [0, 1]
    # a source page id equal to N: positions on that page are skipped
    err, d = run([0, 4], good, [_req(n=8)])
    assert err == ERR_SRC_PAGE, err
    ok, _ = run([0, 1], good, [_req(n=8)])
    assert ok == 0
    assert not np.array_equal(tok_rows(d, 0), tok_rows(base, 0))
    _same(tok_rows(d, 1), tok_rows(base, 1), "skipped page written")
    # a negative destination page id
    err, d = run([0, 1], [-1, 1], [_req(n=8)])
    assert err == ERR_DST_PAGE, err
    _same(tok_rows(d, 0), tok_rows(base, 0), "skipped destination written")
    # both sides bad at the same positions: the destination is resolved first
    err, _ = run([7, 1], [-1, 1], [_req(n=4)])
    assert err == ERR_DST_PAGE, err
    err, _ = run([7, 1], [0, 1], [_req(n=4)])
    assert err == ERR_SRC_PAGE, err
    # a page table shorter than the range
    err, d = run([0], [0, 1], [_req(n=8)])
    assert err == ERR_PT_RANGE, err
    _same(tok_rows(d, 1), tok_rows(base, 1), "position past the table written")
    err, _ = run([0, 1], [0, 1], [_req(do=1, n=8)])
    assert err == ERR_PT_RANGE, err
    # malformed records are skipped whole
    for bad in (_req(n=-1), _req(s0=-1, n=2), _req(d0=-4, n=2),
                _req(s0=2**31 - 2, n=3)):
        err, d = run(good, good, [bad, _req(so=0, do=0, n=0)])
        assert err == ERR_BAD_REQ, (bad, err)
        _same(d, base, "malformed request wrote")
    # buffer sides: the buffer-side start must be 0, the block must be
    # 16-byte aligned and inside the buffer; a block that ends exactly at
    # the buffer's end is fine
    n = 3
    B = BufSpec(L, C, H, D, 2, cap=L * C * n * H * D + 8)
    bufsz = B.nbytes
    for r, want in ((_req(n=n, bo=8), 0), (_req(n=n, bo=0), 0), (_req(n=n, bo=16), ERR_BAD_REQ),
                    (_req(n=n, bo=4), ERR_BAD_REQ), (_req(n=n, bo=-8), ERR_BAD_REQ),
                    (_req(n=n, d0=1), ERR_BAD_REQ)):
        buf = np.zeros(bufsz, np.uint8)
        err = O.gather(src, S, buf, B, [0, 1], [r])
        assert err == want, (r, err, want)
        if want:
            assert not buf.any()
    for r, want in ((_req(n=n, bo=8), 0), (_req(n=n, bo=16), ERR_BAD_REQ),
                    (_req(n=n, s0=2), ERR_BAD_REQ)):
        d = base.copy()
        err = O.scatter(np.ones(bufsz, np.uint8), B, d, Dp, [2, 3], [r])
        assert err == want, (r, err, want)
        if want:
            _same(d, base, "malformed scatter wrote")


def pin_max_position(O):
    """A request's end position (exclusive) may reach 2**31 - 1 and no
    further: a 5-token request ending exactly there, on 65536-token pages
    (page-table entry 32767)."""
    T = 1 << 16
    S = PoolSpec(1, 1, 1, 8, T=T, N=1, e=2, layout="LPCTHD")
    src = normal_bf16_bytes(S.nbytes, 3)
    B = BufSpec(1, 1, 1, 8, 2, cap=5 * 8)
    pt = np.zeros(32768, np.int32)
    start = 2**31 - 6
    buf = np.zeros(B.nbytes, np.uint8)
    assert O.gather(src, S, buf, B, pt, [_req(s0=start, n=5)]) == 0
    _same(buf, src[(T - 6) * 16: (T - 1) * 16], "last positions of the int32 range")
    assert O.gather(src, S, buf, B, pt, [_req(s0=start + 1, n=5)]) == ERR_BAD_REQ


# ---------------------------------------------------------------------------
# the tiny workload end to end
# ---------------------------------------------------------------------------

def pin_tiny_workload(O):
    wl = tiny()
    A, buf, B = wl.sides["A"], wl.sides["buf"], wl.sides["B"]
    g, s = wl.steps
    a = normal_bf16_bytes(A.nbytes, wl.value_seed)
    want_buf = np.zeros(buf.nbytes, np.uint8)
    npr.gather(a, A, want_buf, buf, g.src_pt, g.reqs)
    got_buf = np.zeros(buf.nbytes, np.uint8)
    assert O.gather(a, A, got_buf, buf, g.src_pt, g.reqs) == 0
    _same(got_buf, want_buf, "tiny gather")
    b0 = prefill_bytes(B.nbytes, wl.prefill_tag)
    want_b, got_b = b0.copy(), b0.copy()
    npr.scatter(want_buf, buf, want_b, B, s.dst_pt, s.reqs)
    assert O.scatter(got_buf, buf, got_b, B, s.dst_pt, s.reqs) == 0
    _same(got_b, want_b, "tiny scatter")
    back = np.zeros(buf.nbytes, np.uint8)
    assert O.gather(got_b, B, back, buf, s.dst_pt,
                    [[0, 0, 0, 0, 0, int(s.reqs[0, 5])]]) == 0
    _same(back, got_buf, "tiny round trip")


# ---------------------------------------------------------------------------
# slices (layer range, kv range, head range)
# ---------------------------------------------------------------------------

def pin_slice_hand_example(O):
    """Source: 2 layers, K and V, 4 heads, 8-element rows, one 2-token page.
    Row (layer l, kv c, slot s, head h) holds 1000l + 100c + 10h + s.
    Copy layer 1, V only, heads 2..3 into a 1-layer, 1-kv, 2-head pool whose
    2-token page 0 starts at position 0.  Destination row (slot s, head h)
    must hold 1000 + 100 + 10(2 + h) + s: 1120, 1130, 1121, 1131 in
    [slot][head] order."""
    S = PoolSpec(L=2, C=2, H=4, D=8, T=2, N=1, e=2, layout="LPCTHD")
    Dp = PoolSpec(L=1, C=1, H=2, D=8, T=2, N=1, e=2, layout="LPCTHD")
    src = np.zeros((2, 1, 2, 2, 4, 8), dtype="<u2")
    for l, c, s_, h in itertools.product(range(2), range(2), range(2), range(4)):
        src[l, 0, c, s_, h, :] = 1000 * l + 100 * c + 10 * h + s_
    dst = np.zeros(Dp.elems, dtype="<u2")
    err = O.transfer_slice(src.reshape(-1).view(np.uint8), S, dst.view(np.uint8), Dp,
                           (1, 0, 1, 1, 0, 1, 2, 0, 2), [0], [0], [_req(n=2)])
    assert err == 0
    assert list(dst[::8]) == [1120, 1130, 1121, 1131], dst[::8]


def _slice_case(O, ls, ld, Ts, Td, S_LCH, D_LCH, sl, seed):
    rng = np.random.default_rng(seed)
    (Ls, Cs, Hs), (Ld, Cd, Hd) = S_LCH, D_LCH
    spec = [(Ts // 2 + 1, Td - 1, 3 * Ts + 1), (0, 1, 2 * Ts - 1), (Ts - 1, 0, 1)]
    ks = [-(-(s0 + n) // Ts) for s0, _, n in spec]
    kd = [-(-(d0 + n) // Td) for _, d0, n in spec]
    S = PoolSpec(Ls, Cs, Hs, 8, T=Ts, N=sum(ks) + 3, e=2, layout=ls)
    Dp = PoolSpec(Ld, Cd, Hd, 8, T=Td, N=sum(kd) + 3, e=2, layout=ld)
    sp_, dp_ = rng.permutation(S.N).astype(np.int32), rng.permutation(Dp.N).astype(np.int32)
    reqs, so, do = [], 0, 0
    for (s0, d0, n), a, b in zip(spec, ks, kd):
        reqs.append(_req(so=so, do=do, s0=s0, d0=d0, n=n))
        so, do = so + a, do + b
    src = _pool_bytes(S, seed)
    dst = prefill_bytes(Dp.nbytes, 12)
    exp = dst.copy()
    npr.transfer_slice(src, S, exp, Dp, sl, sp_[:so], dp_[:do], reqs)
    assert O.transfer_slice(src, S, dst, Dp, sl, sp_[:so], dp_[:do], reqs) == 0
    _same(dst, exp, f"slice {sl} {ls}->{ld} T {Ts}->{Td}")


def pin_slice_numpy(O):
    """Layer, kv and head ranges at offsets on both sides, pools of different
    layer / kv / head counts, every layout pair."""
    cases = [((4, 2, 8), (2, 2, 4), (2, 0, 2, 0, 0, 2, 4, 0, 4)),     # TP=2 shard, layer stage
             ((3, 2, 4), (3, 1, 4), (0, 0, 3, 1, 0, 1, 0, 0, 4)),     # V only
             ((3, 2, 4), (5, 2, 6), (0, 2, 3, 0, 0, 2, 1, 3, 2)),     # into a larger pool
             ((2, 1, 1), (2, 1, 3), (0, 0, 2, 0, 0, 1, 0, 2, 1))]     # one head into head 2
    for i, (ls, ld) in enumerate(itertools.product(LAYOUTS, LAYOUTS)):
        for j, (a, b, sl) in enumerate(cases):
            _slice_case(O, ls, ld, 4, 8, a, b, sl, seed=500 + 10 * i + j)


def pin_slice_decomposes_transfer(O):
    """Full ranges equal the plain transfer; K then V, or one head half then
    the other, or one layer half then the other, add up to it too."""
    rng = np.random.default_rng(9)
    L, C, H = 4, 2, 4
    for ls, ld in (("LPCTHD", "PLCHTD"), ("LPCHTD", "LPCTHD")):
        S = PoolSpec(L, C, H, 8, T=4, N=12, e=2, layout=ls)
        Dp = PoolSpec(L, C, H, 8, T=8, N=8, e=2, layout=ld)
        src = _pool_bytes(S, 3)
        spt = rng.permutation(S.N).astype(np.int32)
        dpt = rng.permutation(Dp.N).astype(np.int32)
        reqs = [_req(so=0, do=0, s0=3, d0=5, n=20), _req(so=7, do=4, s0=0, d0=0, n=9)]
        base = prefill_bytes(Dp.nbytes, 4)
        full = base.copy()
        assert O.transfer(src, S, full, Dp, spt, dpt, reqs) == 0
        whole = base.copy()
        assert O.transfer_slice(src, S, whole, Dp, (0, 0, L, 0, 0, C, 0, 0, H), spt, dpt, reqs) == 0
        _same(whole, full, "full slice")
        for parts in (((0, 0, L, 0, 0, 1, 0, 0, H), (0, 0, L, 1, 1, 1, 0, 0, H)),
                      ((0, 0, L, 0, 0, C, 0, 0, 2), (0, 0, L, 0, 0, C, 2, 2, 2)),
                      ((0, 0, 1, 0, 0, C, 0, 0, H), (1, 1, 3, 0, 0, C, 0, 0, H))):
            acc = base.copy()
            for sl in parts:
                assert O.transfer_slice(src, S, acc, Dp, sl, spt, dpt, reqs) == 0
            _same(acc, full, f"parts {parts}")


def pin_slice_tp_roundtrip(O):
    """8 heads split into two 4-head shards (one pool each), then merged back
    into an 8-head pool: the result equals a plain transfer."""
    rng = np.random.default_rng(2)
    S = PoolSpec(2, 2, 8, 8, T=4, N=10, e=2, layout="LPCTHD")
    half = PoolSpec(2, 2, 4, 8, T=8, N=6, e=2, layout="PLCHTD")
    spt = rng.permutation(S.N).astype(np.int32)
    hpt = rng.permutation(half.N).astype(np.int32)
    reqs = [_req(so=0, do=0, s0=1, d0=0, n=30)]
    back_reqs = [_req(so=0, do=0, s0=0, d0=1, n=30)]
    src = _pool_bytes(S, 8)
    shards = []
    for h0 in (0, 4):
        sh = prefill_bytes(half.nbytes, 5)
        assert O.transfer_slice(src, S, sh, half, (0, 0, 2, 0, 0, 2, h0, 0, 4), spt, hpt, reqs) == 0
        shards.append(sh)
    merged = prefill_bytes(S.nbytes, 6)
    mpt = rng.permutation(S.N).astype(np.int32)
    for h0, sh in zip((0, 4), shards):
        assert O.transfer_slice(sh, half, merged, S, (0, 0, 2, 0, 0, 2, 0, h0, 4), hpt, mpt,
                                back_reqs) == 0
    want = prefill_bytes(S.nbytes, 6)
    # positions 1..30 of the source land at 1..30 of the merged pool
    assert O.transfer(src, S, want, S, spt, mpt, [_req(so=0, do=0, s0=1, d0=1, n=30)]) == 0
    _same(merged, want, "TP split and merge")



def pin_slice_errors(O):
    """The slice copy follows the same error rules as the plain transfer."""
    S = PoolSpec(2, 2, 2, 8, T=4, N=4, e=2, layout="LPCTHD")
    Dp = PoolSpec(1, 1, 2, 8, T=4, N=4, e=2, layout="LPCTHD")
    src = random_bytes(S.nbytes, 1)
    base = prefill_bytes(Dp.nbytes, 2)
    sl = (1, 0, 1, 1, 0, 1, 0, 0, 2)
    for spt, dpt, row, bits in (([0, 4], [0, 1], _req(n=8), ERR_SRC_PAGE),
                                ([7, 1], [-1, 1], _req(n=4), ERR_DST_PAGE),
                                ([0], [0, 1], _req(n=8), ERR_PT_RANGE),
                                ([0, 1], [0, 1], _req(n=-2), ERR_BAD_REQ),
                                ([0, 1], [2, 3], _req(s0=1, d0=2, n=5), 0)):
        d = base.copy()
        assert O.transfer_slice(src, S, d, Dp, sl, spt, dpt, [row]) == bits, (spt, dpt, row)
        if bits == ERR_DST_PAGE or bits == ERR_BAD_REQ:
            _same(d, base, "skipped positions written")
    # a slice with no layer, kv component or head copies nothing and checks
    # nothing: damaged tables and malformed records raise no bit
    for empty in ((1, 0, 0, 1, 0, 1, 0, 0, 2), (1, 0, 1, 1, 0, 0, 0, 0, 2),
                  (1, 0, 1, 1, 0, 1, 0, 0, 0)):
        d = base.copy()
        assert O.transfer_slice(src, S, d, Dp, empty, [9, 9], [-1, 7], [_req(n=8), _req(n=-2)]) == 0
        _same(d, base, "an empty slice wrote")



# ---------------------------------------------------------------------------
# slices through a flat buffer (gather_slice / scatter_slice)
# ---------------------------------------------------------------------------

def _slice_buffer_case(layout, sl, seed, T=4):
    """A 3-layer, 2-kv, 4-head pool, three requests (shifted, ragged, empty)
    and a buffer holding exactly the slice, blocks 16-byte aligned with gaps."""
    rng = np.random.default_rng(seed)
    P = PoolSpec(3, 2, 4, 8, T=T, N=12, e=2, layout=layout)
    nl, nc, nh = sl[2], sl[5], sl[8]
    reqs, pt, off, blocks = [], [], 0, []
    perm = rng.permutation(P.N).astype(np.int32)
    for s0, n in ((1, 7), (0, 5), (2, 0)):
        k = -(-(s0 + n) // T)
        reqs.append(_req(so=len(pt), bo=off, s0=s0, n=n))
        pt.extend(perm[len(pt): len(pt) + k])
        off += -(-(nl * nc * n * nh * 8) // 8) * 8 + 8
    B = BufSpec(nl, nc, nh, 8, 2, cap=off)
    return P, B, np.asarray(pt, np.int32), reqs


BUFFER_SLICES = [(0, 0, 3, 0, 0, 2, 0, 0, 4),      # everything
                 (0, 0, 3, 0, 0, 1, 0, 0, 4),      # K only
                 (0, 0, 3, 1, 0, 1, 0, 0, 4),      # V only
                 (1, 0, 2, 0, 0, 2, 2, 0, 2),      # layers 1-2, heads 2-3
                 (2, 0, 1, 1, 0, 1, 3, 0, 1)]      # one row per token


def pin_buffer_slice_numpy(O):
    """gather_slice and scatter_slice against numpy slicing of the 6-D views,
    for every layout and slice shape."""
    for layout, k in itertools.product(LAYOUTS, range(len(BUFFER_SLICES))):
        sl = BUFFER_SLICES[k]
        P, B, pt, reqs = _slice_buffer_case(layout, sl, 50 + k)
        pool = _pool_bytes(P, 60 + k)
        got, want = np.zeros(B.nbytes, np.uint8), np.zeros(B.nbytes, np.uint8)
        assert O.gather_slice(pool, P, got, B, sl, pt, reqs) == 0
        npr.gather_slice(pool, P, want, B, sl, pt, reqs)
        _same(got, want, f"gather_slice {layout} {sl}")
        # scatter the buffer into a second pool at the slice's pool offsets
        ssl = (0, sl[0], sl[2], 0, sl[3], sl[5], 0, sl[6], sl[8])
        dpt = np.random.default_rng(70 + k).permutation(P.N).astype(np.int32)[: len(pt)]
        srows = [_req(do=r[0], bo=r[2], d0=r[3], n=r[5]) for r in reqs]
        d_got = prefill_bytes(P.nbytes, 5)
        d_want = d_got.copy()
        assert O.scatter_slice(got, B, d_got, P, ssl, dpt, srows) == 0
        npr.scatter_slice(got, B, d_want, P, ssl, dpt, srows)
        _same(d_got, d_want, f"scatter_slice {layout} {sl}")


def pin_buffer_slice_full_and_parts(O):
    """The full slice equals the plain gather; K-only and V-only blocks are
    the two kv halves of the full block, and two head halves fill it."""
    for layout in LAYOUTS:
        full = BUFFER_SLICES[0]
        P, B, pt, reqs = _slice_buffer_case(layout, full, 80)
        pool = _pool_bytes(P, 81)
        plain, whole = np.zeros(B.nbytes, np.uint8), np.zeros(B.nbytes, np.uint8)
        assert O.gather(pool, P, plain, B, pt, reqs) == 0
        assert O.gather_slice(pool, P, whole, B, full, pt, reqs) == 0
        _same(whole, plain, f"full slice {layout}")
        parts = {}
        for name, sl in (("k", (0, 0, 3, 0, 0, 1, 0, 0, 4)), ("v", (0, 0, 3, 1, 0, 1, 0, 0, 4)),
                         ("h0", (0, 0, 3, 0, 0, 2, 0, 0, 2)), ("h1", (0, 0, 3, 0, 0, 2, 2, 0, 2))):
            Pp, Bp, ppt, preqs = _slice_buffer_case(layout, sl, 80)
            buf = np.zeros(Bp.nbytes, np.uint8)
            assert O.gather_slice(pool, P, buf, Bp, sl, ppt, preqs) == 0
            parts[name] = (buf, Bp, preqs)
        for (bo, n), r in zip([(q[2], q[5]) for q in reqs], range(len(reqs))):
            if n == 0:
                continue
            W = npr.block(whole, B, bo, n)                       # [3][2][n][4][8]
            K = npr.block(parts["k"][0], parts["k"][1], parts["k"][2][r][2], n)
            V = npr.block(parts["v"][0], parts["v"][1], parts["v"][2][r][2], n)
            H0 = npr.block(parts["h0"][0], parts["h0"][1], parts["h0"][2][r][2], n)
            H1 = npr.block(parts["h1"][0], parts["h1"][1], parts["h1"][2][r][2], n)
            assert np.array_equal(W[:, 0:1], K) and np.array_equal(W[:, 1:2], V), layout
            assert np.array_equal(W[..., 0:2, :], H0) and np.array_equal(W[..., 2:4, :], H1), layout


def pin_buffer_slice_roundtrip(O):
    """V of layers 1-2 offloaded and restored into fresh pages: exactly that
    part of the fresh pages changes, and it equals the source."""
    for layout in LAYOUTS:
        sl = (1, 0, 2, 1, 0, 1, 0, 0, 4)
        P, B, pt, reqs = _slice_buffer_case(layout, sl, 90)
        pool = _pool_bytes(P, 91)
        buf = np.zeros(B.nbytes, np.uint8)
        assert O.gather_slice(pool, P, buf, B, sl, pt, reqs) == 0
        fresh = np.random.default_rng(92).permutation(P.N).astype(np.int32)[: len(pt)]
        back = prefill_bytes(P.nbytes, 9)
        before = back.copy()
        srows = [_req(do=r[0], bo=r[2], d0=r[3], n=r[5]) for r in reqs]
        assert O.scatter_slice(buf, B, back, P, (0, 1, 2, 0, 1, 1, 0, 0, 4), fresh, srows) == 0
        Vs, Vb, V0 = npr.canon(pool, P), npr.canon(back, P), npr.canon(before, P)
        changed = np.zeros(Vb.shape[:5], bool)
        for (so, do, bo, s0, d0, n), in zip([(r[0], r[1], r[2], r[3], r[4], r[5]) for r in reqs]):
            for i in range(n):
                q = s0 + i
                sp, ss = pt[so + q // P.T], q % P.T
                dp, ds = fresh[so + q // P.T], q % P.T
                assert np.array_equal(Vb[1:3, dp, 1, ds], Vs[1:3, sp, 1, ss]), layout
                changed[1:3, dp, 1, ds] = True
        assert np.array_equal(Vb[~changed], V0[~changed]), layout


def pin_buffer_slice_errors(O):
    """The plain gather/scatter error rules hold for slices, and a slice with
    a zero count copies and checks nothing."""
    sl = (0, 0, 1, 1, 0, 1, 0, 0, 2)
    P = PoolSpec(2, 2, 2, 8, T=4, N=4, e=2, layout="LPCTHD")
    B = BufSpec(1, 1, 2, 8, 2, cap=1 * 1 * 8 * 2 * 8)
    pool = _pool_bytes(P, 3)
    for pt, row, bits in (([0, 4], _req(n=8), ERR_SRC_PAGE), ([0], _req(n=8), ERR_PT_RANGE),
                          ([0, 1], _req(n=8, d0=1), ERR_BAD_REQ),
                          ([0, 1], _req(n=8, bo=4), ERR_BAD_REQ),
                          ([0, 1], _req(n=9), ERR_BAD_REQ),
                          ([0, 1], _req(n=8), 0)):
        buf = np.full(B.nbytes, 0xEE, np.uint8)
        assert O.gather_slice(pool, P, buf, B, sl, pt, [row]) == bits, (pt, row)
        if bits == ERR_BAD_REQ:
            assert (buf == 0xEE).all()
    buf = np.full(B.nbytes, 0xEE, np.uint8)
    d = prefill_bytes(P.nbytes, 4)
    before = d.copy()
    for rule in ((0, 0, 1, 0, 1, 1, 0, 0, 2),):
        assert O.scatter_slice(buf, B, d, P, rule, [-1, 4], [_req(n=8)]) == ERR_DST_PAGE
        assert O.scatter_slice(buf, B, d, P, rule, [-1], [_req(n=8)]) == ERR_DST_PAGE | ERR_PT_RANGE
        assert O.scatter_slice(buf, B, d, P, rule, [0, 1], [_req(n=8, s0=1)]) == ERR_BAD_REQ
    _same(d, before, "skipped positions written")
    for empty in ((0, 0, 0, 1, 0, 1, 0, 0, 2), (0, 0, 1, 1, 0, 0, 0, 0, 2), (0, 0, 1, 1, 0, 1, 0, 0, 0)):
        Be = BufSpec(empty[2], empty[5], empty[8], 8, 2, cap=64)
        assert O.gather_slice(pool, P, np.zeros(Be.nbytes, np.uint8), Be, empty, [9], [_req(n=-3)]) == 0
        se = (0, empty[0], empty[2], 0, empty[3], empty[5], 0, empty[6], empty[8])
        assert O.scatter_slice(np.zeros(Be.nbytes, np.uint8), Be, d, P, se, [-1], [_req(n=8)]) == 0
    _same(d, before, "an empty slice wrote")


# ---------------------------------------------------------------------------
# copy-on-write inside one pool
# ---------------------------------------------------------------------------

def pin_same_pool_copy_on_write(O):
    """Sec. 4.1.4: a request forks from a shared prefix whose last page is
    partly filled; its copy of that page goes to a fresh page of the same
    pool before it appends.  Source and destination are the same array; the
    pages written are disjoint from the pages read, so the copy equals the
    numpy statement (which reads everything before writing)."""
    for layout in LAYOUTS:
        P = PoolSpec(2, 2, 3, 8, T=8, N=12, e=2, layout=layout)
        pool = _pool_bytes(P, 41)
        # shared prefix: pages [5, 2, 9], 20 tokens (page 9 holds slots 0..3)
        # fork A copies its partial last page 9 -> fresh page 7 (positions 16..19)
        # fork B duplicates the whole prefix into fresh pages [0, 11, 3]
        src_pt = np.array([5, 2, 9], np.int32)
        dst_pt = np.array([0, 11, 3, 7], np.int32)
        reqs = [_req(so=2, do=3, s0=0, d0=0, n=4),        # page 9 slots 0..3 -> page 7
                _req(so=0, do=0, s0=0, d0=0, n=20)]       # prefix -> pages 0, 11, 3
        want = pool.copy()
        npr.transfer(pool.copy(), P, want, P, src_pt, dst_pt, reqs)
        got = pool.copy()
        assert O.transfer(got, P, got, P, src_pt, dst_pt, reqs) == 0
        _same(got, want, f"copy-on-write {layout}")
        V = npr.canon(got, P)
        assert np.array_equal(V[:, 7, :, :4], V[:, 9, :, :4])            # forked page
        assert np.array_equal(V[:, [0, 11], :, :], V[:, [5, 2], :, :])   # duplicated prefix



# ---------------------------------------------------------------------------
# chained page hashes
# ---------------------------------------------------------------------------

FNV_BASIS = 0xcbf29ce484222325


def pin_fnv_published_vectors(O):
    """FNV-1a 64 test vectors published with the algorithm
    (tests/golden/fnv1a64_vectors.txt)."""
    rows = _golden_rows("fnv1a64_vectors.txt")
    assert len(rows) >= 3
    for text, want in rows:
        data = json.loads(text).encode("ascii")
        assert O.fnv1a64(data) == int(want, 16), (data, hex(O.fnv1a64(data)))


def _hashes(O, payload, rec_bytes, T, rows, n_out):
    out = np.zeros(n_out, np.uint64)
    err = O.page_hashes(payload, rec_bytes, T, rows, out)
    return err, [int(x) for x in out]


def pin_hash_definition(O):
    """A one-page request: its hash is the FNV-1a of the seed's and the page
    digest's little-endian bytes, the digest being the FNV-1a of the page."""
    rng = np.random.default_rng(3)
    page = rng.integers(0, 2**31, size=16, dtype=np.int32)
    for seed in (0, 0x0123456789ABCDEF, 2**64 - 1):
        err, out = _hashes(O, page, 4, 16, [(0, 0, seed, 16)], 1)
        c = O.fnv1a64(page.tobytes())
        want = O.fnv1a64(seed.to_bytes(8, "little") + c.to_bytes(8, "little"))
        assert err == 0 and out[0] == want


def pin_hash_prefix_property(O):
    """Requests that share their first k pages share their first k hashes
    and differ from page k on (a changed page changes every later hash)."""
    rng = np.random.default_rng(5)
    T, n = 8, 70
    a = rng.integers(0, 50000, size=n, dtype=np.int32)
    b = a.copy()
    b[3 * T + 2] += 1                      # page 3 differs
    payload = np.concatenate([a, b, a])
    rows = [(0, 0, 7, n), (n, 9, 7, n), (2 * n, 18, 7, n)]
    err, out = _hashes(O, payload, 4, T, rows, 27)
    assert err == 0
    ha, hb, hc = out[0:9], out[9:18], out[18:27]
    assert ha == hc
    assert ha[:3] == hb[:3] and all(x != y for x, y in zip(ha[3:], hb[3:]))
    assert len(set(ha)) == 9               # no two pages of a chain collide here


def pin_hash_continuation(O):
    """Hashing [0, n) equals hashing [0, kT) and then [kT, n) seeded with
    the hash of page k - 1 (incremental matching)."""
    rng = np.random.default_rng(6)
    T, n, k = 4, 23, 3
    pay = rng.integers(0, 2**31, size=n * 2, dtype=np.int32)     # 8-byte records
    err, whole = _hashes(O, pay, 8, T, [(0, 0, 11, n)], 6)
    err2, head = _hashes(O, pay, 8, T, [(0, 0, 11, k * T)], 3)
    err3, tail = _hashes(O, pay, 8, T, [(k * T, 0, head[-1], n - k * T)], 3)
    assert err == err2 == err3 == 0
    assert whole == head + tail


def pin_hash_partial_last_page(O):
    """Positions past the end of a request are not part of its last page:
    growing the request inside its last page changes that page's hash only."""
    rng = np.random.default_rng(8)
    pay = rng.integers(0, 2**31, size=32, dtype=np.int32)
    _, short = _hashes(O, pay, 4, 8, [(0, 0, 0, 19)], 3)
    _, longer = _hashes(O, pay, 4, 8, [(0, 0, 0, 21)], 3)
    assert short[:2] == longer[:2] and short[2] != longer[2]
    # and the partial page's digest covers only its 3 positions
    c = O.fnv1a64(pay[16:19].tobytes())
    assert short[2] == O.fnv1a64(short[1].to_bytes(8, "little") + c.to_bytes(8, "little"))


def pin_hash_errors(O):
    pay = np.arange(40, dtype=np.int32)
    for row, bits in (((0, 0, 0, 40), 0), ((0, 0, 0, 41), ERR_BAD_REQ), ((-1, 0, 0, 4), ERR_BAD_REQ),
                      ((0, 4, 0, 40), ERR_BAD_REQ), ((0, -1, 0, 4), ERR_BAD_REQ),
                      ((0, 0, 0, -1), ERR_BAD_REQ), ((5, 0, 0, 0), 0)):
        out = np.full(5, 77, np.uint64)
        assert O.page_hashes(pay, 4, 10, [row], out) == bits, row
        if bits:
            assert (out == 77).all()


PINS = [pin_hand_example, pin_hand_example_plchtd, pin_numpy_transfer,
        pin_numpy_transfer_widths, pin_numpy_gather_scatter, pin_identity_tables,
        pin_roundtrip, pin_bijection, pin_errors, pin_max_position, pin_tiny_workload,
        pin_slice_hand_example, pin_slice_numpy, pin_slice_decomposes_transfer,
        pin_slice_tp_roundtrip, pin_slice_errors, pin_buffer_slice_numpy,
        pin_buffer_slice_full_and_parts, pin_buffer_slice_roundtrip, pin_buffer_slice_errors,
        pin_same_pool_copy_on_write,
        pin_fnv_published_vectors, pin_hash_definition, pin_hash_prefix_property,
        pin_hash_continuation, pin_hash_partial_last_page, pin_hash_errors]


def run_all(O) -> list:
    """Names of the pins that fail (an exception of any kind counts)."""
    failed = []
    for pin in PINS:
        try:
            pin(O)
        except Exception as exc:  # noqa: BLE001
            failed.append(f"{pin.__name__}: {type(exc).__name__}: {str(exc)[:200]}")
    return failed


if __name__ == "__main__":
    from oracle.kvx_oracle import Oracle
    failures = run_all(Oracle(sys.argv[1]))
    for f in failures:
        print("FAIL", f)
    sys.exit(1 if failures else 0)
