"""Seeded small cases for parity checks: random page tables, shifted and
ragged ranges, shared source pages, every layout pair and page-size pair.

A case is a ``Workload`` (see paper_2606_31093_amd.workloads) so the same
runner drives the oracle and the HIP path.
"""
from __future__ import annotations

import itertools

import numpy as np

from paper_2606_31093_amd.workloads import LAYOUTS, BufSpec, PoolSpec, Step, Workload


def _cdiv(a, b):
    return -(-a // b)


def transfer_case(ls, ld, Ts, Td, seed, *, e=2, D=8, L=2, C=2, H=3, spec=None,
                  extra_pages=8) -> Workload:
    """Pool -> pool.  ``spec`` lists (src_start, dst_start, n, share) per
    request; share names an earlier request whose source pages it reuses."""
    rng = np.random.default_rng(seed)
    if spec is None:
        spec = [
            (Ts // 2 + 1, Td - 1, 3 * Ts + 1, None),   # both starts mid-page, ragged end
            (0, 1, 2 * Ts - 1, 0),                     # shares request 0's source pages
            (Ts - 1, 2 * Td - 1, 1, None),             # one token
            (0, 0, 0, None),                           # empty
            (0, 0, min(Td, 2 * Ts), None),             # page-aligned
        ]
    ks = [_cdiv(s0 + n, Ts) for s0, _d0, n, share in spec if share is None]
    kd = [_cdiv(d0 + n, Td) for _s0, d0, n, _share in spec]
    S = PoolSpec(L, C, H, D, T=Ts, N=sum(ks) + extra_pages, e=e, layout=ls)
    Dp = PoolSpec(L, C, H, D, T=Td, N=sum(kd) + extra_pages, e=e, layout=ld)
    sperm, dperm = rng.permutation(S.N).astype(np.int32), rng.permutation(Dp.N).astype(np.int32)
    src_pt, dst_pt, rows, src_offs = [], [], [], []
    for s0, d0, n, share in spec:
        k_s, k_d = _cdiv(s0 + n, Ts), _cdiv(d0 + n, Td)
        so = src_offs[share] if share is not None else len(src_pt)
        if share is None:
            src_pt.extend(sperm[len(src_pt): len(src_pt) + k_s])
        src_offs.append(so)
        rows.append([so, len(dst_pt), 0, s0, d0, n])
        dst_pt.extend(dperm[len(dst_pt): len(dst_pt) + k_d])
    step = Step("transfer", "A", "B", np.asarray(src_pt, np.int32), np.asarray(dst_pt, np.int32),
                np.asarray(rows, np.int64).reshape(-1, 6))
    return Workload("case", f"transfer {ls}/T{Ts} -> {ld}/T{Td} e{e} D{D} L{L} C{C} H{H}",
                    {"A": S, "B": Dp}, [step], value_seed=seed, prefill_tag=seed & 0xFF)


def gather_scatter_case(layout, T, e, D, seed, *, L=3, C=2, H=2, pinned=False) -> Workload:
    """Pool -> flat buffer -> a second pool of the same shape on other pages."""
    rng = np.random.default_rng(seed)
    ns = [5 * T // 2 + 1, 0, 1, 2 * T]
    starts = [T // 2 + 1, 0, T - 1, 0]
    align = 16 // e
    blocks, off = [], 0
    for n in ns:
        blocks.append(off)
        off += _cdiv(L * C * n * H * D, align) * align + align    # gaps between blocks
    B = BufSpec(L, C, H, D, e, cap=off)
    need = sum(_cdiv(s0 + n, T) for n, s0 in zip(ns, starts))
    S = PoolSpec(L, C, H, D, T=T, N=need + 5, e=e, layout=layout)
    perm = rng.permutation(S.N).astype(np.int32)
    pt, pos, g_rows = [], 0, []
    for n, s0, bo in zip(ns, starts, blocks):
        k = _cdiv(s0 + n, T)
        g_rows.append([pos, 0, bo, s0, 0, n])
        pt.extend(perm[pos: pos + k])
        pos += k
    s_rows = [[0, r[0], r[2], 0, r[3], r[5]] for r in g_rows]
    dperm = rng.permutation(S.N).astype(np.int32)[: len(pt)]
    steps = [Step("gather", "A", "buf", np.asarray(pt, np.int32), None, np.asarray(g_rows, np.int64)),
             Step("scatter", "buf", "B", None, dperm, np.asarray(s_rows, np.int64))]
    return Workload("case", f"gather/scatter {layout} T{T} e{e} D{D}", {"A": S, "buf": B, "B": S},
                    steps, value_seed=seed, prefill_tag=seed & 0xFF,
                    host_sides=("buf",) if pinned else ())


T_PAIRS = [(16, 64), (32, 8), (4, 4), (1, 16), (8, 1), (64, 64), (2, 128)]


def layout_matrix():
    """Every (source layout, destination layout, T_src, T_dst)."""
    for (ls, ld), (Ts, Td) in itertools.product(itertools.product(LAYOUTS, LAYOUTS), T_PAIRS):
        yield ls, ld, Ts, Td


def slice_case(ls, ld, Ts, Td, S_LCH, D_LCH, sl, seed, *, D=8, e=2) -> Workload:
    """Slice of one pool into another of a different layer/kv/head count."""
    rng = np.random.default_rng(seed)
    (Ls, Cs, Hs), (Ld, Cd, Hd) = S_LCH, D_LCH
    spec = [(Ts // 2 + 1, Td - 1, 3 * Ts + 1), (0, 1, 2 * Ts - 1), (Ts - 1, 0, 1), (0, 0, 0)]
    ks = [_cdiv(s0 + n, Ts) for s0, _, n in spec]
    kd = [_cdiv(d0 + n, Td) for _, d0, n in spec]
    S = PoolSpec(Ls, Cs, Hs, D, T=Ts, N=sum(ks) + 3, e=e, layout=ls)
    Dp = PoolSpec(Ld, Cd, Hd, D, T=Td, N=sum(kd) + 3, e=e, layout=ld)
    sperm, dperm = rng.permutation(S.N).astype(np.int32), rng.permutation(Dp.N).astype(np.int32)
    rows, so, do = [], 0, 0
    for (s0, d0, n), a, b in zip(spec, ks, kd):
        rows.append([so, do, 0, s0, d0, n])
        so, do = so + a, do + b
    step = Step("transfer", "A", "B", sperm[:so], dperm[:do], np.asarray(rows, np.int64),
                slice=tuple(sl))
    return Workload("case", f"slice {sl} {ls}/T{Ts} {S_LCH} -> {ld}/T{Td} {D_LCH}",
                    {"A": S, "B": Dp}, [step], value_seed=seed, prefill_tag=seed & 0xFF)


SLICES = [((4, 2, 8), (2, 2, 4), (2, 0, 2, 0, 0, 2, 4, 0, 4)),     # TP=2 shard of a layer stage
          ((3, 2, 4), (3, 1, 4), (0, 0, 3, 1, 0, 1, 0, 0, 4)),     # V only
          ((3, 2, 4), (3, 1, 4), (0, 0, 3, 0, 0, 1, 0, 0, 4)),     # K only
          ((3, 2, 4), (5, 2, 6), (0, 2, 3, 0, 0, 2, 1, 3, 2)),     # into a larger pool
          ((2, 1, 1), (2, 1, 3), (0, 0, 2, 0, 0, 1, 0, 2, 1)),     # one head into head 2
          ((2, 2, 4), (2, 2, 4), (0, 0, 2, 0, 0, 2, 0, 0, 4)),     # everything
          ((2, 2, 8), (2, 2, 8), (1, 0, 1, 1, 0, 1, 3, 5, 1))]     # one row per token


def random_case(seed: int) -> Workload:
    """A seeded random pool -> pool case: layouts, page sizes (powers of two
    and not), shapes, element widths, 1-6 requests with random starts and
    lengths (some empty, some rereading an earlier request's source pages),
    sometimes a slice with its own layer/kv/head ranges, and sometimes one
    damaged page-table entry or a truncated table.  Destinations never
    overlap, so the result is defined even with the damage."""
    rng = np.random.default_rng(10_000 + seed)
    pick = lambda xs: xs[int(rng.integers(len(xs)))]
    ls, ld = pick(LAYOUTS), pick(LAYOUTS)
    Ts, Td = pick([1, 2, 3, 4, 5, 8, 16, 32, 64]), pick([1, 2, 3, 4, 6, 8, 16, 32, 64])
    e = pick([1, 2, 4, 8])
    D = (16 // e) * pick([1, 2, 3, 5])
    sliced = rng.random() < 0.3
    if sliced:
        Ls, Ld = int(rng.integers(1, 4)), int(rng.integers(1, 4))
        Cs, Cd = int(rng.integers(1, 3)), int(rng.integers(1, 3))
        Hs, Hd = pick([1, 2, 3, 5]), pick([1, 2, 3, 5])
        ranges = []
        for a, b in ((Ls, Ld), (Cs, Cd), (Hs, Hd)):
            n = int(rng.integers(0 if rng.random() < 0.1 else 1, min(a, b) + 1))
            ranges.append((int(rng.integers(0, a - n + 1)), int(rng.integers(0, b - n + 1)), n))
        sl = tuple(x for r in ranges for x in r)
    else:
        Ls = Ld = int(rng.integers(1, 4))
        Cs = Cd = int(rng.integers(1, 3))
        Hs = Hd = pick([1, 2, 3, 5])
        sl = None
    spec = []
    for r in range(int(rng.integers(1, 7))):
        n = 0 if rng.random() < 0.1 else int(rng.integers(1, 3 * max(Ts, Td) + 6))
        share = int(rng.integers(0, r)) if r and rng.random() < 0.2 else None
        spec.append((int(rng.integers(0, 2 * Ts)), int(rng.integers(0, 2 * Td)), n, share))
    ks = [_cdiv(s0 + n, Ts) for s0, _d0, n, share in spec if share is None]
    kd = [_cdiv(d0 + n, Td) for _s0, d0, n, _share in spec]
    S = PoolSpec(Ls, Cs, Hs, D, T=Ts, N=sum(ks) + 2, e=e, layout=ls)
    Dp = PoolSpec(Ld, Cd, Hd, D, T=Td, N=sum(kd) + 2, e=e, layout=ld)
    sperm, dperm = rng.permutation(S.N).astype(np.int32), rng.permutation(Dp.N).astype(np.int32)
    src_pt, dst_pt, rows, src_offs = [], [], [], []
    for s0, d0, n, share in spec:
        k_s, k_d = _cdiv(s0 + n, Ts), _cdiv(d0 + n, Td)
        so = src_offs[share] if share is not None else len(src_pt)
        if share is None:
            src_pt.extend(sperm[len(src_pt): len(src_pt) + k_s])
        src_offs.append(so)
        rows.append([so, len(dst_pt), 0, s0, d0, n])
        dst_pt.extend(dperm[len(dst_pt): len(dst_pt) + k_d])
    src_pt, dst_pt = np.asarray(src_pt, np.int32), np.asarray(dst_pt, np.int32)
    damage = rng.random()
    if damage < 0.08 and len(dst_pt):
        dst_pt[int(rng.integers(len(dst_pt)))] = pick([-1, Dp.N, 2**31 - 1])
    elif damage < 0.16 and len(src_pt):
        src_pt[int(rng.integers(len(src_pt)))] = pick([-1, S.N])
    elif damage < 0.22 and len(src_pt) > 1:
        src_pt = src_pt[: int(rng.integers(1, len(src_pt)))]
    step = Step("transfer", "A", "B", src_pt, dst_pt, np.asarray(rows, np.int64).reshape(-1, 6),
                slice=sl)
    return Workload("case", f"random {seed}: {ls}/T{Ts} ({Ls},{Cs},{Hs}) -> {ld}/T{Td} "
                    f"({Ld},{Cd},{Hd}) e{e} D{D} slice={sl}",
                    {"A": S, "B": Dp}, [step], value_seed=seed, prefill_tag=seed & 0xFF)


RANDOM_CASES = 200


def random_medium_case(seed: int) -> Workload:
    """A seeded random transfer of medium size: 100-900 requests (several
    256-record chunks of the kernel's record scan, many tiles per
    workgroup), random layouts and page sizes on each side, requests that
    reread earlier source pages, and sometimes a damaged destination id."""
    rng = np.random.default_rng(90_000 + seed)
    pick = lambda xs: xs[int(rng.integers(len(xs)))]
    ls, ld = pick(LAYOUTS), pick(LAYOUTS)
    Ts, Td = pick([1, 4, 8, 16, 64, 128]), pick([2, 8, 16, 32, 64, 256])
    e = pick([2, 4])
    D = (16 // e) * pick([2, 4, 8])
    L, C, H = int(rng.integers(1, 5)), int(rng.integers(1, 3)), pick([1, 2, 4])
    nreq = int(rng.integers(100, 900))
    spec = []
    for r in range(nreq):
        n = 0 if rng.random() < 0.05 else int(rng.integers(1, 3 * max(Ts, Td) + 40))
        share = int(rng.integers(0, r)) if r and rng.random() < 0.1 else None
        spec.append((int(rng.integers(0, 2 * Ts)), int(rng.integers(0, 2 * Td)), n, share))
    ks = [_cdiv(s0 + n, Ts) for s0, _d0, n, share in spec if share is None]
    kd = [_cdiv(d0 + n, Td) for _s0, d0, n, _share in spec]
    S = PoolSpec(L, C, H, D, T=Ts, N=sum(ks) + 3, e=e, layout=ls)
    Dp = PoolSpec(L, C, H, D, T=Td, N=sum(kd) + 3, e=e, layout=ld)
    sperm, dperm = rng.permutation(S.N).astype(np.int32), rng.permutation(Dp.N).astype(np.int32)
    src_pt, dst_pt, rows, src_offs = [], [], [], []
    for s0, d0, n, share in spec:
        k_s, k_d = _cdiv(s0 + n, Ts), _cdiv(d0 + n, Td)
        so = src_offs[share] if share is not None else len(src_pt)
        if share is None:
            src_pt.extend(sperm[len(src_pt): len(src_pt) + k_s])
        src_offs.append(so)
        rows.append([so, len(dst_pt), 0, s0, d0, n])
        dst_pt.extend(dperm[len(dst_pt): len(dst_pt) + k_d])
    src_pt, dst_pt = np.asarray(src_pt, np.int32), np.asarray(dst_pt, np.int32)
    if rng.random() < 0.2 and len(dst_pt):
        dst_pt[int(rng.integers(len(dst_pt)))] = -1
    step = Step("transfer", "A", "B", src_pt, dst_pt, np.asarray(rows, np.int64).reshape(-1, 6))
    return Workload("case", f"medium {seed}: {ls}/T{Ts} -> {ld}/T{Td} ({L},{C},{H}) e{e} D{D}, "
                    f"{nreq} requests", {"A": S, "B": Dp}, [step], value_seed=seed,
                    prefill_tag=seed & 0xFF)


RANDOM_MEDIUM_CASES = 24


def random_gs_case(seed: int) -> Workload:
    """A seeded random gather (pool -> flat buffer) and scatter (buffer ->
    a second pool): random layout, page size, shape and element width, 1-5
    requests at random source / destination starts, blocks at random aligned
    offsets with gaps, the buffer in device or pinned host memory, and
    sometimes a damaged record (a block that is misaligned or runs past the
    buffer, a nonzero buffer-side start) or a damaged page id."""
    rng = np.random.default_rng(20_000 + seed)
    pick = lambda xs: xs[int(rng.integers(len(xs)))]
    layout, T = pick(LAYOUTS), pick([1, 2, 3, 4, 8, 16, 64])
    e = pick([1, 2, 4, 8])
    D = (16 // e) * pick([1, 2, 3])
    L, C, H = int(rng.integers(1, 4)), int(rng.integers(1, 3)), pick([1, 2, 3])
    # sometimes a slice: the buffer holds (nl, nc, nh) of the pool's
    # (L, C, H), gathered at one offset and scattered at another of a second
    # pool of another shape
    sliced = rng.random() < 0.3
    if sliced:
        L2, C2, H2 = int(rng.integers(1, 4)), int(rng.integers(1, 3)), pick([1, 2, 3, 5])
        nl = int(rng.integers(1, min(L, L2) + 1))
        nc = int(rng.integers(1, min(C, C2) + 1))
        nh = int(rng.integers(1, min(H, H2) + 1))
        g_off = [int(rng.integers(0, x - n + 1)) for x, n in ((L, nl), (C, nc), (H, nh))]
        s_off = [int(rng.integers(0, x - n + 1)) for x, n in ((L2, nl), (C2, nc), (H2, nh))]
    else:
        (L2, C2, H2), (nl, nc, nh) = (L, C, H), (L, C, H)
    align = 16 // e
    ns = [0 if rng.random() < 0.1 else int(rng.integers(1, 3 * T + 6))
          for _ in range(int(rng.integers(1, 6)))]
    starts = [int(rng.integers(0, 2 * T)) for _ in ns]
    dstarts = [int(rng.integers(0, 2 * T)) for _ in ns]
    blocks, off = [], int(rng.integers(0, 3)) * align
    for n in ns:
        blocks.append(off)
        off += _cdiv(nl * nc * n * nh * D, align) * align + int(rng.integers(0, 3)) * align
    B = BufSpec(nl, nc, nh, D, e, cap=off)
    S = PoolSpec(L, C, H, D, T=T, N=sum(_cdiv(s + n, T) for n, s in zip(ns, starts)) + 2, e=e,
                 layout=layout)
    P2 = PoolSpec(L2, C2, H2, D, T=T, N=sum(_cdiv(s + n, T) for n, s in zip(ns, dstarts)) + 2,
                  e=e, layout=pick(LAYOUTS) if sliced else layout)
    perm, dperm = rng.permutation(S.N).astype(np.int32), rng.permutation(P2.N).astype(np.int32)
    g_rows, s_rows, pt, dpt = [], [], [], []
    for n, s0, d0, bo in zip(ns, starts, dstarts, blocks):
        g_rows.append([len(pt), 0, bo, s0, 0, n])
        s_rows.append([0, len(dpt), bo, 0, d0, n])
        pt.extend(perm[len(pt): len(pt) + _cdiv(s0 + n, T)])
        dpt.extend(dperm[len(dpt): len(dpt) + _cdiv(d0 + n, T)])
    g_rows, s_rows = np.asarray(g_rows, np.int64), np.asarray(s_rows, np.int64)
    pt, dpt = np.asarray(pt, np.int32), np.asarray(dpt, np.int32)
    damage, r = rng.random(), int(rng.integers(len(ns)))
    if damage < 0.05 and e < 8:
        g_rows[r, 2] += 1                      # block not 16-byte aligned
    elif damage < 0.10:
        s_rows[r, 2] = off                     # block runs past the buffer (if n > 0)
    elif damage < 0.14:
        g_rows[r, 4] = 1                       # buffer-side start must be 0
    elif damage < 0.20 and len(pt):
        pt[int(rng.integers(len(pt)))] = S.N
    elif damage < 0.26 and len(dpt):
        dpt[int(rng.integers(len(dpt)))] = -1
    gsl = (g_off[0], 0, nl, g_off[1], 0, nc, g_off[2], 0, nh) if sliced else None
    ssl = (0, s_off[0], nl, 0, s_off[1], nc, 0, s_off[2], nh) if sliced else None
    steps = [Step("gather", "A", "buf", pt, None, g_rows, slice=gsl),
             Step("scatter", "buf", "B", None, dpt, s_rows, slice=ssl)]
    return Workload("case", f"random gather/scatter {seed}: {layout}/T{T} ({L},{C},{H}) e{e} D{D} "
                    f"slices {gsl} {ssl}",
                    {"A": S, "buf": B, "B": P2}, steps, value_seed=seed, prefill_tag=seed & 0xFF,
                    host_sides=("buf",) if rng.random() < 0.3 else ())


RANDOM_GS_CASES = 100


def buffer_slice_case(ls, ld, T, src_lch, dst_lch, gsl, dst_off, seed, *, pinned=False,
                      D=64, e=2) -> Workload:
    """A slice of pool A gathered into a buffer that holds exactly the slice,
    then scattered into a slice of pool B (another shape and layout) at
    ``dst_off`` = (layer0, kv0, head0).  ``gsl`` is the gather's nine-field
    slice (its buffer-side offsets 0)."""
    rng = np.random.default_rng(seed)
    (Ls, Cs, Hs), (Ld, Cd, Hd) = src_lch, dst_lch
    nl, nc, nh = gsl[2], gsl[5], gsl[8]
    align = 16 // e
    ns, starts, dstarts = [3 * T + 2, 1, 0, 2 * T], [T // 2 + 1, T - 1, 0, 0], [1, 0, 3, T]
    blocks, off = [], align
    for n in ns:
        blocks.append(off)
        off += _cdiv(nl * nc * n * nh * D, align) * align + align
    B = BufSpec(nl, nc, nh, D, e, cap=off)
    S = PoolSpec(Ls, Cs, Hs, D, T=T, N=sum(_cdiv(s + n, T) for n, s in zip(ns, starts)) + 2, e=e,
                 layout=ls)
    Dp = PoolSpec(Ld, Cd, Hd, D, T=T, N=sum(_cdiv(s + n, T) for n, s in zip(ns, dstarts)) + 2,
                  e=e, layout=ld)
    perm, dperm = rng.permutation(S.N).astype(np.int32), rng.permutation(Dp.N).astype(np.int32)
    g_rows, s_rows, pt, dpt = [], [], [], []
    for n, s0, d0, bo in zip(ns, starts, dstarts, blocks):
        g_rows.append([len(pt), 0, bo, s0, 0, n])
        s_rows.append([0, len(dpt), bo, 0, d0, n])
        pt.extend(perm[len(pt): len(pt) + _cdiv(s0 + n, T)])
        dpt.extend(dperm[len(dpt): len(dpt) + _cdiv(d0 + n, T)])
    ssl = (0, dst_off[0], nl, 0, dst_off[1], nc, 0, dst_off[2], nh)
    steps = [Step("gather", "A", "buf", np.asarray(pt, np.int32), None,
                  np.asarray(g_rows, np.int64), slice=tuple(gsl)),
             Step("scatter", "buf", "B", None, np.asarray(dpt, np.int32),
                  np.asarray(s_rows, np.int64), slice=ssl)]
    return Workload("case", f"buffer slice {gsl} {ls} {src_lch} -> {ld} {dst_lch} at {dst_off}",
                    {"A": S, "buf": B, "B": Dp}, steps, value_seed=seed, prefill_tag=seed & 0xFF,
                    host_sides=("buf",) if pinned else ())


# (source L, C, H), (destination L, C, H), gather slice, destination offsets
BUFFER_SLICES = [((3, 2, 4), (3, 2, 4), (0, 0, 3, 0, 0, 2, 0, 0, 4), (0, 0, 0)),   # whole pool
                 ((3, 2, 4), (3, 1, 4), (0, 0, 3, 1, 0, 1, 0, 0, 4), (0, 0, 0)),   # V only
                 ((3, 2, 4), (3, 2, 4), (0, 0, 3, 0, 0, 1, 0, 0, 4), (0, 1, 0)),   # K into V
                 ((4, 2, 8), (2, 2, 4), (2, 0, 2, 0, 0, 2, 4, 0, 4), (0, 0, 0)),   # TP shard of a stage
                 ((2, 1, 3), (3, 1, 5), (0, 0, 2, 0, 0, 1, 1, 0, 2), (1, 0, 3)),   # into a larger pool
                 ((2, 2, 2), (2, 2, 2), (1, 0, 1, 1, 0, 1, 1, 0, 1), (0, 0, 0))]   # one row per token


def random_cow_case(seed: int) -> Workload:
    """A seeded random copy inside one pool (copy-on-write, Sec. 4.1.4):
    requests read pages of a shared prefix and write fresh pages of the same
    pool; no page is both read and written, so the result is defined."""
    rng = np.random.default_rng(40_000 + seed)
    pick = lambda xs: xs[int(rng.integers(len(xs)))]
    layout, T = pick(LAYOUTS), pick([1, 2, 4, 5, 8, 16])
    e = pick([1, 2, 4])
    D = (16 // e) * pick([1, 2])
    L, C, H = int(rng.integers(1, 4)), int(rng.integers(1, 3)), pick([1, 2, 3])
    spec = [(int(rng.integers(0, 2 * T)), int(rng.integers(0, 2 * T)),
             int(rng.integers(0, 3 * T + 4))) for _ in range(int(rng.integers(1, 5)))]
    k_read = sum(_cdiv(s0 + n, T) for s0, _d0, n in spec)
    k_write = sum(_cdiv(d0 + n, T) for _s0, d0, n in spec)
    P = PoolSpec(L, C, H, D, T=T, N=k_read + k_write + 3, e=e, layout=layout)
    perm = rng.permutation(P.N).astype(np.int32)
    reads, writes = perm[:k_read], perm[k_read:k_read + k_write]
    src_pt, dst_pt, rows = [], [], []
    for s0, d0, n in spec:
        rows.append([len(src_pt), len(dst_pt), 0, s0, d0, n])
        src_pt.extend(reads[len(src_pt): len(src_pt) + _cdiv(s0 + n, T)])
        dst_pt.extend(writes[len(dst_pt): len(dst_pt) + _cdiv(d0 + n, T)])
    step = Step("transfer", "A", "A", np.asarray(src_pt, np.int32), np.asarray(dst_pt, np.int32),
                np.asarray(rows, np.int64).reshape(-1, 6))
    return Workload("case", f"random copy-on-write {seed}: {layout}/T{T} ({L},{C},{H}) e{e} D{D}",
                    {"A": P}, [step], value_seed=seed, prefill_tag=seed & 0xFF)


def random_layered_case(seed: int) -> Workload:
    """A seeded random transfer (``random_case``) moved in random layer groups."""
    wl = random_case(1000 + seed)
    st = wl.steps[0]
    n_layers = st.slice[2] if st.slice is not None else wl.sides["A"].L
    st.layer_group = int(np.random.default_rng(50_000 + seed).integers(1, max(1, n_layers) + 2))
    wl.title += f", layer groups of {st.layer_group}"
    return wl


RANDOM_COW_CASES = 40
RANDOM_LAYERED_CASES = 40


def random_planned_medium_case(seed: int) -> Workload:
    """A seeded medium transfer whose token-major destination pages hold 128
    or 256 KiB (so a planned call sweeps in the product library too): 8-39
    requests of up to 399 tokens, any source layout, 16-64-token source
    pages, some requests reading an earlier request's source pages."""
    rng = np.random.default_rng(90_000 + seed)
    pick = lambda xs: xs[int(rng.integers(len(xs)))]
    ls, ld = pick(["LPCTHD", "LPCHTD", "PLCTHD", "PLCHTD"]), pick(["LPCTHD", "PLCTHD"])
    Ts, Td = pick([16, 32, 64]), 64
    spec = []
    for r in range(int(rng.integers(8, 40))):
        n = 0 if rng.random() < 0.05 else int(rng.integers(1, 400))
        share = int(rng.integers(0, r)) if r > 0 and rng.random() < 0.1 else None
        s0 = int(rng.integers(0, 2 * Ts)) if share is None else 0
        d0 = int(rng.integers(0, 2 * Td))
        if share is not None:                    # stay inside the pages it reads
            n = min(n, spec[share][0] + spec[share][2])
        spec.append((s0, d0, n, share))
    return transfer_case(ls, ld, Ts, Td, seed=90_000 + seed, e=2, D=128, L=int(rng.integers(1, 4)), C=2,
                         H=pick([4, 8]), spec=spec)
