"""Seeded synthetic workloads for the paged KV-cache transfer path.

This module only *generates inputs*: pool and buffer shapes, request lengths,
page tables, request records, source values and destination prefill
patterns.  It holds none of the copy's arithmetic, and both the CPU oracle
(through the tests) and the HIP path consume what it produces.

Five workloads follow the shapes of the KV-cache movements Omni-Flow's Data
Flow layer performs (Sec. 4.1: role-to-role handoff through the Global Params
Pool, relayout between roles with different page sizes and layouts,
partial-prefix reuse as in Sec. 5.1's incremental matching, and L1 GPU <->
L2 CPU tier migration, Sec. 4.1.2):

  1. tiny gather-then-scatter (2 layers, 16-token pages -> flat -> 32-token pages)
  2. LLM role handoff (36 layers x 8 KV heads x 128, 64-token pages, 32 requests)
  3. heterogeneous relayout (28 x 4 x 128, 16-token LPCTHD -> 64-token PLCHTD)
  4. MLA latent cache (61 layers x 576, 64-token pages, copy of [p, len))
  5. host-tier offload then onload of a 16 GiB page subset (handoff shape)

Each has a ``small`` variant with the same layouts, page sizes and row widths
but fewer layers, heads, pages and tokens, for parity checks the oracle
finishes in seconds.

Request records are ``(n, 6)`` int64 arrays with columns
``src_pt_off, dst_pt_off, buf_off, src_start, dst_start, n_tokens``.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

LAYOUTS = ("LPCTHD", "LPCHTD", "PLCTHD", "PLCHTD")
REQ_COLUMNS = ("src_pt_off", "dst_pt_off", "buf_off", "src_start", "dst_start", "n_tokens")


@dataclass(frozen=True)
class PoolSpec:
    """A paged pool: L layers, C kv components (2 = K and V, 1 = MLA latent),
    H heads, D head_dim, T tokens per page, N pages, e bytes per element."""
    L: int
    C: int
    H: int
    D: int
    T: int
    N: int
    e: int = 2
    layout: str = "LPCTHD"

    @property
    def elems(self) -> int:
        return self.L * self.C * self.H * self.D * self.T * self.N

    @property
    def nbytes(self) -> int:
        return self.elems * self.e

    @property
    def token_bytes(self) -> int:
        """Bytes one token position occupies across all layers."""
        return self.L * self.C * self.H * self.D * self.e


@dataclass(frozen=True)
class BufSpec:
    """A flat buffer of per-request blocks [layer][kv][token][head][dim];
    ``cap`` is its size in elements."""
    L: int
    C: int
    H: int
    D: int
    e: int
    cap: int

    @property
    def nbytes(self) -> int:
        return self.cap * self.e

    @property
    def token_bytes(self) -> int:
        return self.L * self.C * self.H * self.D * self.e


@dataclass
class Step:
    op: str                      # "transfer" | "gather" | "scatter"
    src: str                     # name of the side read
    dst: str                     # name of the side written
    src_pt: np.ndarray | None    # int32 page table of a pool source
    dst_pt: np.ndarray | None    # int32 page table of a pool destination
    reqs: np.ndarray             # (n, 6) int64 request records
    slice: tuple | None = None   # transfer of a layer/kv/head range: nine fields
    layer_group: int = 0         # > 0: layer-pipelined, this many layers per group

    @property
    def n_tokens(self) -> int:
        return int(self.reqs[:, 5].sum()) if len(self.reqs) else 0


@dataclass
class Workload:
    name: str
    title: str
    sides: dict                  # name -> PoolSpec | BufSpec
    steps: list
    value_seed: int
    prefill_tag: int
    host_sides: tuple = ()       # sides that live in pinned host memory
    notes: dict = field(default_factory=dict)

    def algorithmic_bytes(self, step: Step) -> int:
        """Payload read plus payload written by one step: every copied token
        position moves its copied rows once in and once out."""
        if step.slice is not None:
            S = self.sides[step.src]
            nl, nc, nh = step.slice[2], step.slice[5], step.slice[8]
            return 2 * step.n_tokens * nl * nc * nh * S.D * S.e
        return 2 * step.n_tokens * self.sides[step.src].token_bytes


def _ceil_div(a: int, b: int) -> int:
    return -(-a // b)


def _reqs(rows) -> np.ndarray:
    a = np.asarray(rows, dtype=np.int64).reshape(-1, 6)
    return a


def _take_pages(perm: np.ndarray, counts) -> tuple[np.ndarray, list]:
    """Give request r the next counts[r] entries of a page permutation."""
    offs, pos = [], 0
    for c in counts:
        offs.append(pos)
        pos += int(c)
    if pos > len(perm):
        raise ValueError(f"workload needs {pos} pages, pool has {len(perm)}")
    return perm[:pos].astype(np.int32), offs


# --------------------------------------------------------------------------
# the five workloads
# --------------------------------------------------------------------------

def tiny() -> Workload:
    """2 layers, 2 KV heads, head_dim 64; a 100-token request on 7 random
    pages of a 64 x 16-token pool is gathered to a flat buffer, which is then
    scattered into a 32 x 32-token pool on 4 random pages."""
    rng = np.random.default_rng(1001)
    L, C, H, D, e = 2, 2, 2, 64, 2
    n = 100
    src = PoolSpec(L, C, H, D, T=16, N=64, e=e, layout="LPCTHD")
    dst = PoolSpec(L, C, H, D, T=32, N=32, e=e, layout="LPCTHD")
    buf = BufSpec(L, C, H, D, e, cap=L * C * n * H * D)
    src_pt = rng.permutation(src.N)[: _ceil_div(n, src.T)].astype(np.int32)
    dst_pt = rng.permutation(dst.N)[: _ceil_div(n, dst.T)].astype(np.int32)
    gather = Step("gather", "A", "buf", src_pt, None, _reqs([0, 0, 0, 0, 0, n]))
    scatter = Step("scatter", "buf", "B", None, dst_pt, _reqs([0, 0, 0, 0, 0, n]))
    return Workload("tiny", "tiny gather->flat->scatter, 2L x 2H x 64, 16->32-token pages",
                    {"A": src, "buf": buf, "B": dst}, [gather, scatter],
                    value_seed=2001, prefill_tag=1)


def _transfer_workload(name, seed_key, title, src: PoolSpec, dst: PoolSpec, lengths, starts,
                       rng, notes=None) -> Workload:
    """Requests hold positions [0, len); the copy moves [start, len) to the
    same positions.  Each side draws one permutation of its pages and gives
    request r the next ceil(len / T) of them."""
    lengths = [int(x) for x in lengths]
    starts = [int(x) for x in starts]
    src_perm = rng.permutation(src.N)
    dst_perm = rng.permutation(dst.N)
    src_pt, src_off = _take_pages(src_perm, [_ceil_div(n, src.T) for n in lengths])
    dst_pt, dst_off = _take_pages(dst_perm, [_ceil_div(n, dst.T) for n in lengths])
    rows = [[so, do, 0, p, p, n - p] for so, do, p, n in zip(src_off, dst_off, starts, lengths)]
    step = Step("transfer", "A", "B", src_pt, dst_pt, _reqs(rows))
    wl = Workload(name, title, {"A": src, "B": dst}, [step],
                  value_seed=2000 + seed_key, prefill_tag=seed_key, notes=notes or {})
    wl.notes.setdefault("lengths", lengths)
    wl.notes.setdefault("starts", starts)
    return wl


def handoff(small: bool = False) -> Workload:
    """LLM role handoff: 36 layers, 8 KV heads, head_dim 128, 4096 x 64-token
    pools on both sides, 32 requests with lengths uniform in [1024, 8192]."""
    if small:
        rng = np.random.default_rng(1102)
        L, H, N, nreq, lo, hi = 3, 2, 64, 4, 1, 700
    else:
        rng = np.random.default_rng(1002)
        L, H, N, nreq, lo, hi = 36, 8, 4096, 32, 1024, 8192
    pool = PoolSpec(L, 2, H, 128, T=64, N=N, e=2, layout="LPCTHD")
    lengths = rng.integers(lo, hi + 1, size=nreq)
    return _transfer_workload("handoff", 2, f"LLM role handoff {L}L x {H}H x 128, 64-token pages, "
                              f"{nreq} requests", pool, pool, lengths, [0] * nreq, rng)


def relayout(small: bool = False) -> Workload:
    """Heterogeneous-role relayout: 28 layers, 4 KV heads, head_dim 128;
    16-token LPCTHD pages into 64-token PLCHTD pages; 16 requests with
    lengths uniform in [2048, 16384]."""
    if small:
        rng = np.random.default_rng(1103)
        L, Ns, Nd, nreq, lo, hi = 3, 256, 64, 3, 50, 1000
    else:
        rng = np.random.default_rng(1003)
        L, Ns, Nd, nreq, lo, hi = 28, 16384, 4096, 16, 2048, 16384
    src = PoolSpec(L, 2, 4, 128, T=16, N=Ns, e=2, layout="LPCTHD")
    dst = PoolSpec(L, 2, 4, 128, T=64, N=Nd, e=2, layout="PLCHTD")
    lengths = rng.integers(lo, hi + 1, size=nreq)
    return _transfer_workload("relayout", 3, f"relayout {L}L x 4H x 128, 16-token LPCTHD -> 64-token "
                              f"PLCHTD, {nreq} requests", src, dst, lengths, [0] * nreq, rng)


def mla(small: bool = False) -> Workload:
    """MLA-style compressed KV: 61 layers, one 576-wide latent (C = 1, H = 1),
    64-token pages; 64 requests with lengths uniform in [4096, 32768]; only
    positions [p, len) are copied, p uniform in [0, len/2)."""
    if small:
        rng = np.random.default_rng(1104)
        L, nreq, lo, hi, align = 3, 4, 64, 1000, 16
    else:
        rng = np.random.default_rng(1004)
        L, nreq, lo, hi, align = 61, 64, 4096, 32768, 256
    lengths = rng.integers(lo, hi + 1, size=nreq)
    starts = [int(rng.integers(0, n // 2)) for n in lengths]
    pages = sum(_ceil_div(int(n), 64) for n in lengths)
    N = _ceil_div(pages, align) * align
    pool = PoolSpec(L, 1, 1, 576, T=64, N=N, e=2, layout="LPCTHD")
    return _transfer_workload("mla", 4, f"MLA latent {L}L x 576, 64-token pages, {nreq} requests, "
                              f"partial prefix [p, len)", pool, pool, lengths, starts, rng)


def host_tier(small: bool = False) -> Workload:
    """Host-tier offload/onload: the handoff pool; a 16 GiB subset of random
    pages (1820 pages = 28 requests x 65 full pages) is gathered into a
    pinned host buffer [request][layer][kv][token][head][dim] and scattered
    back into a fresh random sample of pool pages."""
    if small:
        rng = np.random.default_rng(1105)
        L, H, N, nreq, per = 3, 2, 64, 3, 4
    else:
        rng = np.random.default_rng(1005)
        L, H, N, nreq, per = 36, 8, 4096, 28, 65
    pool = PoolSpec(L, 2, H, 128, T=64, N=N, e=2, layout="LPCTHD")
    n = per * pool.T
    block = L * 2 * n * H * 128
    buf = BufSpec(L, 2, H, 128, 2, cap=nreq * block)
    out_pages = rng.choice(N, size=nreq * per, replace=False).astype(np.int32)
    in_pages = rng.choice(N, size=nreq * per, replace=False).astype(np.int32)
    g_rows = [[r * per, 0, r * block, 0, 0, n] for r in range(nreq)]
    s_rows = [[0, r * per, r * block, 0, 0, n] for r in range(nreq)]
    steps = [Step("gather", "A", "buf", out_pages, None, _reqs(g_rows)),
             Step("scatter", "buf", "A", None, in_pages, _reqs(s_rows))]
    return Workload("host_tier", f"host-tier offload/onload {L}L x {H}H x 128, {nreq * per} pages "
                    f"({nreq} x {per})", {"A": pool, "buf": buf}, steps,
                    value_seed=2005, prefill_tag=5, host_sides=("buf",))


def host_tier_v(small: bool = False) -> Workload:
    """The host-tier offload/onload of the same pages, V only (Sec. 4.1.3:
    K and V of a page may live on different nodes or tiers): the V half of
    each page is gathered into a pinned buffer that holds only V, then
    scattered into the V half of fresh pages."""
    wl = host_tier(small)
    g, s = wl.steps
    P, B = wl.sides["A"], wl.sides["buf"]
    n = int(g.reqs[0][5])
    block = P.L * 1 * n * P.H * P.D
    nreq = len(g.reqs)
    buf = BufSpec(P.L, 1, P.H, P.D, P.e, cap=nreq * block)
    g_rows = [[r[0], 0, i * block, 0, 0, n] for i, r in enumerate(g.reqs)]
    s_rows = [[0, r[1], i * block, 0, 0, n] for i, r in enumerate(s.reqs)]
    steps = [Step("gather", "A", "buf", g.src_pt, None, _reqs(g_rows),
                  slice=(0, 0, P.L, 1, 0, 1, 0, 0, P.H)),
             Step("scatter", "buf", "A", None, s.dst_pt, _reqs(s_rows),
                  slice=(0, 0, P.L, 0, 1, 1, 0, 0, P.H))]
    return Workload("host_tier_v", wl.title.replace("offload/onload", "V-only offload/onload"),
                    {"A": P, "buf": buf}, steps, value_seed=2015, prefill_tag=15,
                    host_sides=("buf",))


def tp_reshard(small: bool = False) -> Workload:
    """Tensor-parallel reshard of the handoff cache: a consumer running with
    two tensor-parallel ranks holds 4 of the 8 KV heads per pool; this moves
    heads [4, 8) of every layer of the 32 handoff requests into its 4-head
    pool (Sec. 7: transfers across tensor-parallel configurations; Sec. 4.1.1:
    views over slice tuples)."""
    if small:
        rng = np.random.default_rng(1106)
        L, H, N, nreq, lo, hi = 3, 4, 64, 4, 1, 700
    else:
        rng = np.random.default_rng(1006)
        L, H, N, nreq, lo, hi = 36, 8, 4096, 32, 1024, 8192
    src = PoolSpec(L, 2, H, 128, T=64, N=N, e=2, layout="LPCTHD")
    dst = PoolSpec(L, 2, H // 2, 128, T=64, N=N, e=2, layout="LPCTHD")
    lengths = rng.integers(lo, hi + 1, size=nreq)
    wl = _transfer_workload("tp_reshard", 6, f"TP reshard {L}L x heads [{H // 2}, {H}) of {H} x 128 "
                            f"-> {H // 2}-head pool, 64-token pages, {nreq} requests",
                            src, dst, lengths, [0] * nreq, rng)
    wl.steps[0].slice = (0, 0, L, 0, 0, 2, H // 2, 0, H // 2)
    return wl


def cow_fork(small: bool = False) -> Workload:
    """Copy-on-write inside one pool (Sec. 4.1.4): 16 requests of the handoff
    shape are forked, each copied page by page into fresh pages of the same
    pool (a fork duplicates shared pages before it appends).  Source and
    destination pages are disjoint, drawn from one permutation of the pool."""
    if small:
        rng = np.random.default_rng(1107)
        L, H, N, nreq, lo, hi = 3, 2, 64, 3, 1, 600
    else:
        rng = np.random.default_rng(1007)
        L, H, N, nreq, lo, hi = 36, 8, 4096, 16, 1024, 8192
    pool = PoolSpec(L, 2, H, 128, T=64, N=N, e=2, layout="LPCTHD")
    lengths = [int(x) for x in rng.integers(lo, hi + 1, size=nreq)]
    perm = rng.permutation(N).astype(np.int32)
    counts = [_ceil_div(n, pool.T) for n in lengths]
    total = sum(counts)
    if 2 * total > N:
        raise ValueError("pool too small for the fork")
    src_pt, offs = _take_pages(perm[:total], counts)
    dst_pt, _ = _take_pages(perm[total:2 * total], counts)
    rows = [[o, o, 0, 0, 0, n] for o, n in zip(offs, lengths)]
    step = Step("transfer", "A", "A", src_pt, dst_pt, _reqs(rows))
    return Workload("cow_fork", f"copy-on-write fork {L}L x {H}H x 128, {nreq} requests "
                    f"duplicated inside one 64-token pool", {"A": pool}, [step],
                    value_seed=2007, prefill_tag=7, notes={"lengths": lengths})


def handoff_layered(small: bool = False) -> Workload:
    """The handoff moved in groups of 4 layers, with a completion event per
    group, so a consumer can start on early layers while later ones move
    (Sec. 7: hierarchical transmission; Sec. 5.1: pipelined prefill)."""
    wl = handoff(small)
    wl.name = "handoff_layered"
    wl.title = wl.title + ", in 4-layer groups"
    wl.steps[0].layer_group = 1 if small else 4
    return wl


def small_requests(small: bool = False) -> Workload:
    """Many tiny requests at once, as when the newest tokens of every running
    sequence move after a decode step (Sec. 4.1.4: partial pages keep their
    other slots).  16384 requests (256 when small), each moving 1 to 4 tokens
    from a random slot range of a random source page into its own 4-slot
    group of a destination page; 16 groups per 64-token page, so no two
    requests write the same slot.  Pools as in the handoff."""
    if small:
        rng = np.random.default_rng(1112)
        L, H, N, nreq = 3, 2, 64, 256
    else:
        rng = np.random.default_rng(1012)
        L, H, N, nreq = 36, 8, 4096, 16384
    T, group = 64, 4
    pool = PoolSpec(L, 2, H, 128, T=T, N=N, e=2, layout="LPCTHD")
    n = rng.integers(1, group + 1, size=nreq)
    src_pt = rng.integers(0, N, size=nreq).astype(np.int32)
    s0 = np.array([rng.integers(0, T - k + 1) for k in n])
    slots = rng.permutation(N * (T // group))[:nreq]          # distinct (page, group) pairs
    dst_pt = (slots // (T // group)).astype(np.int32)
    d0 = (slots % (T // group)) * group
    rows = [[r, r, 0, int(s0[r]), int(d0[r]), int(n[r])] for r in range(nreq)]
    step = Step("transfer", "A", "B", src_pt, dst_pt, _reqs(rows))
    return Workload("small_requests", f"{nreq} small requests (1-{group} tokens each), "
                    f"{L}L x {H}H x 128, 64-token pages", {"A": pool, "B": pool}, [step],
                    value_seed=2012, prefill_tag=12)


NAMES = ("tiny", "handoff", "relayout", "mla", "host_tier", "tp_reshard", "cow_fork",
         "handoff_layered", "small_requests", "host_tier_v")


def get(name: str, small: bool = False) -> Workload:
    """A workload by name; ``small`` shrinks every one but ``tiny``."""
    if name == "tiny":
        return tiny()
    return {"handoff": handoff, "relayout": relayout, "mla": mla,
            "host_tier": host_tier, "tp_reshard": tp_reshard,
            "cow_fork": cow_fork, "handoff_layered": handoff_layered,
            "small_requests": small_requests, "host_tier_v": host_tier_v}[name](small=small)


# --------------------------------------------------------------------------
# values
# --------------------------------------------------------------------------

def normal_bf16_bytes(nbytes: int, seed: int) -> np.ndarray:
    """N(0,1) samples rounded to bf16 (nearest-even), as raw bytes (CPU)."""
    if nbytes % 2:
        raise ValueError("bf16 data needs an even byte count")
    x = np.random.default_rng(seed).standard_normal(nbytes // 2, dtype=np.float32)
    b = x.view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return b.astype(np.uint16).view(np.uint8)


def random_bytes(nbytes: int, seed: int) -> np.ndarray:
    return np.random.default_rng(seed).integers(0, 256, size=nbytes, dtype=np.uint8)


def prefill_words(groups: np.ndarray, tag: int) -> np.ndarray:
    """Offset-coded destination prefill: the 8-byte group with index g (byte
    offset 8g in its allocation) holds the little-endian word
    0x5A<<56 | tag<<48 | g, so any byte can be regenerated from its offset."""
    g = np.asarray(groups, dtype=np.uint64)
    w = (np.uint64(0x5A) << np.uint64(56)) | (np.uint64(tag & 0xFF) << np.uint64(48)) | g
    return w.astype("<u8")


def prefill_bytes(nbytes: int, tag: int, start_byte: int = 0) -> np.ndarray:
    """``prefill_words`` for the byte range [start_byte, start_byte + nbytes)."""
    if nbytes % 8 or start_byte % 8:
        raise ValueError("prefill covers whole 8-byte groups")
    g = np.arange(start_byte // 8, (start_byte + nbytes) // 8, dtype=np.uint64)
    return prefill_words(g, tag).view(np.uint8)


def fill_normal_bf16_(t, seed: int, chunk_elems: int = 1 << 28) -> None:
    """Fill a torch uint8 tensor (even size) with N(0,1) bf16 values drawn
    from a torch generator on the tensor's device."""
    import torch
    v = t.view(torch.bfloat16)
    g = torch.Generator(device=t.device)
    g.manual_seed(seed)
    for s in range(0, v.numel(), chunk_elems):
        e = min(v.numel(), s + chunk_elems)
        v[s:e].copy_(torch.randn(e - s, generator=g, device=t.device, dtype=torch.float32))


def fill_random_bytes_(t, seed: int, chunk: int = 1 << 30) -> None:
    import torch
    g = torch.Generator(device=t.device)
    g.manual_seed(seed)
    for s in range(0, t.numel(), chunk):
        e = min(t.numel(), s + chunk)
        t[s:e].copy_(torch.randint(0, 256, (e - s,), generator=g, device=t.device,
                                   dtype=torch.uint8))


def fill_prefill_(t, tag: int, chunk_groups: int = 1 << 27) -> None:
    """The offset-coded prefill of ``prefill_bytes`` written into a torch
    uint8 tensor on its own device."""
    import torch
    if t.numel() % 8:
        raise ValueError("prefill covers whole 8-byte groups")
    w = t.view(torch.int64)
    hi = (0x5A << 56) | ((tag & 0xFF) << 48)
    for s in range(0, w.numel(), chunk_groups):
        e = min(w.numel(), s + chunk_groups)
        w[s:e].copy_(torch.arange(s, e, device=t.device, dtype=torch.int64) | hi)


# --------------------------------------------------------------------------
# device placement (torch is used for memory only)
# --------------------------------------------------------------------------

def alloc_side(spec, device="cuda", pinned=False):
    """Bytes for one side: device memory, or pinned host memory."""
    import torch
    if pinned:
        return torch.empty(spec.nbytes, dtype=torch.uint8, pin_memory=True)
    return torch.empty(spec.nbytes, dtype=torch.uint8, device=device)


def value_side(wl: Workload) -> str:
    """The side that holds the source values (the first step's source)."""
    return wl.steps[0].src


def init_sides_(wl: Workload, tensors: dict) -> None:
    """Source values into the value side, offset-coded prefill elsewhere."""
    vs = value_side(wl)
    for name, t in tensors.items():
        spec = wl.sides[name]
        if name == vs:
            if spec.e == 2:
                fill_normal_bf16_(t, wl.value_seed)
            else:
                fill_random_bytes_(t, wl.value_seed)
        else:
            fill_prefill_(t, wl.prefill_tag)


# --------------------------------------------------------------------------
# chained page hashes (prefix matching, Sec. 5.1)
# --------------------------------------------------------------------------

@dataclass
class HashWorkload:
    name: str
    title: str
    rec_bytes: int               # bytes per position record (4: an int32 token id)
    T: int                       # positions per page
    positions: int               # records in the payload
    rows: list                   # (payload_off, out_off, seed, n_positions)
    out_len: int                 # hashes produced
    payload_seed: int

    def payload_bytes(self) -> int:
        return self.positions * self.rec_bytes


def page_hash(small: bool = False) -> HashWorkload:
    """Prefix-matching hashes over token ids: 4096 requests with lengths
    uniform in [1024, 8192] (64 in [1, 700] when small), 64-token pages,
    int32 token ids; every eighth request continues the chain of the one
    before it (seeded with a nonzero chain state), the rest start fresh."""
    rng = np.random.default_rng(1108 if small else 1008)
    nreq, lo, hi = (64, 1, 700) if small else (4096, 1024, 8192)
    T = 64
    lengths = rng.integers(lo, hi + 1, size=nreq)
    seeds = rng.integers(1, 2**63, size=nreq)
    rows, pos, out = [], 0, 0
    for r, n in enumerate(lengths):
        n = int(n)
        seed = int(seeds[r]) if r % 8 == 7 else 0
        rows.append((pos, out, seed, n))
        pos += n
        out += -(-n // T)
    return HashWorkload("page_hash", f"chained page hashes, {nreq} requests of int32 token ids, "
                        f"{T}-token pages", 4, T, pos, rows, out, payload_seed=2008)


def hash_payload(wl: HashWorkload) -> np.ndarray:
    """Token ids (uniform in [0, 2^17)) as int32 records."""
    return np.random.default_rng(wl.payload_seed).integers(
        0, 1 << 17, size=wl.positions * (wl.rec_bytes // 4), dtype=np.int32)
