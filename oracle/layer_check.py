"""Per-layer checking of full-size runs against the CPU oracle.

TEST INFRASTRUCTURE ONLY (tests, smoke, the benchmark's CPU-baseline leg).
Layers never mix in the copy: layer l of the destination depends only on
layer l of the source.  A layer slice of any pool is itself a pool of the
same layout with one layer, and the layer-l part of each request's flat
block is itself a one-layer block.  So a run over pools of tens of GiB is
checked one layer at a time: copy the layer slices to the host, run the
oracle with one-layer shapes from the regenerated destination prefill, and
compare bytes.
"""
from __future__ import annotations

import dataclasses
import time

import numpy as np

from oracle import kvx_oracle
from paper_2606_31093_amd.workloads import BufSpec, prefill_words


def one_layer(spec):
    return dataclasses.replace(spec, L=1) if not isinstance(spec, BufSpec) else \
        dataclasses.replace(spec, L=1, cap=spec.cap // spec.L)


def layer_major(spec) -> bool:
    return spec.layout.startswith("L")


def pool_layer(t, spec, l: int) -> np.ndarray:
    """Host bytes of layer l of a pool held in torch uint8 tensor t."""
    per = spec.nbytes // spec.L
    if layer_major(spec):
        return t[l * per:(l + 1) * per].cpu().numpy()
    per_page = per // spec.N
    return t.view(spec.N, spec.L, per_page)[:, l, :].contiguous().cpu().numpy().reshape(-1)


def pool_layer_prefill(spec, l: int, tag: int) -> np.ndarray:
    """The offset-coded prefill of layer l of a pool (as ``fill_prefill_``
    wrote it over the whole pool)."""
    per = spec.nbytes // spec.L
    if layer_major(spec):
        g = np.arange(l * per // 8, (l + 1) * per // 8, dtype=np.uint64)
    else:
        per_page = per // spec.N
        g = ((np.arange(spec.N, dtype=np.uint64)[:, None] * spec.L + l) * (per_page // 8)
             + np.arange(per_page // 8, dtype=np.uint64)[None, :]).reshape(-1)
    return prefill_words(g, tag).view(np.uint8).copy()


def buf_layer(t, spec, l: int, blocks) -> tuple[np.ndarray, list]:
    """Layer l of every request block of a flat buffer, packed back to back.
    ``blocks`` lists (element offset, n_tokens) per request; returns the
    packed bytes and the one-layer block offsets (elements)."""
    per_tok = spec.C * spec.H * spec.D * spec.e
    parts, offs, pos = [], [], 0
    for off, n in blocks:
        start = off * spec.e + l * n * per_tok
        parts.append(t[start:start + n * per_tok].cpu().numpy())
        offs.append(pos // spec.e)
        pos += n * per_tok
    return (np.concatenate(parts) if parts else np.zeros(0, np.uint8)), offs


@dataclasses.dataclass
class LayerResult:
    layer: int
    equal: bool
    oracle_seconds: float
    moved_bytes: int      # algorithmic bytes (read + write) of this layer
    # runs the same oracle call again on the same host arrays (the copy is
    # idempotent), for timing several layers at once on several threads
    rerun: object = dataclasses.field(default=None, repr=False)


def check_transfer_layer(src_t, S, dst_t, D, step, l: int, tag: int,
                         dst_before: np.ndarray | None = None) -> LayerResult:
    """Run the oracle on layer l of a pool -> pool step and compare it with
    the device result.  The destination starts from its offset-coded
    prefill, or from ``dst_before`` (host bytes of the layer before the
    copy) when the step copies within one pool."""
    s1, d1 = one_layer(S), one_layer(D)
    got = pool_layer(dst_t, D, l)
    if dst_before is not None:
        want = dst_before.copy()
        src = dst_before if src_t is dst_t else pool_layer(src_t, S, l)
    else:
        want = pool_layer_prefill(D, l, tag)
        src = pool_layer(src_t, S, l)

    def run() -> int:
        return kvx_oracle.default().transfer(src, s1, want, d1, step.src_pt, step.dst_pt, step.reqs)

    t0 = time.perf_counter()
    err = run()
    dt = time.perf_counter() - t0
    moved = 2 * int(step.reqs[:, 5].sum()) * S.C * S.H * S.D * S.e
    return LayerResult(l, err == 0 and np.array_equal(got, want), dt, moved, run)


def check_transfer_slice_layer(src_t, S, dst_t, D, step, l: int, tag: int) -> LayerResult:
    """Layer l of a slice transfer (l counts from the slice's first layer):
    source layer src_layer0 + l lands in destination layer dst_layer0 + l."""
    sl = list(step.slice)
    ls, ld = sl[0] + l, sl[1] + l
    s1, d1 = one_layer(S), one_layer(D)
    src = pool_layer(src_t, S, ls)
    got = pool_layer(dst_t, D, ld)
    want = pool_layer_prefill(D, ld, tag)
    one = [0, 0, 1] + sl[3:]

    def run() -> int:
        return kvx_oracle.default().transfer_slice(src, s1, want, d1, one, step.src_pt,
                                                   step.dst_pt, step.reqs)

    t0 = time.perf_counter()
    err = run()
    dt = time.perf_counter() - t0
    moved = 2 * int(step.reqs[:, 5].sum()) * sl[5] * sl[8] * S.D * S.e
    return LayerResult(l, err == 0 and np.array_equal(got, want), dt, moved, run)


def gather_scatter_layer(pool_before: np.ndarray, S, buf_t, B, pool_after: np.ndarray,
                         gather, scatter, l: int) -> tuple[bool, bool]:
    """Layer l of a gather (pool -> flat buffer) followed by a scatter (flat
    buffer -> the same pool): the oracle gathers the layer from the pool as
    it was before, compares with the device buffer, scatters into a copy of
    the pool layer and compares with the device pool afterwards."""
    s1 = one_layer(S)
    blocks = [(int(r[2]), int(r[5])) for r in gather.reqs]
    got_buf, offs = buf_layer(buf_t, B, l, blocks)
    b1 = dataclasses.replace(B, L=1, cap=got_buf.nbytes // B.e)
    g_rows = gather.reqs.copy()
    g_rows[:, 2] = offs
    want_buf = np.zeros_like(got_buf)
    O = kvx_oracle.default()
    ok_g = O.gather(pool_before, s1, want_buf, b1, gather.src_pt, g_rows) == 0 and \
        np.array_equal(got_buf, want_buf)
    s_rows = scatter.reqs.copy()
    s_rows[:, 2] = offs
    want_pool = pool_before.copy()
    ok_s = O.scatter(want_buf, b1, want_pool, s1, scatter.dst_pt, s_rows) == 0 and \
        np.array_equal(pool_after, want_pool)
    return ok_g, ok_s


def gather_scatter_slice_layer(pool_before: np.ndarray, S, buf_t, B, pool_after: np.ndarray,
                               gather, scatter, l: int) -> tuple[bool, bool]:
    """Layer l of a sliced gather and scatter through a buffer that holds
    exactly the slice (l counts from the slice's first layer; the gather
    reads pool layer gather.slice[0] + l and the scatter writes pool layer
    scatter.slice[1] + l, which ``pool_before`` / ``pool_after`` hold)."""
    gs, ss = list(gather.slice), list(scatter.slice)
    s1 = one_layer(S)
    blocks = [(int(r[2]), int(r[5])) for r in gather.reqs]
    got_buf, offs = buf_layer(buf_t, B, l, blocks)
    b1 = dataclasses.replace(B, L=1, cap=got_buf.nbytes // B.e)
    g_rows = gather.reqs.copy()
    g_rows[:, 2] = offs
    want_buf = np.zeros_like(got_buf)
    O = kvx_oracle.default()
    ok_g = O.gather_slice(pool_before, s1, want_buf, b1, [0, 0, 1] + gs[3:], gather.src_pt,
                          g_rows) == 0 and np.array_equal(got_buf, want_buf)
    s_rows = scatter.reqs.copy()
    s_rows[:, 2] = offs
    want_pool = pool_before.copy()
    ok_s = O.scatter_slice(want_buf, b1, want_pool, s1, [0, 0, 1] + ss[3:], scatter.dst_pt,
                           s_rows) == 0 and np.array_equal(pool_after, want_pool)
    return ok_g, ok_s
