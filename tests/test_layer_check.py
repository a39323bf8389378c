"""oracle/layer_check.py, the per-layer checker behind every full-size parity
test and the benchmark's bit-exact flag, checked on the CPU.

Each case runs a whole small workload through the oracle, then checks the
result layer by layer with layer_check on CPU torch tensors, exactly as the
full-size GPU tests check device results.  Every layer must agree: a slip in
the layer slicing (a wrong per-page stride for a page-major layout, a wrong
block offset in a flat buffer, a prefill regenerated at the wrong offsets)
would make some layer differ here.  Planted mistakes in layer_check's
helpers must each make some layer fail.
"""
import dataclasses

import numpy as np
import pytest

import cases
from oracle import layer_check
from paper_2606_31093_amd.workloads import LAYOUTS, get, prefill_words
from runner import initial_bytes, run_oracle

torch = pytest.importorskip("torch")


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a))


def layer_results(wl):
    """Per-layer verdicts of layer_check on the whole-workload oracle result
    of ``wl``: a list of (step index, layer, equal)."""
    init = initial_bytes(wl)
    final, errs = run_oracle(wl, init)
    assert not any(errs), f"{wl.title}: oracle error bits {errs}"
    out = []
    steps = wl.steps
    if len(steps) == 1 and steps[0].op == "transfer":
        st = steps[0]
        S, D = wl.sides[st.src], wl.sides[st.dst]
        if st.src == st.dst:                   # copy inside one pool
            pool0, pool1 = _t(init[st.src]), _t(final[st.src])
            for l in range(S.L):
                before = layer_check.pool_layer(pool0, S, l)
                r = layer_check.check_transfer_layer(pool1, S, pool1, D, st, l, wl.prefill_tag,
                                                     before)
                out.append((0, l, r.equal))
            return out
        src_t, dst_t = _t(final[st.src]), _t(final[st.dst])
        n_layers = st.slice[2] if st.slice is not None else S.L
        for l in range(n_layers):
            if st.slice is not None:
                r = layer_check.check_transfer_slice_layer(src_t, S, dst_t, D, st, l,
                                                           wl.prefill_tag)
            else:
                r = layer_check.check_transfer_layer(src_t, S, dst_t, D, st, l, wl.prefill_tag)
            out.append((0, l, r.equal))
        return out
    # gather into a flat buffer, then scatter into a pool
    g, s = steps
    assert g.op == "gather" and s.op == "scatter"
    S, B = wl.sides[g.src], wl.sides[g.dst]
    P2 = wl.sides[s.dst]
    pool0, buf_t = _t(init[g.src]), _t(final[g.dst])
    after_t = _t(final[s.dst])
    before_t = pool0 if s.dst == g.src else _t(init[s.dst])
    n_layers = g.slice[2] if g.slice is not None else S.L
    for l in range(n_layers):
        if g.slice is not None:
            lg, ls = g.slice[0] + l, s.slice[1] + l
            ok_g, ok_s = layer_check.gather_scatter_slice_layer(
                layer_check.pool_layer(pool0, S, lg), S, buf_t, B,
                layer_check.pool_layer(after_t, P2, ls), g, s, l)
        else:
            before = layer_check.pool_layer(before_t, P2, l)
            src_l = layer_check.pool_layer(pool0, S, l)
            if s.dst == g.src:
                ok_g, ok_s = layer_check.gather_scatter_layer(
                    before, S, buf_t, B, layer_check.pool_layer(after_t, P2, l), g, s, l)
            else:
                ok_g, ok_s = _gather_scatter_two_pools(src_l, S, buf_t, B, before, P2,
                                                       layer_check.pool_layer(after_t, P2, l),
                                                       g, s, l)
        out.append((0, l, ok_g))
        out.append((1, l, ok_s))
    return out


def _gather_scatter_two_pools(src_l, S, buf_t, B, dst_before, P2, dst_after, g, s, l):
    """A gather from one pool and a scatter into another (the tiny workload's
    shape), through layer_check's buffer slicing."""
    from oracle import kvx_oracle
    blocks = [(int(r[2]), int(r[5])) for r in g.reqs]
    got_buf, offs = layer_check.buf_layer(buf_t, B, l, blocks)
    b1 = dataclasses.replace(B, L=1, cap=got_buf.nbytes // B.e)
    g_rows = g.reqs.copy()
    g_rows[:, 2] = offs
    want_buf = np.zeros_like(got_buf)
    O = kvx_oracle.default()
    ok_g = O.gather(src_l, layer_check.one_layer(S), want_buf, b1, g.src_pt, g_rows) == 0 and \
        np.array_equal(got_buf, want_buf)
    s_rows = s.reqs.copy()
    s_rows[:, 2] = offs
    want = dst_before.copy()
    ok_s = O.scatter(want_buf, b1, want, layer_check.one_layer(P2), s.dst_pt, s_rows) == 0 and \
        np.array_equal(dst_after, want)
    return ok_g, ok_s


SMALL = ["tiny", "handoff", "relayout", "mla", "host_tier", "tp_reshard", "cow_fork",
         "small_requests", "host_tier_v"]


def _small(name):
    return get(name) if name == "tiny" else get(name, small=True)


@pytest.mark.parametrize("name", SMALL)
def test_every_layer_of_small_workloads(name):
    res = layer_results(_small(name))
    assert res and all(ok for _, _, ok in res), [r for r in res if not r[2]]


@pytest.mark.parametrize("ld", LAYOUTS)
@pytest.mark.parametrize("ls", LAYOUTS)
def test_every_layer_of_layout_pairs(ls, ld):
    """Every layout pair (page-major destinations included), three layers,
    pages of different sizes on the two sides."""
    wl = cases.transfer_case(ls, ld, 4, 8, seed=77, L=3)
    res = layer_results(wl)
    assert len(res) == 3 and all(ok for _, _, ok in res)


@pytest.mark.parametrize("k", range(len(cases.SLICES)))
@pytest.mark.parametrize("ls,ld", [("LPCTHD", "PLCHTD"), ("PLCTHD", "LPCHTD")])
def test_every_layer_of_slices(k, ls, ld):
    S_LCH, D_LCH, sl = cases.SLICES[k]
    res = layer_results(cases.slice_case(ls, ld, 4, 8, S_LCH, D_LCH, sl, seed=90 + k))
    assert res and all(ok for _, _, ok in res)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_every_layer_of_gather_buffers(layout):
    res = layer_results(cases.gather_scatter_case(layout, 8, 2, 16, seed=5))
    assert len(res) == 6 and all(ok for _, _, ok in res)


# --------------------------------------------------------------------------
# planted mistakes: each must make some layer of the sweep below fail
# --------------------------------------------------------------------------

def _pool_layer_as_layer_major(t, spec, l):
    per = spec.nbytes // spec.L
    return t[l * per:(l + 1) * per].cpu().numpy()


def _pool_layer_wrong_page_stride(t, spec, l):
    per = spec.nbytes // spec.L
    if layer_check.layer_major(spec):
        return t[l * per:(l + 1) * per].cpu().numpy()
    per_page = per // spec.N
    return t.view(spec.L, spec.N, per_page)[l].contiguous().cpu().numpy().reshape(-1)


def _prefill_as_layer_major(spec, l, tag):
    per = spec.nbytes // spec.L
    g = np.arange(l * per // 8, (l + 1) * per // 8, dtype=np.uint64)
    return prefill_words(g, tag).view(np.uint8).copy()


def _buf_layer_without_token_count(t, spec, l, blocks):
    per_tok = spec.C * spec.H * spec.D * spec.e
    parts, offs, pos = [], [], 0
    for off, n in blocks:
        start = off * spec.e + l * per_tok           # should be l * n * per_tok
        parts.append(t[start:start + n * per_tok].cpu().numpy())
        offs.append(pos // spec.e)
        pos += n * per_tok
    return (np.concatenate(parts) if parts else np.zeros(0, np.uint8)), offs


def _one_layer_keeps_layers(spec):
    return spec


MISTAKES = {
    "pool_layer reads page-major pools as layer-major": ("pool_layer", _pool_layer_as_layer_major),
    "pool_layer with (layer, page) strides swapped": ("pool_layer", _pool_layer_wrong_page_stride),
    "prefill of page-major pools at layer-major offsets": ("pool_layer_prefill", _prefill_as_layer_major),
    "buffer layer offset without the block's token count": ("buf_layer", _buf_layer_without_token_count),
    "one-layer shape keeps every layer": ("one_layer", _one_layer_keeps_layers),
}


def _sweep_passes() -> bool:
    """True if every layer of a set of cases that spans page-major pools,
    flat buffers and slices passes."""
    wls = [_small("relayout"), _small("host_tier"), _small("handoff"),
           cases.transfer_case("PLCTHD", "PLCTHD", 4, 8, seed=3, L=3)]
    for wl in wls:
        try:
            res = layer_results(wl)
        except Exception:                      # a shape error is a failure too
            return False
        if not all(ok for _, _, ok in res):
            return False
    return True


def test_sweep_passes_unmodified():
    assert _sweep_passes()


@pytest.mark.parametrize("what", list(MISTAKES))
def test_planted_mistake_is_caught(what, monkeypatch):
    attr, fn = MISTAKES[what]
    monkeypatch.setattr(layer_check, attr, fn)
    assert not _sweep_passes(), f"layer checks pass with a planted mistake: {what}"
