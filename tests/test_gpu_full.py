"""Full-size workloads on the GPU, in the launch configuration bench.py
times, checked against the CPU oracle on every layer (layers never mix: a
layer slice of a pool is a one-layer pool of the same layout), including the
bytes the copy must leave untouched.  The per-layer oracle calls run on a
pool of host threads (ctypes releases the GIL)."""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

# Host threads for the per-layer checks.  Each holds about three layer
# slices in host memory (up to 4 GiB for the MLA workload).
THREADS = max(1, min(8, len(os.sched_getaffinity(0))))


@pytest.fixture(scope="module")
def torch():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_31093_amd import kvx
    kvx.lib()
    return torch


def _setup(torch, k):
    from paper_2606_31093_amd import kvx, workloads
    wl = workloads.get(k)
    dev = torch.device("cuda", 0)
    mem = {n: workloads.alloc_side(s, dev, pinned=n in wl.host_sides) for n, s in wl.sides.items()}
    workloads.init_sides_(wl, mem)
    dsteps = [dict(st=st,
                   spt=kvx.device_table(st.src_pt) if st.src_pt is not None else None,
                   dpt=kvx.device_table(st.dst_pt) if st.dst_pt is not None else None,
                   reqs=kvx.device_reqs(st.reqs)) for st in wl.steps]
    torch.cuda.synchronize()
    return wl, mem, dsteps


def _run(torch, wl, mem, d, planned=True):
    """One step as bench.py launches it: a transfer goes through
    kvx_transfer_planned with the plan of its destination pages
    (planned=False: the plain call).  The library's measured launch choice
    would alternate the sweep and the persistent grid on these first calls,
    and the grid rewrites every byte the sweep wrote, so planned calls here
    are held to the sweep (the grid is the unplanned cases' launch)."""
    from paper_2606_31093_amd import kvx
    kvx.kvx_set_launch_choice(kvx.CHOOSE_SWEEP if planned else kvx.CHOOSE_MEASURED)
    try:
        return _launch(torch, wl, mem, d, planned)
    finally:
        kvx.kvx_set_launch_choice(kvx.CHOOSE_MEASURED)


def _launch(torch, wl, mem, d, planned):
    from paper_2606_31093_amd import kvx
    st = d["st"]
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    S, D = wl.sides[st.src], wl.sides[st.dst]
    if st.op == "transfer" and planned and st.layer_group:
        plan, pages, tokens = kvx.device_plan(st.reqs, S.T, D.T)
        n_layers = st.slice[2] if st.slice is not None else S.L
        events = [torch.cuda.Event() for _ in range(-(-n_layers // st.layer_group))]
        kvx.kvx_transfer_layered_planned(mem[st.src], S, mem[st.dst], D, d["spt"], d["dpt"], d["reqs"],
                                         st.layer_group, events, plan, pages, tokens, st.slice, err)
    elif st.op == "transfer" and planned:
        plan, pages, tokens = kvx.device_plan(st.reqs, S.T, D.T)
        kvx.kvx_transfer_planned(mem[st.src], S, mem[st.dst], D, d["spt"], d["dpt"], d["reqs"],
                                 plan, pages, tokens, st.slice, err)
    elif st.op == "transfer" and st.slice is not None:
        kvx.kvx_transfer_slice(mem[st.src], S, mem[st.dst], D, st.slice, d["spt"], d["dpt"],
                               d["reqs"], err)
    elif st.op == "transfer":
        kvx.kvx_transfer(mem[st.src], S, mem[st.dst], D, d["spt"], d["dpt"], d["reqs"], err)
    elif st.op == "gather" and st.slice is not None:
        kvx.kvx_gather_slice(mem[st.src], S, mem[st.dst], D, st.slice, d["spt"], d["reqs"], err)
    elif st.op == "gather":
        kvx.kvx_gather(mem[st.src], S, mem[st.dst], D, d["spt"], d["reqs"], err)
    elif st.slice is not None:
        kvx.kvx_scatter_slice(mem[st.src], S, mem[st.dst], D, st.slice, d["dpt"], d["reqs"], err)
    else:
        kvx.kvx_scatter(mem[st.src], S, mem[st.dst], D, d["dpt"], d["reqs"], err)
    torch.cuda.synchronize()
    return int(err.item())


def _each_layer(fn, n_layers):
    """fn(l) for every layer on the thread pool; returns the results in order."""
    with ThreadPoolExecutor(THREADS) as ex:
        return list(ex.map(fn, range(n_layers)))


def _free(torch, *objs):
    del objs
    torch.cuda.empty_cache()


@pytest.mark.parametrize("k,planned", [("handoff", True), ("handoff", False), ("handoff_layered", True),
                                       ("relayout", True), ("relayout", False), ("mla", True),
                                       ("mla", False), ("tp_reshard", True),
                                       ("cow_fork", True), ("small_requests", True)])
def test_full_transfer(torch, k, planned):
    from oracle import layer_check
    wl, mem, dsteps = _setup(torch, k)
    st = dsteps[0]["st"]
    src = mem[st.src]
    S, D = wl.sides[st.src], wl.sides[st.dst]
    n_layers = st.slice[2] if st.slice is not None else S.L
    same_pool = st.src == st.dst
    # a copy inside one pool starts from the pool's values, not a prefill: keep
    # a device copy of the pool as it was
    pool_before = mem[st.dst].clone() if same_pool else None
    before = int(src.view(torch.int64).sum().item()) if not same_pool else None
    print(f"{k}: {wl.title}; {n_layers} layers on {THREADS} threads", flush=True)
    for _ in range(2):                       # repeated launches write the same bytes
        assert _run(torch, wl, mem, dsteps[0], planned) == 0
    if not same_pool:
        assert int(src.view(torch.int64).sum().item()) == before, "source pool modified"

    def check(l):
        if st.slice is not None:
            r = layer_check.check_transfer_slice_layer(mem[st.src], S, mem[st.dst], D, st, l,
                                                       wl.prefill_tag)
        else:
            dst_before = layer_check.pool_layer(pool_before, D, l) if same_pool else None
            r = layer_check.check_transfer_layer(mem[st.src], S, mem[st.dst], D, st, l,
                                                 wl.prefill_tag, dst_before)
        print(f"  layer {l}: oracle {r.oracle_seconds:.2f} s, equal={r.equal}", flush=True)
        return r.equal

    results = _each_layer(check, n_layers)
    bad = [l for l, ok in enumerate(results) if not ok]
    assert not bad, f"{k}: layers {bad} differ from the oracle"
    if st.slice is not None:
        # layers of the destination outside the slice keep their prefill
        ld0, nl = st.slice[1], st.slice[2]
        for l in [x for x in range(D.L) if not ld0 <= x < ld0 + nl]:
            assert np.array_equal(layer_check.pool_layer(mem[st.dst], D, l),
                                  layer_check.pool_layer_prefill(D, l, wl.prefill_tag))
    _free(torch, mem, dsteps, pool_before)


def _offload_onload(torch, name, slice_check):
    from oracle import layer_check
    wl, mem, dsteps = _setup(torch, name)
    g, s = wl.steps
    S, B = wl.sides["A"], wl.sides["buf"]
    pool_before = mem["A"].clone()
    assert _run(torch, wl, mem, dsteps[0]) == 0       # offload to pinned host memory
    assert _run(torch, wl, mem, dsteps[1]) == 0       # onload into fresh pages
    print(f"{name}: {wl.title}; {S.L} layers on {THREADS} threads", flush=True)
    per_page = S.nbytes // S.L // S.N

    def check(l):
        before = layer_check.pool_layer(pool_before, S, l)
        after = layer_check.pool_layer(mem["A"], S, l)
        if slice_check:
            ok_g, ok_s = layer_check.gather_scatter_slice_layer(before, S, mem["buf"], B, after,
                                                                g, s, l)
        else:
            ok_g, ok_s = layer_check.gather_scatter_layer(before, S, mem["buf"], B, after, g, s, l)
            # round trip: new page k holds the pre-offload bytes of original page k
            old = before.reshape(S.N, per_page)[g.src_pt]
            new = after.reshape(S.N, per_page)[s.dst_pt]
            ok_s = ok_s and np.array_equal(old, new)
        print(f"  layer {l}: offload equal={ok_g}, onload equal={ok_s}", flush=True)
        return ok_g and ok_s

    results = _each_layer(check, S.L)
    bad = [l for l, ok in enumerate(results) if not ok]
    assert not bad, f"{name}: layers {bad} differ from the oracle"
    _free(torch, mem, dsteps, pool_before)


def test_full_host_offload_onload(torch):
    _offload_onload(torch, "host_tier", slice_check=False)


def test_full_host_v_only_offload_onload(torch):
    """The host-tier pages, V only: the offload fills a V-only pinned buffer
    and the onload writes only the V half of the fresh pages."""
    _offload_onload(torch, "host_tier_v", slice_check=True)
