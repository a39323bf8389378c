"""HIP path vs the CPU oracle, bit for bit, at sizes the oracle finishes in
seconds: the tiny workload, shrunken versions of the four large ones, every
layout pair and page-size pair, every element width, pinned host buffers,
tiles spanning more source pages than a wavefront has lanes, and the
documented error behaviour."""
import zlib

import numpy as np
import pytest

import cases
from paper_2606_31093_amd.workloads import PoolSpec, BufSpec, Step, Workload, get
from runner import assert_same, initial_bytes, run_gpu, run_oracle

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_31093_amd import kvx
    kvx.lib()    # raises if libkvx.so is missing: no fallback


def check(wl, raw_reqs=None, oracle_reqs=None):
    init = initial_bytes(wl)
    want, werr = run_oracle(wl, init, oracle_reqs)
    got, gerr = run_gpu(wl, init, raw_reqs)
    assert gerr == werr, f"{wl.title}: device error bits {gerr}, oracle {werr}"
    assert_same(got, want, wl.title)
    return got, gerr


def test_tiny_workload():
    check(get("tiny"))


@pytest.mark.parametrize("name", ["handoff", "relayout", "mla", "host_tier", "tp_reshard",
                                  "cow_fork", "handoff_layered", "small_requests", "host_tier_v"])
def test_small_workloads(name):
    check(get(name, small=True))


@pytest.mark.parametrize("ls,ld,Ts,Td", list(cases.layout_matrix()),
                         ids=lambda v: str(v))
def test_layout_matrix(ls, ld, Ts, Td):
    # a seed fixed by the case itself (Python salts str hashes per process)
    seed = zlib.crc32(repr((ls, ld, Ts, Td)).encode()) & 0xFFFF
    check(cases.transfer_case(ls, ld, Ts, Td, seed=seed))


@pytest.mark.parametrize("e,D,C,H", [(1, 16, 2, 3), (2, 8, 2, 3), (4, 4, 1, 5), (8, 2, 2, 1),
                                     (8, 8, 2, 2), (1, 48, 1, 1), (2, 576, 1, 1),
                                     (2, 128, 2, 8), (4, 12, 2, 2)])
@pytest.mark.parametrize("ls,ld", [("LPCTHD", "LPCTHD"), ("LPCTHD", "PLCHTD"),
                                   ("LPCHTD", "PLCTHD")])
def test_element_widths(e, D, C, H, ls, ld):
    check(cases.transfer_case(ls, ld, 4, 8, seed=e * 1000 + D, e=e, D=D, C=C, H=H))


@pytest.mark.parametrize("layout", ["LPCTHD", "LPCHTD", "PLCTHD", "PLCHTD"])
@pytest.mark.parametrize("T,e,D", [(16, 2, 64), (4, 2, 8), (8, 1, 16), (2, 4, 12), (1, 8, 2),
                                   (64, 2, 576)])
@pytest.mark.parametrize("pinned", [False, True], ids=["device_buf", "pinned_host_buf"])
def test_gather_scatter(layout, T, e, D, pinned):
    check(cases.gather_scatter_case(layout, T, e, D, seed=T * 31 + e * 7 + D, pinned=pinned))


@pytest.mark.parametrize("ls,ld,Ts,Td", [("LPCTHD", "LPCTHD", 16, 16), ("LPCTHD", "LPCTHD", 4, 16),
                                         ("LPCTHD", "PLCHTD", 16, 64), ("PLCHTD", "LPCHTD", 8, 4)])
def test_transfer_into_pinned_host_pool(ls, ld, Ts, Td):
    """A destination pool in pinned host memory (ordinary stores over PCIe),
    on contiguous-run and row-resolving launches."""
    wl = cases.transfer_case(ls, ld, Ts, Td, seed=Ts * 13 + Td)
    wl.host_sides = ("B",)
    check(wl)


@pytest.mark.parametrize("k", range(len(cases.BUFFER_SLICES)))
@pytest.mark.parametrize("ls,ld", [("LPCTHD", "LPCTHD"), ("PLCHTD", "LPCTHD"), ("LPCHTD", "PLCTHD")])
@pytest.mark.parametrize("T", [1, 8, 64])
def test_buffer_slices(k, ls, ld, T):
    """A slice of one pool gathered into a buffer of exactly the slice and
    scattered into a slice of another pool (K only, V only, K into V, a
    tensor-parallel shard of a layer stage, a larger pool, one row)."""
    a, b, sl, off = cases.BUFFER_SLICES[k]
    check(cases.buffer_slice_case(ls, ld, T, a, b, sl, off, seed=k * 10 + T,
                                  pinned=(k + T) % 2 == 1))


def test_offset_views_into_pinned_host_memory():
    """A flat buffer and a pool that start inside larger pinned allocations
    (16-byte aligned views at an offset): the device addresses the library
    derives must keep the offset."""
    import torch
    from paper_2606_31093_amd import kvx
    wl = cases.gather_scatter_case("LPCTHD", 16, 2, 64, seed=57)
    g, sc = wl.steps
    A, B, P2 = wl.sides["A"], wl.sides["buf"], wl.sides["B"]
    init = initial_bytes(wl)
    want, werr = run_oracle(wl, init)
    pad = 4096 + 48
    hbuf = torch.zeros(B.nbytes + 2 * pad, dtype=torch.uint8, pin_memory=True)
    hpool = torch.zeros(P2.nbytes + 2 * pad, dtype=torch.uint8, pin_memory=True)
    hbuf.fill_(0xA5)
    hpool.fill_(0xA5)
    buf = hbuf[pad:pad + B.nbytes]
    pool = hpool[pad:pad + P2.nbytes]
    buf.copy_(torch.from_numpy(init["buf"]))
    pool.copy_(torch.from_numpy(init["B"]))
    src = torch.from_numpy(init["A"]).cuda()
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    kvx.kvx_gather(src, A, buf, B, kvx.device_table(g.src_pt), kvx.device_reqs(g.reqs), err)
    kvx.kvx_scatter(buf, B, pool, P2, kvx.device_table(sc.dst_pt), kvx.device_reqs(sc.reqs), err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0 and werr == [0, 0]
    assert np.array_equal(buf.numpy(), want["buf"])
    assert np.array_equal(pool.numpy(), want["B"])
    for whole in (hbuf, hpool):                       # nothing outside the views
        h = whole.numpy()
        assert (h[:pad] == 0xA5).all() and (h[-pad:] == 0xA5).all()


@pytest.mark.parametrize("layout", ["LPCTHD", "PLCHTD"])
def test_scatter_into_pinned_host_pool(layout):
    """Gather into a pinned host buffer, then scatter from it into a pool that
    is also pinned host memory."""
    wl = cases.gather_scatter_case(layout, 16, 2, 64, seed=41, pinned=True)
    wl.host_sides = ("buf", "B")
    check(wl)


@pytest.mark.parametrize("ls,ld", [("LPCTHD", "LPCTHD"), ("LPCTHD", "PLCHTD"),
                                   ("PLCHTD", "LPCHTD")])
def test_more_pieces_than_lanes(ls, ld):
    """One destination page of 128 tokens fed by 1-token source pages: up to
    128 source pages per tile, beyond the 64 a wavefront broadcasts."""
    check(cases.transfer_case(ls, ld, 1, 128, seed=77, H=2,
                              spec=[(3, 5, 200, None), (0, 0, 128, None), (1, 0, 64, None)]))


def test_partial_last_iteration():
    """A row-resolving tile of 1157 vectors (37 source pages of 32 tokens into
    one 2048-token page): the last pass of the vector loop covers only part
    of a wavefront, and those lanes still read page ids held by lanes past
    the end of the tile."""
    check(cases.transfer_case("LPCTHD", "LPCTHD", 32, 2048, seed=31, L=2, C=1, H=1, D=8,
                              spec=[(0, 0, 1157, None), (7, 3, 900, None)]))


@pytest.mark.parametrize("seed", range(cases.RANDOM_CASES))
def test_random_cases(seed):
    """Seeded random pool -> pool cases (layouts, page sizes, shapes, element
    widths, ranges, shared pages, slices, damaged tables)."""
    check(cases.random_case(seed))


@pytest.mark.parametrize("seed", range(cases.RANDOM_MEDIUM_CASES))
def test_random_medium_transfers(seed):
    """Seeded random transfers of 100-900 requests: several record chunks,
    many tiles per workgroup, random layouts and page sizes."""
    check(cases.random_medium_case(seed))


@pytest.mark.parametrize("seed", range(cases.RANDOM_GS_CASES))
def test_random_gather_scatter(seed):
    """Seeded random gathers into a flat buffer (device or pinned host) and
    scatters back into a second pool, with damaged records and page ids."""
    check(cases.random_gs_case(seed))


@pytest.mark.parametrize("seed", range(cases.RANDOM_COW_CASES))
def test_random_copy_on_write(seed):
    """Seeded random copies inside one pool into fresh pages."""
    check(cases.random_cow_case(seed))


@pytest.mark.parametrize("seed", range(cases.RANDOM_LAYERED_CASES))
def test_random_layered(seed):
    """Seeded random transfers moved in random layer groups."""
    check(cases.random_layered_case(seed))


def test_many_requests_and_empty_ones():
    spec = [((7 * i) % 13, (5 * i) % 11, (i * 37) % 90 if i % 4 else 0, None) for i in range(60)]
    check(cases.transfer_case("LPCTHD", "PLCHTD", 16, 32, seed=5, H=2, D=64, spec=spec))


# ---------------------------------------------------------------------------
# slices (layer range, kv range, head range)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("ls,ld", [("LPCTHD", "LPCTHD"), ("LPCTHD", "PLCHTD"), ("LPCHTD", "LPCHTD"),
                                   ("PLCTHD", "LPCHTD"), ("PLCHTD", "PLCTHD")])
@pytest.mark.parametrize("k", range(len(cases.SLICES)))
@pytest.mark.parametrize("Ts,Td", [(4, 8), (16, 16), (1, 32)])
def test_slices(ls, ld, k, Ts, Td):
    a, b, sl = cases.SLICES[k]
    check(cases.slice_case(ls, ld, Ts, Td, a, b, sl, seed=k * 97 + Ts * 7 + Td))


def test_slice_wide_rows():
    check(cases.slice_case("LPCTHD", "LPCTHD", 64, 64, (3, 1, 1), (2, 1, 1),
                           (1, 0, 2, 0, 0, 1, 0, 0, 1), seed=4, D=576))


def test_tp_split_and_merge():
    """Eight heads split into two four-head shards, then merged back."""
    S = PoolSpec(2, 2, 8, 64, T=16, N=12, e=2, layout="LPCTHD")
    half = PoolSpec(2, 2, 4, 64, T=32, N=6, e=2, layout="PLCHTD")
    rng = np.random.default_rng(3)
    spt = rng.permutation(S.N).astype(np.int32)
    hpt = rng.permutation(half.N).astype(np.int32)
    mpt = rng.permutation(S.N).astype(np.int32)
    r1 = np.asarray([[0, 0, 0, 5, 0, 100]], np.int64)
    r2 = np.asarray([[0, 0, 0, 0, 5, 100]], np.int64)
    steps = [Step("transfer", "A", "H0", spt, hpt, r1, slice=(0, 0, 2, 0, 0, 2, 0, 0, 4)),
             Step("transfer", "A", "H1", spt, hpt, r1, slice=(0, 0, 2, 0, 0, 2, 4, 0, 4)),
             Step("transfer", "H0", "M", hpt, mpt, r2, slice=(0, 0, 2, 0, 0, 2, 0, 0, 4)),
             Step("transfer", "H1", "M", hpt, mpt, r2, slice=(0, 0, 2, 0, 0, 2, 0, 4, 4))]
    wl = Workload("case", "tp split/merge", {"A": S, "H0": half, "H1": half, "M": S}, steps,
                  value_seed=8, prefill_tag=8)
    got, errs = check(wl)
    assert errs == [0, 0, 0, 0]


@pytest.mark.parametrize("src_pt,dst_pt,row,bits", [
    ([0, 4], [0, 1], [0, 0, 0, 0, 0, 8], 1),
    ([7, 1], [-1, 1], [0, 0, 0, 0, 0, 4], 2),
    ([0], [0, 1], [0, 0, 0, 0, 0, 8], 4),
    ([0, 1], [0, 1], [0, 0, 0, 0, 0, -2], 8),
])
def test_slice_device_errors(src_pt, dst_pt, row, bits):
    S = PoolSpec(2, 2, 2, 8, T=4, N=4, e=2, layout="LPCTHD")
    Dp = PoolSpec(1, 1, 2, 8, T=4, N=4, e=2, layout="LPCHTD")
    wl = Workload("case", "slice errors", {"A": S, "B": Dp},
                  [Step("transfer", "A", "B", np.asarray(src_pt, np.int32),
                        np.asarray(dst_pt, np.int32), np.asarray([row], np.int64),
                        slice=(1, 0, 1, 1, 0, 1, 0, 0, 2))], value_seed=2, prefill_tag=3)
    _, errs = check(wl)
    assert errs == [bits]


@pytest.mark.parametrize("layout", ["LPCTHD", "LPCHTD", "PLCTHD", "PLCHTD"])
def test_same_pool_copy_on_write(layout):
    """A fork copies its partial last page, and another its whole prefix,
    into fresh pages of the same pool (source and destination are one
    allocation)."""
    P = PoolSpec(2, 2, 3, 64, T=8, N=12, e=2, layout=layout)
    rows = np.asarray([[2, 3, 0, 0, 0, 4], [0, 0, 0, 0, 0, 20], [0, 4, 0, 3, 0, 9]], np.int64)
    wl = Workload("case", f"copy-on-write {layout}", {"A": P},
                  [Step("transfer", "A", "A", np.asarray([5, 2, 9], np.int32),
                        np.asarray([0, 11, 3, 7, 1, 4], np.int32), rows)],
                  value_seed=41, prefill_tag=1)
    check(wl)


# ---------------------------------------------------------------------------
# layer-pipelined transfer
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("group", [1, 2, 3, 5])
@pytest.mark.parametrize("with_slice", [False, True])
def test_layered_matches_oracle(group, with_slice):
    if with_slice:
        wl = cases.slice_case("LPCTHD", "PLCHTD", 4, 8, (5, 2, 4), (4, 2, 2),
                              (1, 0, 4, 0, 0, 2, 2, 0, 2), seed=group)
    else:
        wl = cases.transfer_case("LPCHTD", "LPCTHD", 16, 32, seed=group, L=5)
    wl.steps[0].layer_group = group
    check(wl)


def test_layered_events_guard_consumers():
    """A consumer stream waits on each group's event, then snapshots that
    group's destination layers; every snapshot matches the oracle."""
    import torch
    from paper_2606_31093_amd import kvx
    from oracle import kvx_oracle
    wl = get("handoff", small=True)
    st = wl.steps[0]
    S = wl.sides["A"]
    S6 = PoolSpec(6, S.C, S.H, S.D, S.T, S.N, S.e, S.layout)
    init = initial_bytes(Workload("case", "", {"A": S6, "B": S6}, [st], 5, 5))
    want = init["B"].copy()
    assert kvx_oracle.default().transfer(init["A"], S6, want, S6, st.src_pt, st.dst_pt,
                                         st.reqs) == 0
    a = torch.from_numpy(init["A"]).cuda()
    b = torch.from_numpy(init["B"]).cuda()
    per_layer = S6.nbytes // S6.L
    events = [torch.cuda.Event() for _ in range(3)]
    producer, consumer = torch.cuda.Stream(), torch.cuda.Stream()
    snaps = []
    with torch.cuda.stream(producer):
        kvx.kvx_transfer_layered(a, S6, b, S6, kvx.device_table(st.src_pt),
                                 kvx.device_table(st.dst_pt), kvx.device_reqs(st.reqs), 2, events,
                                 stream=producer)
    for g in range(3):
        consumer.wait_event(events[g])
        with torch.cuda.stream(consumer):
            snaps.append(b[2 * g * per_layer:(2 * g + 2) * per_layer].clone())
    torch.cuda.synchronize()
    for g, snap in enumerate(snaps):
        assert np.array_equal(snap.cpu().numpy(),
                              want[2 * g * per_layer:(2 * g + 2) * per_layer]), f"group {g}"


def test_layered_records_events_when_empty():
    import torch
    from paper_2606_31093_amd import kvx
    S = PoolSpec(3, 2, 1, 8, T=4, N=4, e=2, layout="LPCTHD")
    a = torch.zeros(S.nbytes, dtype=torch.uint8, device="cuda")
    events = [torch.cuda.Event() for _ in range(3)]
    empty = torch.empty(0, dtype=torch.uint8, device="cuda")
    kvx.kvx_transfer_layered(a, S, a.clone(), S, None, None, empty, 1, events)
    torch.cuda.synchronize()
    assert all(ev.query() for ev in events)


# ---------------------------------------------------------------------------
# sizes at the edges
# ---------------------------------------------------------------------------

def test_huge_pages():
    """Pages of 65536 tokens on both sides (tiles of 65536 rows), one page of
    2^20 tokens read into smaller pages, and a head-major destination whose
    rows are masked per page."""
    check(cases.transfer_case("LPCTHD", "LPCTHD", 1 << 16, 1 << 16, seed=12, L=1, C=1, H=1, D=8,
                              spec=[(5, 70000, 60000, None), (0, 0, 3, None)]))
    check(cases.transfer_case("LPCTHD", "PLCHTD", 1 << 20, 4096, seed=13, L=1, C=1, H=2, D=8,
                              spec=[(1000, 17, 9000, None)], extra_pages=1))


def test_thousands_of_requests():
    """4096 records, most of them tiny, some empty: every workgroup walks all
    of them."""
    rng = np.random.default_rng(21)
    spec = [(int(rng.integers(0, 16)), int(rng.integers(0, 8)), int(rng.integers(0, 5)), None)
            for _ in range(4096)]
    check(cases.transfer_case("LPCTHD", "LPCTHD", 16, 8, seed=21, L=2, C=2, H=1, D=8, spec=spec,
                              extra_pages=0))


def test_max_records():
    """KVX_MAX_REQS (65536) records of 0-2 tokens in one call: the record scan
    runs through 256 chunks.  Each record writes its own destination page;
    sources are random, shared pages."""
    rng = np.random.default_rng(65536)
    n = 65536
    S = PoolSpec(1, 1, 1, 8, T=4, N=512, e=2, layout="LPCTHD")
    Dp = PoolSpec(1, 1, 1, 8, T=2, N=n, e=2, layout="LPCTHD")
    toks = rng.integers(0, 3, size=n)
    s0 = rng.integers(0, 3, size=n) % np.maximum(1, 5 - toks)       # s0 + toks <= 4: one page
    src_pt = rng.integers(0, S.N, size=n).astype(np.int32)
    dst_pt = rng.permutation(n).astype(np.int32)
    rows = np.stack([np.arange(n), np.arange(n), np.zeros(n), s0, np.zeros(n), toks], 1)
    wl = Workload("case", "65536 records", {"A": S, "B": Dp},
                  [Step("transfer", "A", "B", src_pt, dst_pt, rows.astype(np.int64))],
                  value_seed=7, prefill_tag=7)
    check(wl)


def test_graph_replays_match_eager():
    """The transfer captured in a HIP graph and replayed several times, with
    eager work in between, gives the eager result every time."""
    import torch
    from paper_2606_31093_amd import kvx
    wl = get("handoff", small=True)
    st = wl.steps[0]
    init = initial_bytes(wl)
    want, _ = run_oracle(wl, init)
    a = torch.from_numpy(init["A"]).cuda()
    b = torch.from_numpy(init["B"]).cuda()
    spt, dpt, reqs = kvx.device_table(st.src_pt), kvx.device_table(st.dst_pt), kvx.device_reqs(st.reqs)
    b0 = b.clone()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        kvx.kvx_transfer(a, wl.sides["A"], b, wl.sides["B"], spt, dpt, reqs, stream=s)   # warm up
    torch.cuda.current_stream().wait_stream(s)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        kvx.kvx_transfer(a, wl.sides["A"], b, wl.sides["B"], spt, dpt, reqs)
    for _ in range(3):
        b.copy_(b0)                    # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(b.cpu().numpy(), want["B"])


@pytest.mark.parametrize("pinned", [False, True], ids=["device", "pinned_host"])
def test_empty_buffer_without_memory(pinned):
    """A gather into and a scatter out of a buffer of capacity 0, which a
    zero-size tensor gives a NULL base: records of 0 tokens copy nothing and
    raise nothing, a record of 3 tokens raises KVX_DERR_BAD_REQ, and no pool
    byte changes."""
    S = PoolSpec(2, 2, 2, 16, T=4, N=6, e=2, layout="LPCHTD")
    B = BufSpec(2, 2, 2, 16, 2, cap=0)
    pt = np.array([3, 1, 4, 0], np.int32)
    g_rows = np.array([[0, 0, 0, 0, 0, 0], [1, 0, 0, 2, 0, 0], [2, 0, 0, 1, 0, 3]], np.int64)
    s_rows = np.array([[0, 0, 0, 0, 0, 0], [0, 1, 0, 0, 3, 0], [0, 2, 0, 0, 1, 3]], np.int64)
    wl = Workload("case", "empty buffer", {"A": S, "buf": B, "B": S},
                  [Step("gather", "A", "buf", pt, None, g_rows),
                   Step("scatter", "buf", "B", None, pt, s_rows)],
                  value_seed=5, prefill_tag=7, host_sides=("buf",) if pinned else ())
    _, gerr = check(wl)
    assert gerr == [8, 8]          # the 3-token record, in the gather and in the scatter


def test_calls_from_four_host_threads():
    """Four host threads, each with its own stream and destination pool,
    call the library 25 times at once (ctypes releases the GIL): every
    destination equals the oracle's, and every thread's error word and last
    error message stay its own."""
    import threading
    import torch
    from paper_2606_31093_amd import kvx
    wl = get("handoff", small=True)
    st = wl.steps[0]
    init = initial_bytes(wl)
    want, _ = run_oracle(wl, init)
    a = torch.from_numpy(init["A"]).cuda()
    spt, dpt, reqs = kvx.device_table(st.src_pt), kvx.device_table(st.dst_pt), kvx.device_reqs(st.reqs)
    outs = [torch.from_numpy(init["B"]).cuda() for _ in range(4)]
    errs = torch.zeros(4, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    failures = []

    def work(t):
        try:
            s = torch.cuda.Stream()
            for _ in range(25):
                kvx.kvx_transfer(a, wl.sides["A"], outs[t], wl.sides["B"], spt, dpt, reqs,
                                 errs[t:t + 1], stream=s)
            with pytest.raises(kvx.KvxError):           # a host error on this thread only
                kvx.kvx_transfer(a, wl.sides["A"], outs[t], wl.sides["B"], spt, dpt,
                                 torch.zeros(40, dtype=torch.uint8), stream=s)
            assert "reqs" in kvx.kvx_last_error()       # this thread's message
            s.synchronize()
        except Exception as e:                          # reported on the main thread
            failures.append(repr(e))

    threads = [threading.Thread(target=work, args=(t,)) for t in range(4)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    torch.cuda.synchronize()
    assert not failures, failures
    assert errs.cpu().tolist() == [0, 0, 0, 0]
    for o in outs:
        assert np.array_equal(o.cpu().numpy(), want["B"])


def test_concurrent_calls_on_three_streams():
    """Two transfers out of the same source pool into two destination pools
    and a page-hash call, each on its own stream and in flight together:
    the library keeps no state between calls, so each result equals the
    oracle's for that call alone."""
    import torch
    from oracle import kvx_oracle
    from paper_2606_31093_amd import kvx
    from paper_2606_31093_amd import workloads as W
    wl = get("handoff", small=True)
    st = wl.steps[0]
    init = initial_bytes(wl)
    want, _ = run_oracle(wl, init)
    a = torch.from_numpy(init["A"]).cuda()
    b1 = torch.from_numpy(init["B"]).cuda()
    b2 = torch.from_numpy(init["B"]).cuda()
    spt, dpt, reqs = kvx.device_table(st.src_pt), kvx.device_table(st.dst_pt), kvx.device_reqs(st.reqs)
    hw = W.page_hash(small=True)
    pay = W.hash_payload(hw)
    hwant = np.zeros(hw.out_len, np.uint64)
    assert kvx_oracle.default().page_hashes(pay, hw.rec_bytes, hw.T, hw.rows, hwant) == 0
    tpay = torch.from_numpy(pay.view(np.uint8).copy()).cuda()
    hreqs = kvx.device_hash_reqs(hw.rows)
    hout = torch.zeros(hw.out_len, dtype=torch.int64, device="cuda")
    errs = torch.zeros(3, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in range(3)]
    for rep in range(3):
        kvx.kvx_transfer(a, wl.sides["A"], b1, wl.sides["B"], spt, dpt, reqs, errs[0:1], stream=streams[0])
        kvx.kvx_transfer(a, wl.sides["A"], b2, wl.sides["B"], spt, dpt, reqs, errs[1:2], stream=streams[1])
        kvx.kvx_page_hashes(tpay, hw.rec_bytes, hw.T, hreqs, hout, errs[2:3], stream=streams[2])
    torch.cuda.synchronize()
    assert errs.cpu().tolist() == [0, 0, 0]
    assert np.array_equal(b1.cpu().numpy(), want["B"])
    assert np.array_equal(b2.cpu().numpy(), want["B"])
    assert np.array_equal(a.cpu().numpy(), init["A"])
    assert np.array_equal(hout.cpu().numpy().view(np.uint64), hwant)


# ---------------------------------------------------------------------------
# error behaviour
# ---------------------------------------------------------------------------

def _err_wl(src_pt, dst_pt, rows, N=4, T=4):
    S = PoolSpec(1, 2, 1, 8, T=T, N=N, e=2, layout="LPCTHD")
    return Workload("case", f"errors {rows}", {"A": S, "B": S},
                    [Step("transfer", "A", "B", np.asarray(src_pt, np.int32),
                          np.asarray(dst_pt, np.int32), np.asarray(rows, np.int64).reshape(-1, 6))],
                    value_seed=3, prefill_tag=9)


@pytest.mark.parametrize("src_pt,dst_pt,row,bits", [
    ([0, 4], [0, 1], [0, 0, 0, 0, 0, 8], 1),          # source page id == N
    ([0, 1], [-1, 1], [0, 0, 0, 0, 0, 8], 2),         # negative destination page id
    ([7, 1], [-1, 1], [0, 0, 0, 0, 0, 4], 2),         # both bad: destination first
    ([7, 1], [0, 1], [0, 0, 0, 0, 0, 4], 1),
    ([0], [0, 1], [0, 0, 0, 0, 0, 8], 4),             # source table too short
    ([0, 1], [0, 1], [0, 1, 0, 0, 0, 8], 4),          # destination table too short
    ([0, 1], [0, 1], [0, 0, 0, 0, 0, -1], 8),         # negative count
    ([0, 1], [0, 1], [0, 0, 0, -1, 0, 2], 8),         # negative start
    ([0, 1], [0, 1], [0, 0, 0, 2**31 - 2, 0, 3], 8),  # end beyond 2^31 - 1
    ([0, 1, 2, 3], [2, 0, 1, 3], [0, 0, 0, 3, 6, 9], 0),
])
def test_device_errors(src_pt, dst_pt, row, bits):
    _, errs = check(_err_wl(src_pt, dst_pt, [row, [0, 0, 0, 0, 0, 2]]))
    assert errs == [bits]


def test_buffer_record_errors():
    """Buffer-side start must be 0; the block must be 16-byte aligned and
    inside the buffer (ending exactly at its end is fine)."""
    S = PoolSpec(1, 2, 1, 8, T=4, N=4, e=2, layout="LPCTHD")
    n = 3
    B = BufSpec(1, 2, 1, 8, 2, cap=2 * n * 8 + 8)
    for row, bits in (([0, 0, 8, 0, 0, n], 0), ([0, 0, 0, 0, 0, n], 0), ([0, 0, 16, 0, 0, n], 8),
                      ([0, 0, 4, 0, 0, n], 8), ([0, 0, -8, 0, 0, n], 8), ([0, 0, 0, 0, 1, n], 8)):
        wl = Workload("case", f"gather {row}", {"A": S, "buf": B},
                      [Step("gather", "A", "buf", np.asarray([0, 1], np.int32), None,
                            np.asarray([row], np.int64))], value_seed=1, prefill_tag=2)
        _, errs = check(wl)
        assert errs == [bits]
    for row, bits in (([0, 0, 8, 0, 0, n], 0), ([0, 0, 16, 0, 0, n], 8), ([0, 0, 0, 2, 0, n], 8)):
        wl = Workload("case", f"scatter {row}", {"buf": B, "B": S},
                      [Step("scatter", "buf", "B", None, np.asarray([2, 3], np.int32),
                            np.asarray([row], np.int64))], value_seed=1, prefill_tag=2)
        _, errs = check(wl)
        assert errs == [bits]


def test_reserved_field_must_be_zero():
    """A record whose reserved word is not 0 is skipped with BAD_REQ (a rule
    of the C record format, so the oracle sees the record as absent)."""
    from paper_2606_31093_amd import kvx
    wl = _err_wl([0, 1], [2, 3], [[0, 0, 0, 0, 0, 8], [0, 0, 0, 0, 0, 3]])
    recs = kvx.pack_reqs(wl.steps[0].reqs)
    recs["reserved"][0] = 1
    init = initial_bytes(wl)
    want, werr = run_oracle(wl, init, [wl.steps[0].reqs[1:]])
    got, gerr = run_gpu(wl, init, [recs])
    assert werr == [0] and gerr == [8]
    assert_same(got, want, wl.title)


def test_max_position():
    T = 1 << 16
    S = PoolSpec(1, 1, 1, 8, T=T, N=1, e=2, layout="LPCTHD")
    B = BufSpec(1, 1, 1, 8, 2, cap=5 * 8)
    wl = Workload("case", "max position", {"A": S, "buf": B},
                  [Step("gather", "A", "buf", np.zeros(32768, np.int32), None,
                        np.asarray([[0, 0, 0, 2**31 - 6, 0, 5]], np.int64))],
                  value_seed=4, prefill_tag=4)
    _, errs = check(wl)
    assert errs == [0]


def test_zero_records_enqueue_nothing():
    import torch
    from paper_2606_31093_amd import kvx
    S = PoolSpec(1, 2, 1, 8, T=4, N=4, e=2, layout="LPCTHD")
    a = torch.zeros(S.nbytes, dtype=torch.uint8, device="cuda")
    b = torch.ones(S.nbytes, dtype=torch.uint8, device="cuda")
    reqs = torch.empty(0, dtype=torch.uint8, device="cuda")
    kvx.kvx_transfer(a, S, b, S, None, None, reqs)
    torch.cuda.synchronize()
    assert bool((b == 1).all())


def test_side_stream():
    """Work runs on the stream passed in, ordered with other work there."""
    import torch
    from paper_2606_31093_amd import kvx
    wl = get("handoff", small=True)
    init = initial_bytes(wl)
    want, _ = run_oracle(wl, init)
    st = wl.steps[0]
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        a = torch.from_numpy(init["A"]).to("cuda")
        b = torch.from_numpy(init["B"]).to("cuda")
        kvx.kvx_transfer(a, wl.sides["A"], b, wl.sides["B"], kvx.device_table(st.src_pt),
                         kvx.device_table(st.dst_pt), kvx.device_reqs(st.reqs), stream=s)
        got = b.cpu().numpy()
    assert np.array_equal(got, want["B"])


def test_host_validation_errors_raise():
    import torch
    from paper_2606_31093_amd import kvx
    S = PoolSpec(1, 2, 1, 8, T=4, N=4, e=2, layout="LPCTHD")
    a = torch.zeros(S.nbytes, dtype=torch.uint8, device="cuda")
    reqs = kvx.device_reqs([[0, 0, 0, 0, 0, 1]])
    pt = kvx.device_table([0])
    host = torch.zeros(S.nbytes, dtype=torch.uint8)   # pageable host memory
    with pytest.raises(kvx.KvxError) as ei:
        kvx.kvx_transfer(a, S, host, S, pt, pt, reqs)
    assert ei.value.status == -5
    big = torch.zeros(S.nbytes + 16, dtype=torch.uint8, device="cuda")
    with pytest.raises(kvx.KvxError) as ei:
        kvx.kvx_transfer(a, S, big[1:1 + S.nbytes], S, pt, pt, reqs)   # misaligned base
    assert ei.value.status == -3
