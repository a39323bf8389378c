"""The sweep launch of planned transfers (kvx_transfer_planned), bit for bit
against the oracle.

The test build (libkvx_test.so) takes the sweep for every planned transfer
whatever its size and destination layout, with at most 2048 workgroups per
pass (larger cases loop
over page slots), so small cases exercise it: every layout pair and
page-size pair, element widths, slices, copies inside one pool, the seeded
random cases (damaged tables, empty requests, shared source pages, slices)
and the device error rules.  A wrong token total only changes the choice of
launch.  A plan that disagrees with the records (a wrong page total, a
damaged prefix or slot, slots out of order, page sizes of other pools, or
random slot contents) raises KVX_DERR_BAD_PLAN, and every access still
stays inside the pools and tables.  The product library sweeps when the
records copy 64 KiB or more per page on average; a shape with 256 KiB pages
checks it there, and the full-size handoff, MLA, relayout, TP reshard and
fork are checked on every layer in test_gpu_full."""
import numpy as np
import pytest

import cases
from paper_2606_31093_amd.workloads import PoolSpec, Step, Workload
from runner import assert_same, initial_bytes, run_gpu, run_oracle

pytestmark = pytest.mark.gpu

# the token total passed with a correct plan: only the choice of launch changes
TOKENS = {"true": lambda t: t, "zero": lambda t: 0, "double": lambda t: 2 * t + 3}


def planned(tokens="true"):
    return lambda buf, pages, t: (buf, pages, TOKENS[tokens](t))


@pytest.fixture(scope="module")
def test_lib():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_31093_amd import build_lib, kvx
    kvx.lib()    # the product library first: raises if it is missing
    return kvx.load(build_lib.TEST_LIBRARY)


def check(wl, library, tokens="true"):
    init = initial_bytes(wl)
    want, werr = run_oracle(wl, init)
    got, gerr = run_gpu(wl, init, planned=planned(tokens), library=library)
    assert gerr == werr, f"{wl.title}: device error bits {gerr}, oracle {werr}"
    assert_same(got, want, wl.title)


@pytest.mark.parametrize("ls,ld,Ts,Td", list(cases.layout_matrix()), ids=lambda v: str(v))
def test_layout_matrix(test_lib, ls, ld, Ts, Td):
    import zlib
    check(cases.transfer_case(ls, ld, Ts, Td, seed=zlib.crc32(repr((ls, ld, Ts, Td, 7)).encode()) & 0xFFFF),
          test_lib)


@pytest.mark.parametrize("tokens", list(TOKENS))
@pytest.mark.parametrize("ls,ld,Ts,Td", [("LPCTHD", "LPCTHD", 16, 16), ("LPCTHD", "PLCHTD", 16, 64),
                                         ("PLCTHD", "LPCHTD", 8, 4), ("LPCHTD", "LPCTHD", 1, 16)])
def test_token_totals(test_lib, ls, ld, Ts, Td, tokens):
    check(cases.transfer_case(ls, ld, Ts, Td, seed=Ts * 7 + Td), test_lib, tokens)


@pytest.mark.parametrize("e,D,C,H", [(1, 16, 2, 3), (2, 8, 2, 3), (4, 4, 1, 5), (8, 2, 2, 1),
                                     (2, 576, 1, 1), (2, 128, 2, 8)])
@pytest.mark.parametrize("ls,ld", [("LPCTHD", "LPCTHD"), ("LPCTHD", "PLCHTD")])
def test_element_widths(test_lib, e, D, C, H, ls, ld):
    check(cases.transfer_case(ls, ld, 4, 8, seed=e * 100 + D, e=e, D=D, C=C, H=H), test_lib)


@pytest.mark.parametrize("k", range(len(cases.SLICES)))
@pytest.mark.parametrize("ls,ld", [("LPCTHD", "LPCTHD"), ("PLCHTD", "LPCTHD"), ("LPCHTD", "PLCTHD")])
@pytest.mark.parametrize("Ts,Td", [(4, 8), (16, 16)])
def test_slices(test_lib, k, ls, ld, Ts, Td):
    S_LCH, D_LCH, sl = cases.SLICES[k]
    check(cases.slice_case(ls, ld, Ts, Td, S_LCH, D_LCH, sl, seed=300 + k), test_lib)


@pytest.mark.parametrize("layout", ["LPCTHD", "LPCHTD", "PLCTHD", "PLCHTD"])
def test_same_pool(test_lib, layout):
    P = PoolSpec(2, 2, 3, 64, T=8, N=12, e=2, layout=layout)
    rows = np.asarray([[2, 3, 0, 0, 0, 4], [0, 0, 0, 0, 0, 20], [0, 4, 0, 3, 0, 9]], np.int64)
    wl = Workload("case", f"copy-on-write {layout}", {"A": P},
                  [Step("transfer", "A", "A", np.asarray([5, 2, 9], np.int32),
                        np.asarray([0, 11, 3, 7, 1, 4], np.int32), rows)],
                  value_seed=41, prefill_tag=1)
    check(wl, test_lib)


@pytest.mark.parametrize("seed", range(cases.RANDOM_CASES))
def test_random_cases(test_lib, seed):
    check(cases.random_case(seed), test_lib, list(TOKENS)[seed % len(TOKENS)])


@pytest.mark.parametrize("seed", range(6))
def test_random_cow_cases(test_lib, seed):
    check(cases.random_cow_case(seed), test_lib)


def _err_wl(src_pt, dst_pt, rows):
    S = PoolSpec(2, 2, 2, 8, T=4, N=4, e=2, layout="LPCTHD")
    return Workload("case", f"errors {src_pt} {dst_pt} {rows}", {"A": S, "B": S},
                    [Step("transfer", "A", "B", np.asarray(src_pt, np.int32),
                          np.asarray(dst_pt, np.int32), np.asarray(rows, np.int64).reshape(-1, 6))],
                    value_seed=3, prefill_tag=9)


@pytest.mark.parametrize("src_pt,dst_pt,row", [
    ([0, 4], [0, 1], [0, 0, 0, 0, 0, 8]),           # source page id == N
    ([0, 1], [-1, 1], [0, 0, 0, 0, 0, 8]),          # negative destination page id
    ([7, 1], [-1, 1], [0, 0, 0, 0, 0, 4]),          # both bad: destination first
    ([0], [0, 1], [0, 0, 0, 0, 0, 8]),              # source table too short
    ([0, 1], [0, 1], [0, 1, 0, 0, 0, 8]),           # destination table too short
    ([0, 1], [0, 1], [0, 0, 0, 0, 0, -1]),          # negative count
    ([0, 1], [0, 1], [0, 0, 0, 2**31 - 2, 0, 3]),   # end beyond 2^31 - 1
    ([0, 1, 2, 3], [2, 0, 1, 3], [0, 0, 0, 3, 6, 9]),
])
def test_device_errors(test_lib, src_pt, dst_pt, row):
    check(_err_wl(src_pt, dst_pt, [row, [0, 0, 0, 0, 0, 2]]), test_lib)


@pytest.mark.parametrize("group", [1, 2, 3, 5])
@pytest.mark.parametrize("with_slice", [False, True])
def test_layered(test_lib, group, with_slice):
    """kvx_transfer_layered_planned: one sweep launch per layer group."""
    if with_slice:
        wl = cases.slice_case("LPCTHD", "PLCHTD", 4, 8, (5, 2, 4), (4, 2, 2),
                              (1, 0, 4, 0, 0, 2, 2, 0, 2), seed=group)
    else:
        wl = cases.transfer_case("LPCHTD", "LPCTHD", 16, 32, seed=group, L=5)
    wl.steps[0].layer_group = group
    check(wl, test_lib)


@pytest.mark.parametrize("seed", range(12))
def test_random_layered_cases(test_lib, seed):
    check(cases.random_layered_case(seed), test_lib, list(TOKENS)[seed % len(TOKENS)])


def test_layered_plan_that_disagrees_is_reported(test_lib):
    import torch
    from paper_2606_31093_amd import kvx
    wl = cases.transfer_case("LPCTHD", "LPCTHD", 4, 8, seed=23, L=4)
    st = wl.steps[0]
    S, D = wl.sides["A"], wl.sides["B"]
    init = initial_bytes(wl)
    a, b = torch.from_numpy(init["A"]).cuda(), torch.from_numpy(init["B"]).cuda()
    buf, pages, tokens = kvx.host_plan(st.reqs, S.T, D.T)
    kvx.plan_slots(buf, len(st.reqs))[1, 2] += 1          # one slot's first destination slot
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    events = [torch.cuda.Event() for _ in range(2)]
    kvx.kvx_transfer_layered_planned(a, S, b, D, kvx.device_table(st.src_pt), kvx.device_table(st.dst_pt),
                                     kvx.device_reqs(st.reqs), 2, events, torch.from_numpy(buf).cuda(),
                                     pages, tokens, None, err, library=test_lib)
    torch.cuda.synchronize()
    assert int(err.item()) & kvx.DERR_BAD_PLAN
    assert all(ev.query() for ev in events)


def test_many_records(test_lib):
    """300 records, some empty."""
    spec = [(i % 5, (i * 3) % 7, 0 if i % 17 == 0 else 1 + (i * 13) % 40, None) for i in range(300)]
    check(cases.transfer_case("LPCTHD", "PLCTHD", 16, 8, seed=5, spec=spec), test_lib)


def _bad_plan_run(library, alter, wl=None):
    """One planned transfer with the plan changed by ``alter(buf, pages,
    n_reqs)`` -> (buf, pages); returns the device error bits."""
    import torch
    from paper_2606_31093_amd import kvx
    wl = wl or cases.transfer_case("LPCTHD", "LPCTHD", 4, 8, seed=21)
    st = wl.steps[0]
    S, D = wl.sides["A"], wl.sides["B"]
    init = initial_bytes(wl)
    a = torch.from_numpy(init["A"]).cuda()
    b = torch.from_numpy(init["B"]).cuda()
    spt, dpt, reqs = kvx.device_table(st.src_pt), kvx.device_table(st.dst_pt), kvx.device_reqs(st.reqs)
    buf, pages, tokens = kvx.host_plan(st.reqs, S.T, D.T)
    assert pages >= 4
    buf, pages = alter(buf.copy(), pages, len(st.reqs))
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    kvx.kvx_transfer_planned(a, S, b, D, spt, dpt, reqs, torch.from_numpy(buf).cuda(), pages, tokens,
                             None, err, library=library)
    torch.cuda.synchronize()
    return int(err.item())


def _slot_field(k, delta):
    def alter(buf, pages, n):
        kvx_slots(buf, n)[pages // 2, k] += delta
        return buf, pages
    return alter


def kvx_slots(buf, n):
    from paper_2606_31093_amd import kvx
    return kvx.plan_slots(buf, n)


BAD_PLANS = {
    "fewer pages": lambda buf, pages, n: (buf, pages - 1),
    "more pages": lambda buf, pages, n: (np.concatenate([buf, buf[n + 1:n + 5]]), pages + 1),
    "prefix + 1": lambda buf, pages, n: (np.concatenate([buf[:n + 1] + 1, buf[n + 1:]]), pages),
    "prefix reversed": lambda buf, pages, n: (np.concatenate([buf[:n + 1][::-1], buf[n + 1:]]), pages),
    "dst_idx": _slot_field(0, 1), "src_idx": _slot_field(1, -1), "dst_slot": _slot_field(2, 1),
    "n_tokens": _slot_field(3, -1), "src_slot": _slot_field(4, 1), "req": _slot_field(5, 1),
    "slots swapped": lambda buf, pages, n: (np.concatenate(
        [buf[:n + 1], np.roll(buf[n + 1:].reshape(pages, 4), 1, axis=0).ravel()]), pages),
}


@pytest.mark.parametrize("how", list(BAD_PLANS))
def test_plan_that_disagrees_is_reported(test_lib, how):
    from paper_2606_31093_amd import kvx
    assert _bad_plan_run(test_lib, BAD_PLANS[how]) & kvx.DERR_BAD_PLAN


def test_plan_of_other_page_sizes_is_reported(test_lib):
    """A plan built for 8-token source pages used on 4-token ones."""
    import torch
    from paper_2606_31093_amd import kvx
    wl = cases.transfer_case("LPCTHD", "LPCTHD", 4, 8, seed=22)
    st = wl.steps[0]
    S, D = wl.sides["A"], wl.sides["B"]
    init = initial_bytes(wl)
    a, b = torch.from_numpy(init["A"]).cuda(), torch.from_numpy(init["B"]).cuda()
    buf, pages, tokens = kvx.host_plan(st.reqs, 8, D.T)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    kvx.kvx_transfer_planned(a, S, b, D, kvx.device_table(st.src_pt), kvx.device_table(st.dst_pt),
                             kvx.device_reqs(st.reqs), torch.from_numpy(buf).cuda(), pages, tokens,
                             None, err, library=test_lib)
    torch.cuda.synchronize()
    assert int(err.item()) & kvx.DERR_BAD_PLAN


@pytest.mark.parametrize("seed", range(4))
def test_random_slots_stay_in_bounds(test_lib, seed):
    """Slots of random words: reported, and every access stays inside the
    pools and tables (the slot fields are range-checked before use)."""
    from paper_2606_31093_amd import kvx
    rng = np.random.default_rng(seed)

    def alter(buf, pages, n):
        words = kvx_slots(buf, n)
        small = rng.integers(-3, 12, size=words.shape)
        huge = rng.integers(-2**31, 2**31 - 1, size=words.shape)
        words[:] = np.where(rng.random(words.shape) < 0.8, small, huge).astype(np.int32)
        return buf, pages

    assert _bad_plan_run(test_lib, alter) & kvx.DERR_BAD_PLAN


@pytest.mark.parametrize("seed", range(20))
def test_random_medium_cases(test_lib, seed):
    """Medium transfers with 128-256 KiB token-major destination pages,
    through the product library (which sweeps them) and the test build."""
    wl = cases.random_planned_medium_case(seed)
    check(wl, None)
    check(wl, test_lib)


def test_graph_replays_of_the_product_sweep():
    """A planned transfer the product library sweeps (256 KiB pages),
    captured in a HIP graph and replayed three times with eager work in
    between, gives the oracle's bytes and no error bit every time."""
    import torch
    from paper_2606_31093_amd import kvx
    spec = [(0, 0, 200, None), (5, 70, 333, None), (63, 1, 1, None), (10, 64, 128, 0)]
    wl = cases.transfer_case("LPCTHD", "PLCTHD", 64, 64, seed=31, e=2, D=128, L=3, C=2, H=8, spec=spec)
    st = wl.steps[0]
    S, D = wl.sides["A"], wl.sides["B"]
    init = initial_bytes(wl)
    want, _ = run_oracle(wl, init)
    a, b = torch.from_numpy(init["A"]).cuda(), torch.from_numpy(init["B"]).cuda()
    b0 = b.clone()
    spt, dpt, reqs = kvx.device_table(st.src_pt), kvx.device_table(st.dst_pt), kvx.device_reqs(st.reqs)
    plan, pages, tokens = kvx.device_plan(st.reqs, S.T, D.T)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        kvx.kvx_transfer_planned(a, S, b, D, spt, dpt, reqs, plan, pages, tokens, None, err, stream=s)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        kvx.kvx_transfer_planned(a, S, b, D, spt, dpt, reqs, plan, pages, tokens, None, err)
    for _ in range(3):
        b.copy_(b0)                    # eager work between replays
        err.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert int(err.item()) == 0
        assert np.array_equal(b.cpu().numpy(), want["B"])


@pytest.mark.parametrize("tokens", ["true", "double"])
@pytest.mark.parametrize("ls,ld", [("LPCTHD", "LPCTHD"), ("PLCHTD", "PLCTHD"), ("LPCTHD", "PLCHTD")])
def test_product_library_sweeps_large_tiles(ls, ld, tokens):
    """256 KiB pages (2 kv x 64 tokens x 8 heads x 256-byte rows): the product
    library itself takes the sweep, into token-major and head-major
    destinations."""
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    spec = [(0, 0, 200, None), (5, 70, 333, None), (63, 1, 1, None), (0, 0, 0, None), (10, 64, 128, 0)]
    wl = cases.transfer_case(ls, ld, 64, 64, seed=17, e=2, D=128, L=3, C=2, H=8, spec=spec)
    check(wl, None, tokens)
