"""Where the library's inputs may live, on the GPU: page tables, request
records and plans in pinned host memory (read over PCIe by the kernel), the
error word refused in pinned host memory, and descriptors larger than their
allocation refused on the host before anything is enqueued."""
import ctypes

import numpy as np
import pytest

from paper_2606_31093_amd.workloads import BufSpec, PoolSpec, Step, get
from runner import assert_same, initial_bytes, run_oracle

pytestmark = pytest.mark.gpu

MiB = 1 << 20


@pytest.fixture(scope="module")
def torch():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_31093_amd import kvx
    kvx.lib()
    return torch


def _pinned(torch, arr):
    t = torch.empty(arr.nbytes, dtype=torch.uint8, pin_memory=True)
    t.copy_(torch.from_numpy(np.ascontiguousarray(arr).view(np.uint8).reshape(-1)))
    return t


@pytest.mark.parametrize("name", ["handoff", "relayout", "small_requests"])
def test_tables_and_records_in_pinned_host_memory(torch, name):
    """Page tables and records read by the kernel from pinned host memory
    give the oracle's bytes; one damaged page id raises its bit in the
    device error word."""
    from paper_2606_31093_amd import kvx
    wl = get(name, small=True)
    st = wl.steps[0]
    src_pt = st.src_pt.copy()
    src_pt[1] = 1 << 20                          # out of range: position of page 1 skipped
    wl.steps[0] = Step(st.op, st.src, st.dst, src_pt, st.dst_pt, st.reqs, st.slice)
    init = initial_bytes(wl)
    want, werr = run_oracle(wl, init)
    assert werr == [kvx.DERR_SRC_PAGE]
    S, D = wl.sides["A"], wl.sides["B"]
    a = torch.from_numpy(init["A"]).cuda()
    b = torch.from_numpy(init["B"]).cuda()
    spt = _pinned(torch, src_pt.astype(np.int32)).view(torch.int32)
    dpt = _pinned(torch, st.dst_pt.astype(np.int32)).view(torch.int32)
    reqs = _pinned(torch, kvx.pack_reqs(st.reqs))
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    kvx.kvx_transfer(a, S, b, D, spt, dpt, reqs, err)
    torch.cuda.synchronize()
    assert int(err.item()) == kvx.DERR_SRC_PAGE
    assert_same({"B": b.cpu().numpy()}, {"B": want["B"]}, wl.title)


@pytest.mark.parametrize("build", ["product", "test"])
def test_plan_tables_and_records_in_pinned_host_memory(torch, build):
    """A planned transfer whose plan, page tables and records are all in
    pinned host memory gives the oracle's bytes.  256 KiB pages into a
    token-major destination, so the product library takes the sweep; the
    test build sweeps with a capped grid, looping over page slots."""
    import cases
    from paper_2606_31093_amd import build_lib, kvx
    library = kvx.load(build_lib.TEST_LIBRARY) if build == "test" else None
    spec = [(0, 0, 200, None), (5, 70, 333, None), (63, 1, 1, None), (0, 0, 0, None), (10, 64, 128, 0)]
    wl = cases.transfer_case("LPCTHD", "PLCTHD", 64, 64, seed=29, e=2, D=128, L=3, C=2, H=8, spec=spec)
    st = wl.steps[0]
    S, D = wl.sides["A"], wl.sides["B"]
    init = initial_bytes(wl)
    want, werr = run_oracle(wl, init)
    assert werr == [0]
    a = torch.from_numpy(init["A"]).cuda()
    b = torch.from_numpy(init["B"]).cuda()
    buf, pages, tokens = kvx.host_plan(st.reqs, S.T, D.T)
    plan = _pinned(torch, buf)
    spt = _pinned(torch, st.src_pt.astype(np.int32)).view(torch.int32)
    dpt = _pinned(torch, st.dst_pt.astype(np.int32)).view(torch.int32)
    reqs = _pinned(torch, kvx.pack_reqs(st.reqs))
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    kvx.kvx_transfer_planned(a, S, b, D, spt, dpt, reqs, plan, pages, tokens, None, err, library=library)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    assert_same({"B": b.cpu().numpy()}, {"B": want["B"]}, wl.title)


def test_gather_scatter_tables_in_pinned_host_memory(torch):
    from paper_2606_31093_amd import kvx
    wl = get("host_tier", small=True)
    g, s = wl.steps
    init = initial_bytes(wl)
    want, werr = run_oracle(wl, init)
    assert werr == [0, 0]
    S, B = wl.sides["A"], wl.sides["buf"]
    a = torch.from_numpy(init["A"]).cuda()
    buf = torch.from_numpy(init["buf"]).cuda()
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    # the host blocks must stay allocated until the kernels have read them
    g_pt = _pinned(torch, g.src_pt.astype(np.int32)).view(torch.int32)
    g_reqs = _pinned(torch, kvx.pack_reqs(g.reqs))
    s_pt = _pinned(torch, s.dst_pt.astype(np.int32)).view(torch.int32)
    s_reqs = _pinned(torch, kvx.pack_reqs(s.reqs))
    kvx.kvx_gather(a, S, buf, B, g_pt, g_reqs, err)
    kvx.kvx_scatter(buf, B, a, S, s_pt, s_reqs, err)
    torch.cuda.synchronize()
    del g_pt, g_reqs, s_pt, s_reqs
    assert int(err.item()) == 0
    assert_same({"A": a.cpu().numpy(), "buf": buf.cpu().numpy()},
                {"A": want["A"], "buf": want["buf"]}, wl.title)


def test_error_word_in_pinned_host_memory_is_refused(torch):
    from paper_2606_31093_amd import kvx
    wl = get("handoff", small=True)
    st = wl.steps[0]
    S, D = wl.sides["A"], wl.sides["B"]
    a = torch.zeros(S.nbytes, dtype=torch.uint8, device="cuda")
    b = torch.zeros(D.nbytes, dtype=torch.uint8, device="cuda")
    host_err = torch.zeros(1, dtype=torch.int32, pin_memory=True)
    with pytest.raises(kvx.KvxError) as ei:
        kvx.kvx_transfer(a, S, b, D, kvx.device_table(st.src_pt), kvx.device_table(st.dst_pt),
                         kvx.device_reqs(st.reqs), host_err)
    assert ei.value.status == -5 and "dev_err" in str(ei.value)
    torch.cuda.synchronize()
    assert bool((b == 0).all())


# --------------------------------------------------------------------------
# descriptors larger than their allocation (raw addresses through the C ABI,
# so the binding's own size checks do not run first).  Allocations come from
# hipMalloc / hipHostMalloc directly, so their extents are exact.  Every
# refused call is built so that, were it not refused, the kernel would still
# touch only bytes inside the real allocations.
# --------------------------------------------------------------------------

def _hip():
    """The HIP runtime torch loaded (the same object, found by path)."""
    import torch  # noqa: F401
    path = None
    with open("/proc/self/maps") as f:
        for line in f:
            if "libamdhip64.so" in line:
                path = line.split()[-1]
                break
    assert path, "no HIP runtime mapped"
    L = ctypes.CDLL(path)
    vp, sz = ctypes.c_void_p, ctypes.c_size_t
    L.hipMalloc.argtypes = [ctypes.POINTER(vp), sz]
    L.hipHostMalloc.argtypes = [ctypes.POINTER(vp), sz, ctypes.c_uint]
    L.hipFree.argtypes = [vp]
    L.hipHostFree.argtypes = [vp]
    L.hipMemset.argtypes = [vp, ctypes.c_int, sz]
    L.hipMemcpy.argtypes = [vp, vp, sz, ctypes.c_int]
    return L


class _Alloc:
    def __init__(self, hip, nbytes, host=False):
        self.hip, self.host, self.ptr = hip, host, ctypes.c_void_p()
        rc = (hip.hipHostMalloc(ctypes.byref(self.ptr), nbytes, 0) if host
              else hip.hipMalloc(ctypes.byref(self.ptr), nbytes))
        assert rc == 0, f"allocation of {nbytes} bytes failed ({rc})"
        if not host:
            assert hip.hipMemset(self.ptr, 0, nbytes) == 0
        else:
            ctypes.memset(self.ptr, 0, nbytes)
        self.addr = self.ptr.value

    def free(self):
        (self.hip.hipHostFree if self.host else self.hip.hipFree)(self.ptr)


def _upload(hip, arr):
    raw = np.ascontiguousarray(arr).view(np.uint8).reshape(-1)
    a = _Alloc(hip, max(raw.nbytes, 16))
    assert hip.hipMemcpy(ctypes.c_void_p(a.addr), raw.ctypes.data_as(ctypes.c_void_p), raw.nbytes,
                         1) == 0     # host to device
    return a


def _raw_transfer(S, a_ptr, D, b_ptr, spt_ptr, spt_len, dpt_ptr, dpt_len, reqs_ptr, n_reqs,
                  err_ptr):
    from paper_2606_31093_amd import kvx
    return kvx.lib().kvx_transfer(ctypes.byref(kvx.pool_desc(S, a_ptr)),
                                  ctypes.byref(kvx.pool_desc(D, b_ptr)), spt_ptr, spt_len,
                                  dpt_ptr, dpt_len, reqs_ptr, n_reqs, err_ptr, None)


def test_descriptors_beyond_their_allocation_are_refused(torch):
    """A pool or page table that claims more bytes than the allocation around
    its pointer holds is refused with KVX_ERR_RANGE; the same call with sizes
    that fit succeeds.  The request touches pages 0-3 (1 MiB) and table
    entries 0-3 only."""
    from paper_2606_31093_amd import kvx
    hip = _hip()
    S = PoolSpec(1, 2, 8, 128, T=64, N=32, e=2, layout="LPCTHD")       # 8 MiB
    big = PoolSpec(1, 2, 8, 128, T=64, N=32 * 64, e=2, layout="LPCTHD")  # 512 MiB claimed
    a, b = _Alloc(hip, S.nbytes), _Alloc(hip, S.nbytes)
    pt = _upload(hip, np.arange(4, dtype=np.int32))
    reqs = _upload(hip, kvx.pack_reqs([[0, 0, 0, 0, 0, 256]]))
    err = _Alloc(hip, 4)
    A, B, P, R, E = a.addr, b.addr, pt.addr, reqs.addr, err.addr
    try:
        assert _raw_transfer(S, A, S, B, P, 4, P, 4, R, 1, E) == 0
        torch.cuda.synchronize()
        cases = [
            ((big, A, S, B, P, 4, P, 4, R, 1, E), "src base"),
            ((S, A, big, B, P, 4, P, 4, R, 1, E), "dst base"),
            ((S, A + S.nbytes // 2, S, B, P, 4, P, 4, R, 1, E), "src base"),   # from mid-allocation
            ((S, A, S, B, P, 1 << 24, P, 4, R, 1, E), "src_pt"),
            ((S, A, S, B, P, 4, P, 1 << 24, R, 1, E), "dst_pt"),
        ]
        for args, name in cases:
            assert _raw_transfer(*args) == -5, name
            assert name in kvx.kvx_last_error() and "needs" in kvx.kvx_last_error()
        torch.cuda.synchronize()
        word = np.zeros(1, np.uint32)
        assert hip.hipMemcpy(word.ctypes.data_as(ctypes.c_void_p), ctypes.c_void_p(E), 4, 2) == 0
        assert int(word[0]) == 0
    finally:
        for x in (a, b, pt, reqs, err):
            x.free()


def test_plan_beyond_its_allocation_is_refused(torch):
    """A plan whose page count needs more bytes than its allocation holds is
    refused with KVX_ERR_RANGE; the exact plan succeeds."""
    from paper_2606_31093_amd import kvx
    hip = _hip()
    S = PoolSpec(1, 2, 8, 128, T=64, N=32, e=2, layout="LPCTHD")       # 8 MiB
    rows = [[0, 0, 0, 0, 0, 256]]
    buf, pages, tokens = kvx.host_plan(rows, S.T, S.T)
    a, b = _Alloc(hip, S.nbytes), _Alloc(hip, S.nbytes)
    pt = _upload(hip, np.arange(4, dtype=np.int32))
    reqs = _upload(hip, kvx.pack_reqs(rows))
    plan = _upload(hip, buf)
    err = _Alloc(hip, 4)
    assert buf.nbytes == kvx.plan_bytes(1, pages) and buf.nbytes % 16 == 0

    def call(n_pages):
        return kvx.lib().kvx_transfer_planned(ctypes.byref(kvx.pool_desc(S, a.addr)),
                                              ctypes.byref(kvx.pool_desc(S, b.addr)), None, pt.addr, 4,
                                              pt.addr, 4, reqs.addr, 1, plan.addr, n_pages, tokens, err.addr,
                                              None)
    try:
        assert call(pages) == 0
        torch.cuda.synchronize()
        assert call(pages + (1 << 20)) == -5                       # 32 MiB past a 144-byte plan
        assert "plan" in kvx.kvx_last_error() and "needs" in kvx.kvx_last_error()
        torch.cuda.synchronize()
    finally:
        for x in (a, b, pt, reqs, plan, err):
            x.free()


@pytest.mark.parametrize("host", [False, True], ids=["device_buffer", "pinned_host_buffer"])
def test_buffer_beyond_its_allocation_is_refused(torch, host):
    """A gather whose buffer descriptor claims 256 MiB of a 4 MiB allocation
    is refused, in device memory and in pinned host memory; the request's
    block (256 KiB) lies inside the allocation either way."""
    from paper_2606_31093_amd import kvx
    hip = _hip()
    S = PoolSpec(1, 2, 8, 128, T=64, N=32, e=2, layout="LPCTHD")
    a = _Alloc(hip, S.nbytes)
    buf = _Alloc(hip, 4 * MiB, host=host)
    pt = _upload(hip, np.arange(4, dtype=np.int32))
    reqs = _upload(hip, kvx.pack_reqs([[0, 0, 0, 0, 0, 64]]))
    err = _Alloc(hip, 4)

    def gather(cap_bytes):
        B = BufSpec(1, 2, 8, 128, 2, cap=cap_bytes // 2)
        return kvx.lib().kvx_gather(ctypes.byref(kvx.pool_desc(S, a.addr)),
                                    ctypes.byref(kvx.buf_desc(B, buf.addr)), pt.addr, 4,
                                    reqs.addr, 1, err.addr, None)

    try:
        assert gather(4 * MiB) == 0
        torch.cuda.synchronize()
        assert gather(256 * MiB) == -5
        assert "dst base" in kvx.kvx_last_error()
        torch.cuda.synchronize()
    finally:
        for x in (a, buf, pt, reqs, err):
            x.free()
