"""Chained page hashes on the GPU against the CPU oracle, word for word."""
import numpy as np
import pytest

from paper_2606_31093_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_31093_amd import kvx
    kvx.lib()
    return torch


def _both(torch, payload, rec_bytes, T, rows, out_len, raw=None, library=None):
    from oracle import kvx_oracle
    from paper_2606_31093_amd import kvx
    want = np.full(out_len, 0x5A5A, np.uint64)
    werr = kvx_oracle.default().page_hashes(payload, rec_bytes, T, rows, want)
    p = torch.from_numpy(np.ascontiguousarray(payload).view(np.uint8).reshape(-1).copy()).cuda()
    out = torch.full((out_len,), 0x5A5A, dtype=torch.int64, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    recs = raw if raw is not None else kvx.pack_hash_reqs(rows)
    reqs = torch.from_numpy(recs.view(np.uint8).copy()).cuda()
    kvx.kvx_page_hashes(p, rec_bytes, T, reqs, out, err, library=library)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint64)
    return got, int(err.item()), want, werr


def test_small_workload(torch):
    wl = W.page_hash(small=True)
    pay = W.hash_payload(wl)
    got, gerr, want, werr = _both(torch, pay, wl.rec_bytes, wl.T, wl.rows, wl.out_len)
    assert gerr == werr == 0
    assert np.array_equal(got, want)


@pytest.mark.parametrize("rec_bytes", [4, 8, 12, 64])
@pytest.mark.parametrize("T", [1, 3, 16, 64, 1000])
def test_shapes(torch, rec_bytes, T):
    rng = np.random.default_rng(rec_bytes * 1000 + T)
    lengths = [0, 1, T - 1 if T > 1 else 2, T, T + 1, 5 * T + 3, 777]
    rows, pos, out = [], 0, 0
    for i, n in enumerate(lengths):
        rows.append((pos, out, int(rng.integers(0, 2**63)) if i % 2 else 0, n))
        pos += n
        out += -(-n // T)
    pay = rng.integers(0, 2**31, size=pos * rec_bytes // 4, dtype=np.int32)
    got, gerr, want, werr = _both(torch, pay, rec_bytes, T, rows, out + 3)
    assert gerr == werr == 0
    assert np.array_equal(got, want)


def test_record_errors(torch):
    pay = np.arange(40, dtype=np.int32)
    rows = [(0, 0, 0, 40), (0, 4, 0, 41), (-1, 10, 0, 4), (0, 12, 0, -1), (30, 20, 0, 10)]
    got, gerr, want, werr = _both(torch, pay, 4, 10, rows, 22)
    assert gerr == werr == 8
    assert np.array_equal(got, want)
    from paper_2606_31093_amd import kvx
    recs = kvx.pack_hash_reqs([(0, 0, 0, 40)])
    recs["reserved"][0] = 1
    got, gerr, _, _ = _both(torch, pay, 4, 10, [], 4, raw=recs)
    assert gerr == 8 and (got == 0x5A5A).all()


def test_full_workload(torch):
    wl = W.page_hash()
    pay = W.hash_payload(wl)
    print(f"{wl.title}: {wl.positions} positions, {wl.out_len} pages", flush=True)
    got, gerr, want, werr = _both(torch, pay, wl.rec_bytes, wl.T, wl.rows, wl.out_len)
    assert gerr == werr == 0
    assert np.array_equal(got, want)


def test_chain_lengths_and_scattered_outputs(torch):
    """Page counts around every multiple of the chain's and the digest's
    batches (16 digests, 64 pages), 300 requests so that the chain spans
    several wavefronts with lanes of very different lengths, outputs placed
    in a shuffled order with gaps, and requests that reread the same
    payload."""
    rng = np.random.default_rng(77)
    T = 4
    pages = [1, 15, 16, 17, 31, 32, 33, 63, 64, 65, 127, 128, 129, 200]
    pages = pages + [int(p) for p in rng.integers(0, 150, size=300 - len(pages))]
    n = [max(0, p * T - int(rng.integers(0, T))) if p else 0 for p in pages]
    slots = rng.permutation(len(n))
    out_offs, cursor = [0] * len(n), 5
    for i in slots:                      # outputs in a shuffled order, with gaps
        out_offs[i] = cursor
        cursor += -(-n[i] // T) + int(rng.integers(0, 3))
    total = sum(n)
    rows = []
    for i, k in enumerate(n):
        off = int(rng.integers(0, total - k + 1)) if i % 3 == 0 else sum(n[:i])
        rows.append((off, out_offs[i], int(rng.integers(0, 2**63)) if i % 4 else 0, k))
    pay = rng.integers(0, 2**31, size=total, dtype=np.int32)
    got, gerr, want, werr = _both(torch, pay, 4, T, rows, cursor + 7)
    assert gerr == werr == 0
    assert np.array_equal(got, want)


def _random_hash_case(seed):
    rng = np.random.default_rng(30_000 + seed)
    rec_bytes = int(rng.choice([4, 8, 12, 16, 40]))
    T = int(rng.choice([1, 2, 3, 7, 16, 64, 100]))
    nreq = int(rng.integers(1, 40))
    n = [0 if rng.random() < 0.1 else int(rng.integers(1, 6 * T + 10)) for _ in range(nreq)]
    positions = max(1, sum(n) // 2 + max(n))
    rows, out = [], int(rng.integers(0, 4))
    for k in n:
        off = int(rng.integers(0, positions - k + 1))      # payload ranges may overlap
        seed_v = int(rng.integers(0, 2**63)) if rng.random() < 0.4 else 0
        rows.append((off, out, seed_v, k))
        out += -(-k // T) + int(rng.integers(0, 3))
    out_len = out + int(rng.integers(0, 3))
    if rng.random() < 0.2:                                   # a malformed record
        r = int(rng.integers(nreq))
        po, oo, sv, k = rows[r]
        rows[r] = rng.choice([(po, oo, sv, -1), (positions, oo, sv, k + 1), (po, out_len, sv, k + T)])
        rows[r] = tuple(int(x) for x in rows[r])
    pay = rng.integers(0, 2**31, size=positions * rec_bytes // 4, dtype=np.int32)
    return pay, rec_bytes, T, rows, out_len


@pytest.mark.parametrize("seed", range(50))
def test_random_hash_cases(torch, seed):
    pay, rec_bytes, T, rows, out_len = _random_hash_case(seed)
    got, gerr, want, werr = _both(torch, pay, rec_bytes, T, rows, out_len)
    assert gerr == werr
    assert np.array_equal(got, want)


def _rows_for(n, T, rng, seeded=0.3):
    rows, pos, out = [], 0, 0
    for k in n:
        seed_v = int(rng.integers(0, 2**63)) if rng.random() < seeded else 0
        rows.append((pos, out, seed_v, int(k)))
        pos += int(k)
        out += -(-int(k) // T)
    return rows, pos, out


def test_more_requests_than_one_group_per_compute_unit(torch):
    """20000 requests: 64 per group, more groups than workgroups, so each
    workgroup takes several groups in turn and reuses its shared state."""
    rng = np.random.default_rng(91)
    T = 4
    n = rng.integers(0, 3 * T + 2, size=20000)
    rows, pos, out = _rows_for(n, T, rng)
    pay = rng.integers(0, 2**31, size=max(pos, 1), dtype=np.int32)
    got, gerr, want, werr = _both(torch, pay, 4, T, rows, out)
    assert gerr == werr == 0
    assert np.array_equal(got, want)


def test_maximum_request_count(torch):
    """KVX_MAX_REQS (65536) records of 0-2 pages in one call."""
    rng = np.random.default_rng(92)
    T = 2
    n = rng.integers(0, 2 * T + 1, size=65536)
    rows, pos, out = _rows_for(n, T, rng)
    pay = rng.integers(0, 2**31, size=max(pos, 1), dtype=np.int32)
    got, gerr, want, werr = _both(torch, pay, 4, T, rows, out)
    assert gerr == werr == 0
    assert np.array_equal(got, want)


@pytest.mark.parametrize("case", ["all_empty", "equal_lengths", "one_long", "ladder"])
def test_group_shapes(torch, case):
    """Groups whose page counts are all zero, all equal (ties in the order
    the pages are handed out), one long request among one-page ones, and a
    ladder of distinct lengths."""
    rng = np.random.default_rng(len(case))
    T = 8
    nreq = 700                                  # 3 requests per group on 256 compute units
    if case == "all_empty":
        n = np.zeros(nreq, int)
    elif case == "equal_lengths":
        n = np.full(nreq, 5 * T)
    elif case == "one_long":
        n = np.full(nreq, 1)
        n[::97] = 3000 * T
    else:
        n = np.arange(nreq) % 70 * T + np.arange(nreq) % 3
    rows, pos, out = _rows_for(n, T, rng)
    pay = rng.integers(0, 2**31, size=max(pos, 1), dtype=np.int32)
    got, gerr, want, werr = _both(torch, pay, 4, T, rows, out + 1)
    assert gerr == werr == 0
    assert np.array_equal(got, want)


@pytest.mark.parametrize("where", ["payload", "out", "both"])
def test_pinned_host_payload_and_output(torch, where):
    """Token ids and/or the output words in pinned host memory, read and
    written over PCIe: digests arrive far more slowly, so the chain side
    waits on them much longer than with device memory."""
    from oracle import kvx_oracle
    from paper_2606_31093_amd import kvx
    rng = np.random.default_rng(len(where) + 500)
    T = 16
    n = rng.integers(1, 40 * T, size=300)
    rows, pos, out_len = _rows_for(n, T, rng)
    pay = rng.integers(0, 2**31, size=pos, dtype=np.int32)
    want = np.zeros(out_len, np.uint64)
    assert kvx_oracle.default().page_hashes(pay, 4, T, rows, want) == 0
    host_pay = where in ("payload", "both")
    host_out = where in ("out", "both")
    p = torch.from_numpy(pay.view(np.uint8).copy())
    p = p.pin_memory() if host_pay else p.cuda()
    out = torch.zeros(out_len, dtype=torch.int64, pin_memory=True) if host_out else \
        torch.zeros(out_len, dtype=torch.int64, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    kvx.kvx_page_hashes(p, 4, T, kvx.device_hash_reqs(rows), out, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    assert np.array_equal(out.cpu().numpy().view(np.uint64), want)


def test_chain_wait_gives_up_cleanly(torch):
    """The test build of the library bounds the chain's wait at one empty
    poll: the chain stops before the first digests exist, the kernel still
    finishes, raises KVX_DERR_STALLED and leaves the outputs incomplete.  The
    next call, through the product library with its normal bound, is exact."""
    from paper_2606_31093_amd import build_lib, kvx
    stall = kvx.load(build_lib.TEST_LIBRARY)
    wl = W.page_hash(small=True)
    pay = W.hash_payload(wl)
    got, gerr, want, werr = _both(torch, pay, wl.rec_bytes, wl.T, wl.rows, wl.out_len,
                                  library=stall)
    assert werr == 0
    assert gerr & kvx.DERR_STALLED
    assert not np.array_equal(got, want)
    got, gerr, want, werr = _both(torch, pay, wl.rec_bytes, wl.T, wl.rows, wl.out_len)
    assert gerr == werr == 0
    assert np.array_equal(got, want)


def test_graph_replays_match_eager(torch):
    """The hash kernel captured in a HIP graph and replayed several times,
    with the output cleared eagerly in between, gives the oracle's words
    every time."""
    from paper_2606_31093_amd import kvx
    from oracle import kvx_oracle
    wl = W.page_hash(small=True)
    pay = W.hash_payload(wl)
    want = np.zeros(wl.out_len, np.uint64)
    assert kvx_oracle.default().page_hashes(pay, wl.rec_bytes, wl.T, wl.rows, want) == 0
    p = torch.from_numpy(pay.view(np.uint8).copy()).cuda()
    reqs = kvx.device_hash_reqs(wl.rows)
    out = torch.zeros(wl.out_len, dtype=torch.int64, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        kvx.kvx_page_hashes(p, wl.rec_bytes, wl.T, reqs, out, err, stream=s)      # warm up
    torch.cuda.current_stream().wait_stream(s)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        kvx.kvx_page_hashes(p, wl.rec_bytes, wl.T, reqs, out, err)
    for _ in range(3):
        out.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert int(err.item()) == 0
        assert np.array_equal(out.cpu().numpy().view(np.uint64), want)
