"""The C-ABI boundary on the CPU: the library loads and exports every
function include/kvx.h declares; the Python structures match the C layout;
host-side validation returns the documented status for each kind of bad
argument without touching a GPU; the launch-constant division is exact."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2606_31093_amd import build_lib, kvx
from paper_2606_31093_amd.workloads import BufSpec, PoolSpec

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kvx.h")


@pytest.fixture(scope="module")
def lib():
    if build_lib.is_stale():
        build_lib.build()
    return kvx.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^[A-Za-z_][\w \*]*?\b(kvx_\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("kvx_transfer", "kvx_gather", "kvx_scatter", "kvx_pool_bytes", "kvx_strerror",
              "kvx_last_error", "kvx_abi_version"):
        assert n in names


def test_library_exports_every_declared_function(lib):
    for name in declared_functions():
        assert hasattr(lib, name), f"{name} declared in kvx.h but not exported"
    out = subprocess.run(["nm", "-D", "--defined-only", build_lib.LIBRARY], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\b(kvx_\w+)$", out, flags=re.M))
    assert set(declared_functions()) <= exported


def test_abi_version(lib):
    m = re.search(r"#define KVX_ABI_VERSION (\d+)", open(HEADER).read())
    assert kvx.kvx_abi_version() == int(m.group(1))


def test_struct_layout_matches_c(tmp_path):
    """sizeof/offsetof from a C compiler against the ctypes/numpy mirrors."""
    src = tmp_path / "layout.c"
    src.write_text(r'''
#include <stddef.h>
#include <stdio.h>
#include "kvx.h"
#define F(T, f) printf(#T "." #f " %zu\n", offsetof(T, f))
int main(void) {
  printf("kvx_pool %zu\nkvx_buf %zu\nkvx_req %zu\n", sizeof(kvx_pool), sizeof(kvx_buf), sizeof(kvx_req));
  F(kvx_pool, base); F(kvx_pool, num_layers); F(kvx_pool, num_kv); F(kvx_pool, num_heads);
  F(kvx_pool, head_dim); F(kvx_pool, page_tokens); F(kvx_pool, num_pages); F(kvx_pool, elem_bytes);
  F(kvx_pool, layout);
  F(kvx_buf, base); F(kvx_buf, num_layers); F(kvx_buf, num_kv); F(kvx_buf, num_heads);
  F(kvx_buf, head_dim); F(kvx_buf, elem_bytes); F(kvx_buf, reserved); F(kvx_buf, capacity_elems);
  F(kvx_req, src_pt_off); F(kvx_req, dst_pt_off); F(kvx_req, buf_off); F(kvx_req, src_start);
  F(kvx_req, dst_start); F(kvx_req, n_tokens); F(kvx_req, reserved);
  printf("kvx_slice %zu\n", sizeof(kvx_slice));
  F(kvx_slice, src_layer0); F(kvx_slice, dst_layer0); F(kvx_slice, num_layers);
  F(kvx_slice, src_kv0); F(kvx_slice, dst_kv0); F(kvx_slice, num_kv);
  F(kvx_slice, src_head0); F(kvx_slice, dst_head0); F(kvx_slice, num_heads);
  F(kvx_slice, reserved);
  printf("kvx_hash_req %zu\n", sizeof(kvx_hash_req));
  F(kvx_hash_req, payload_off); F(kvx_hash_req, out_off); F(kvx_hash_req, seed);
  F(kvx_hash_req, n_positions); F(kvx_hash_req, reserved);
  return 0;
}''')
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), "-o", str(exe), str(src)],
                   check=True)
    got = dict(line.rsplit(" ", 1) for line in
               subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")
               if line)
    got = {k: int(v) for k, v in got.items()}
    assert got["kvx_pool"] == ctypes.sizeof(kvx.Pool)
    assert got["kvx_buf"] == ctypes.sizeof(kvx.Buf)
    assert got["kvx_req"] == kvx.REQ_DTYPE.itemsize
    for name, _ in kvx.Pool._fields_:
        assert got[f"kvx_pool.{name}"] == getattr(kvx.Pool, name).offset
    for name, _ in kvx.Buf._fields_:
        assert got[f"kvx_buf.{name}"] == getattr(kvx.Buf, name).offset
    for name in kvx.REQ_DTYPE.names:
        assert got[f"kvx_req.{name}"] == kvx.REQ_DTYPE.fields[name][1]
    assert got["kvx_hash_req"] == kvx.HASH_REQ_DTYPE.itemsize
    for name in kvx.HASH_REQ_DTYPE.names:
        assert got[f"kvx_hash_req.{name}"] == kvx.HASH_REQ_DTYPE.fields[name][1]
    assert got["kvx_slice"] == ctypes.sizeof(kvx.Slice)
    for name, _ in kvx.Slice._fields_:
        assert got[f"kvx_slice.{name}"] == getattr(kvx.Slice, name).offset


def test_strerror(lib):
    for status, text in ((0, "success"), (-1, "NULL"), (-2, "shape"), (-3, "aligned"),
                         (-4, "layout"), (-5, "range"), (-6, "HIP"), (-99, "unknown")):
        assert text.lower() in kvx.kvx_strerror(status).lower()


def test_pool_bytes(lib):
    s = PoolSpec(36, 2, 8, 128, T=64, N=4096, e=2, layout="LPCTHD")
    assert kvx.pool_bytes(s) == s.nbytes == 36 * 2**30
    assert kvx.pool_bytes(PoolSpec(1, 3, 1, 8, T=4, N=1)) == -1        # num_kv 3
    assert kvx.pool_bytes(PoolSpec(1, 1, 1, 7, T=4, N=1)) == -1        # 14-byte rows


FAKE = 1 << 20      # a 16-byte aligned address that is never dereferenced


def _call_transfer(S, D, n_reqs=1, src_pt_len=1, dst_pt_len=1, reqs=FAKE, src_pt=FAKE,
                   dst_pt=FAKE, err=None, sbase=FAKE, dbase=FAKE):
    L = kvx.lib()
    sp = kvx.pool_desc(S, sbase)
    dp = kvx.pool_desc(D, dbase)
    return L.kvx_transfer(ctypes.byref(sp), ctypes.byref(dp), src_pt, src_pt_len, dst_pt, dst_pt_len,
                          reqs, n_reqs, err, None)


GOOD = PoolSpec(2, 2, 4, 64, T=16, N=8, e=2, layout="LPCTHD")


@pytest.mark.parametrize("S,D,kw,status", [
    (GOOD, PoolSpec(2, 2, 4, 64, T=16, N=8, e=2, layout="PLCHTD"), dict(n_reqs=0), 0),
    (GOOD, PoolSpec(3, 2, 4, 64, T=16, N=8, e=2), {}, -2),             # layers differ
    (GOOD, PoolSpec(2, 2, 4, 32, T=16, N=8, e=2), {}, -2),             # head_dim differs
    (GOOD, PoolSpec(2, 2, 4, 64, T=16, N=8, e=4), {}, -2),             # elem_bytes differs
    (PoolSpec(2, 3, 4, 64, T=16, N=8), PoolSpec(2, 3, 4, 64, T=16, N=8), {}, -4),   # num_kv 3
    (PoolSpec(2, 2, 4, 64, T=16, N=8, layout=7), GOOD, {}, -4),        # layout 7
    (PoolSpec(2, 2, 4, 4, T=16, N=8), PoolSpec(2, 2, 4, 4, T=16, N=8), {}, -3),     # 8-byte rows
    (PoolSpec(2, 2, 4, 64, T=16, N=8, e=3), PoolSpec(2, 2, 4, 64, T=16, N=8, e=3), {}, -2),
    (PoolSpec(2, 2, 4, 64, T=0, N=8), GOOD, {}, -2),                   # page_tokens 0
    (PoolSpec(2, 2, 4, 64, T=(1 << 20) + 1, N=8), GOOD, {}, -2),       # page_tokens too large
    (PoolSpec(2, 2, 4, 64, T=16, N=0), GOOD, {}, -2),                  # no pages
    (PoolSpec(0, 2, 4, 64, T=16, N=8), PoolSpec(0, 2, 4, 64, T=16, N=8), {}, -2),
    (GOOD, GOOD, dict(sbase=FAKE + 8), -3),                             # misaligned base
    (GOOD, GOOD, dict(dbase=0), -1),                                   # NULL base
    (GOOD, GOOD, dict(reqs=None), -1),                                 # NULL records
    (GOOD, GOOD, dict(reqs=FAKE + 4), -3),                             # misaligned records
    (GOOD, GOOD, dict(n_reqs=-1), -5),
    (GOOD, GOOD, dict(n_reqs=65537), -5),
    (GOOD, GOOD, dict(src_pt_len=-1), -5),
    (GOOD, GOOD, dict(src_pt=None), -1),                               # NULL table with entries
    (GOOD, GOOD, dict(dst_pt=FAKE + 2), -3),                           # misaligned table
    (GOOD, GOOD, dict(err=FAKE + 2), -3),                              # misaligned error word
])
def test_transfer_host_validation(lib, S, D, kw, status):
    assert _call_transfer(S, D, **kw) == status
    if status:
        assert kvx.kvx_last_error() != ""
    else:
        assert kvx.kvx_last_error() == ""


def test_gather_scatter_host_validation(lib):
    L = kvx.lib()
    sp = kvx.pool_desc(GOOD, FAKE)
    b = BufSpec(2, 2, 4, 64, 2, cap=1 << 16)
    bd = kvx.buf_desc(b, FAKE)
    assert L.kvx_gather(ctypes.byref(sp), ctypes.byref(bd), FAKE, 1, FAKE, 0, None, None) == 0
    assert L.kvx_scatter(ctypes.byref(bd), ctypes.byref(sp), FAKE, 1, FAKE, 0, None, None) == 0
    bad = kvx.buf_desc(BufSpec(2, 2, 4, 64, 2, cap=-1), FAKE)
    assert L.kvx_gather(ctypes.byref(sp), ctypes.byref(bad), FAKE, 1, FAKE, 1, None, None) == -5
    bd.reserved = 1
    assert L.kvx_scatter(ctypes.byref(bd), ctypes.byref(sp), FAKE, 1, FAKE, 1, None, None) == -5
    bd.reserved = 0
    wrong = kvx.buf_desc(BufSpec(2, 2, 8, 64, 2, cap=1 << 16), FAKE)
    assert L.kvx_gather(ctypes.byref(sp), ctypes.byref(wrong), FAKE, 1, FAKE, 1, None, None) == -2
    assert L.kvx_gather(None, ctypes.byref(bd), FAKE, 1, FAKE, 1, None, None) == -1
    assert L.kvx_scatter(ctypes.byref(bd), None, FAKE, 1, FAKE, 1, None, None) == -1


def _call_slice(S, D, sl, n_reqs=1, **kw):
    L = kvx.lib()
    sp, dp = kvx.pool_desc(S, FAKE), kvx.pool_desc(D, FAKE)
    x = sl if sl is None else kvx.slice_desc(sl)
    return L.kvx_transfer_slice(ctypes.byref(sp), ctypes.byref(dp),
                                None if x is None else ctypes.byref(x), FAKE, 1, FAKE, 1,
                                FAKE, n_reqs, None, None)


BIG = PoolSpec(4, 2, 8, 64, T=16, N=8, e=2, layout="LPCTHD")
SMALL = PoolSpec(2, 1, 4, 64, T=32, N=8, e=2, layout="PLCHTD")


@pytest.mark.parametrize("S,D,sl,n_reqs,status", [
    (BIG, SMALL, (2, 0, 2, 1, 0, 1, 4, 0, 4), 0, 0),              # valid: nothing to enqueue
    (BIG, SMALL, (2, 0, 2, 1, 0, 0, 4, 0, 4), 1, 0),              # zero kv count: nothing to do
    (BIG, SMALL, None, 1, -1),                                      # NULL slice
    (BIG, SMALL, (3, 0, 2, 0, 0, 1, 0, 0, 4), 1, -5),             # layers past the source
    (BIG, SMALL, (0, 1, 2, 0, 0, 1, 0, 0, 4), 1, -5),             # layers past the destination
    (BIG, SMALL, (0, 0, 2, 0, 0, 2, 0, 0, 4), 1, -5),             # two kv into a one-kv pool
    (BIG, SMALL, (0, 0, 2, 0, 0, 1, 6, 0, 4), 1, -5),             # heads past the source
    (BIG, SMALL, (0, 0, 2, 0, 0, 1, 0, 1, 4), 1, -5),             # heads past the destination
    (BIG, SMALL, (0, 0, -1, 0, 0, 1, 0, 0, 4), 1, -5),            # negative count
    (BIG, SMALL, (-1, 0, 1, 0, 0, 1, 0, 0, 4), 1, -5),            # negative offset
    (BIG, PoolSpec(2, 1, 4, 32, T=32, N=8, e=2), (0, 0, 1, 0, 0, 1, 0, 0, 1), 1, -2),  # head_dim
    (BIG, PoolSpec(2, 1, 4, 64, T=32, N=8, e=4), (0, 0, 1, 0, 0, 1, 0, 0, 1), 1, -2),  # elem size
])
def test_slice_host_validation(lib, S, D, sl, n_reqs, status):
    assert _call_slice(S, D, sl, n_reqs) == status


def _call_buffer_slice(op, P, B, sl, n_reqs=1):
    L = kvx.lib()
    pd, bd = kvx.pool_desc(P, FAKE), kvx.buf_desc(B, FAKE)
    x = None if sl is None else ctypes.byref(kvx.slice_desc(sl))
    if op == "gather":
        return L.kvx_gather_slice(ctypes.byref(pd), ctypes.byref(bd), x, FAKE, 1, FAKE, n_reqs,
                                  None, None)
    return L.kvx_scatter_slice(ctypes.byref(bd), ctypes.byref(pd), x, FAKE, 1, FAKE, n_reqs,
                               None, None)


V_ONLY = BufSpec(2, 1, 4, 64, 2, cap=1 << 16)


@pytest.mark.parametrize("op,P,B,sl,n_reqs,status", [
    ("gather", GOOD, V_ONLY, (0, 0, 2, 1, 0, 1, 0, 0, 4), 0, 0),      # V only, nothing to enqueue
    ("scatter", GOOD, V_ONLY, (0, 0, 2, 0, 1, 1, 0, 0, 4), 0, 0),
    ("gather", GOOD, V_ONLY, None, 1, -1),                           # NULL slice
    ("scatter", GOOD, V_ONLY, None, 1, -1),
    ("gather", GOOD, BufSpec(2, 2, 4, 64, 2, cap=1 << 16), (0, 0, 2, 1, 0, 1, 0, 0, 4), 1, -2),
    ("gather", GOOD, V_ONLY, (0, 1, 2, 1, 0, 1, 0, 0, 4), 1, -5),   # buffer-side layer offset
    ("scatter", GOOD, V_ONLY, (0, 0, 2, 1, 1, 1, 0, 0, 4), 1, -5),  # buffer-side kv offset
    ("gather", GOOD, V_ONLY, (1, 0, 2, 1, 0, 1, 0, 0, 4), 1, -5),   # layers past the pool
    ("scatter", GOOD, V_ONLY, (0, 0, 2, 0, 2, 1, 0, 0, 4), 1, -5),  # kv past the pool
    ("gather", GOOD, BufSpec(2, 1, 2, 64, 2, cap=1 << 16), (0, 0, 2, 1, 0, 1, 3, 0, 2), 1, -5),
    ("gather", GOOD, BufSpec(2, 1, 4, 32, 2, cap=1 << 16), (0, 0, 2, 1, 0, 1, 0, 0, 4), 1, -2),
    ("scatter", GOOD, BufSpec(1, 1, 4, 64, 2, cap=1 << 16), (0, 0, 2, 0, 1, 1, 0, 0, 4), 1, -2),
])
def test_buffer_slice_host_validation(lib, op, P, B, sl, n_reqs, status):
    assert _call_buffer_slice(op, P, B, sl, n_reqs) == status
    if status:
        assert kvx.kvx_last_error() != ""


def test_layered_host_validation(lib):
    L = kvx.lib()
    sp, dp = kvx.pool_desc(BIG, FAKE), kvx.pool_desc(BIG, FAKE)
    ev = (ctypes.c_void_p * 4)(FAKE, FAKE, FAKE, None)

    def call(group, events, n_events, n_reqs=1):
        return L.kvx_transfer_layered(ctypes.byref(sp), ctypes.byref(dp), None, FAKE, 1, FAKE, 1,
                                      FAKE, n_reqs, group, events, n_events, None, None)
    assert call(0, ev, 4) == -5                 # group size must be >= 1
    assert call(1, ev, 3) == -5                 # 4 layers need 4 events
    assert call(2, None, 2) == -1               # no event array
    assert call(1, ev, 4) == -1                 # events[3] is NULL
    assert "events[3]" in kvx.kvx_last_error()


@pytest.mark.parametrize("args,status", [
    ((FAKE, 100, 4, 64, FAKE, 0, FAKE, 10), 0),            # nothing to hash
    ((FAKE, 100, 6, 64, FAKE, 1, FAKE, 10), -2),           # records not whole words
    ((FAKE, 100, 0, 64, FAKE, 1, FAKE, 10), -2),
    ((FAKE, 100, 4, 0, FAKE, 1, FAKE, 10), -2),            # no page size
    ((FAKE, -1, 4, 64, FAKE, 1, FAKE, 10), -5),
    ((FAKE, 100, 4, 64, FAKE, -1, FAKE, 10), -5),
    ((FAKE, 100, 4, 64, None, 1, FAKE, 10), -1),           # no records
    ((None, 100, 4, 64, FAKE, 1, FAKE, 10), -1),           # no payload
    ((FAKE, 100, 4, 64, FAKE, 1, None, 10), -1),           # no output
    ((FAKE + 2, 100, 4, 64, FAKE, 1, FAKE, 10), -3),       # misaligned payload
    ((FAKE, 100, 4, 64, FAKE, 1, FAKE + 4, 10), -3),       # misaligned output
])
def test_page_hash_host_validation(lib, args, status):
    assert kvx.lib().kvx_page_hashes(*args, FAKE, None) == status


def test_page_hash_requires_error_word(lib):
    """Without an error word a stalled chain would leave outputs incomplete
    with no signal, so the call refuses a NULL dev_err, even with nothing to
    hash."""
    for n_reqs in (0, 1):
        assert kvx.lib().kvx_page_hashes(FAKE, 100, 4, 64, FAKE, n_reqs, FAKE, 10, None, None) == -1
        assert "dev_err" in kvx.kvx_last_error()
    assert kvx.lib().kvx_page_hashes(FAKE, 100, 4, 64, FAKE, 1, FAKE, 10, FAKE + 2, None) == -3


def test_slice_reserved_must_be_zero(lib):
    x = kvx.slice_desc((0, 0, 1, 0, 0, 1, 0, 0, 1))
    x.reserved = 3
    assert _call_slice(BIG, SMALL, x) == -5


def test_last_error_is_per_call(lib):
    assert _call_transfer(GOOD, GOOD, n_reqs=-1) == -5
    assert "n_reqs" in kvx.kvx_last_error()
    assert _call_transfer(GOOD, GOOD, n_reqs=0) == 0
    assert kvx.kvx_last_error() == ""


def test_pack_reqs_round_trip():
    rows = np.array([[1, 2, 3, 4, 5, 6], [7, 8, 9, 10, 11, 12]], np.int64)
    rec = kvx.pack_reqs(rows)
    assert rec.itemsize == 40 and (rec["reserved"] == 0).all()
    back = np.stack([rec[n].astype(np.int64) for n in ("src_pt_off", "dst_pt_off", "buf_off",
                                                       "src_start", "dst_start", "n_tokens")], 1)
    assert (back == rows).all()
    with pytest.raises(ValueError):
        kvx.pack_reqs([[0, 0, 0, 2**31, 0, 1]])


def test_fastdiv_exact(tmp_path):
    """The multiply-shift division used for launch constants is exact for
    every dividend below 2^31: exhaustive over small divisors and dividends,
    and on edges and random values for large ones."""
    src = tmp_path / "fd.cpp"
    src.write_text(r'''
#include <cstdio>
#include <cstdint>
#include <random>
#include "kvx_internal.h"
int main() {
  std::mt19937_64 rng(1234);
  long bad = 0, checked = 0;
  auto check = [&](uint32_t d, uint32_t n) {
    kvx::FastDiv f = kvx::make_fastdiv(d);
    ++checked;
    if (kvx::fd_div(f, n) != n / d) { if (bad < 5) printf("d=%u n=%u\n", d, n); ++bad; }
  };
  for (uint32_t d = 1; d < 1200; ++d)
    for (uint32_t n = 0; n < 70000; ++n) check(d, n);
  const uint32_t top = 0x7fffffffu;
  for (int i = 0; i < 200000; ++i) {
    uint32_t d = 1 + (uint32_t)(rng() % top);
    if (i % 3 == 0) d = 1 + (uint32_t)(rng() % 70000);
    uint32_t n = (uint32_t)(rng() % (uint64_t(top) + 1));
    check(d, n);
    uint64_t q = n / d;
    for (int64_t e = -1; e <= 1; ++e) { int64_t m = (int64_t)(q * d) + e; if (m >= 0 && m <= top) check(d, (uint32_t)m); }
    check(d, top);
  }
  for (uint32_t s = 0; s < 31; ++s) for (int e = -1; e <= 1; ++e) {
    int64_t d = ((int64_t)1 << s) + e; if (d < 1 || d > top) continue;
    for (uint32_t n : {0u, 1u, (uint32_t)d - 1, (uint32_t)d, top, top - 1}) check((uint32_t)d, n);
  }
  printf("checked %ld bad %ld\n", checked, bad);
  return bad != 0;
}''')
    exe = tmp_path / "fd"
    cmd = [build_lib.hipcc(), "-O2", "-std=c++17", "-I", os.path.join(ROOT, "include"),
           "-I", build_lib.CSRC, "-o", str(exe), str(src)]
    subprocess.run(cmd, check=True, capture_output=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stdout


def test_missing_library_raises(monkeypatch, tmp_path):
    """No fallback: a missing libkvx.so is an error, not a silent CPU path."""
    monkeypatch.setattr(kvx, "_LIB", None)
    monkeypatch.setenv("KVX_LIBRARY", str(tmp_path / "absent.so"))
    with pytest.raises(RuntimeError, match="not built"):
        kvx.lib()
    with pytest.raises(RuntimeError):
        kvx.kvx_abi_version()


def test_binding_rejects_wrong_table_and_error_word_types():
    """Host-side checks in the binding, before any library call: a page table
    must be contiguous int32 and the error word one 32-bit integer."""
    torch = pytest.importorskip("torch")
    from paper_2606_31093_amd.workloads import PoolSpec
    P = PoolSpec(1, 1, 1, 8, T=4, N=2, e=2, layout="LPCTHD")
    a = torch.zeros(P.nbytes, dtype=torch.uint8)
    reqs = torch.zeros(40, dtype=torch.uint8)
    t32 = torch.zeros(2, dtype=torch.int32)
    for bad in (torch.zeros(2, dtype=torch.int64), torch.zeros(2, dtype=torch.float32),
                torch.zeros(4, dtype=torch.int32)[::2]):
        with pytest.raises(ValueError, match="int32"):
            kvx.kvx_transfer(a, P, a, P, bad, t32, reqs)
        with pytest.raises(ValueError, match="int32"):
            kvx.kvx_transfer(a, P, a, P, t32, bad, reqs)
        with pytest.raises(ValueError, match="int32"):
            kvx.kvx_transfer_slice(a, P, a, P, (0, 0, 1, 0, 0, 1, 0, 0, 1), bad, t32, reqs)
    with pytest.raises(ValueError, match="dev_err"):
        kvx.kvx_transfer(a, P, a, P, t32, t32, reqs, dev_err=torch.zeros(1, dtype=torch.int64))
    with pytest.raises(ValueError, match="dev_err"):
        kvx.kvx_page_hashes(torch.zeros(16, dtype=torch.uint8), 4, 4,
                            torch.zeros(32, dtype=torch.uint8), torch.zeros(1, dtype=torch.int64),
                            dev_err=torch.zeros(1, dtype=torch.float32))
    strided = torch.zeros(80, dtype=torch.uint8)[::2]          # 40 bytes, but every other one
    with pytest.raises(ValueError, match="contiguous"):
        kvx.kvx_transfer(a, P, a, P, t32, t32, strided)
    with pytest.raises(ValueError, match="contiguous"):
        kvx.kvx_page_hashes(torch.zeros(16, dtype=torch.uint8), 4, 4,
                            torch.zeros(64, dtype=torch.uint8)[::2], torch.zeros(1, dtype=torch.int64),
                            torch.zeros(1, dtype=torch.int32))


def test_binding_shares_torchs_hip_runtime():
    """Loading the library through the binding, in a fresh process that has
    not imported torch, maps exactly one HIP runtime and one HSA runtime:
    the ones torch ships, which own the tensors and streams the calls take."""
    import subprocess
    import sys
    code = (
        "import sys; sys.path.insert(0, %r)\n"
        "from paper_2606_31093_amd import kvx\n"
        "kvx.lib()\n"
        "m = sorted({l.split()[-1] for l in open('/proc/self/maps')\n"
        "            if 'libamdhip64' in l or 'libhsa-runtime64' in l})\n"
        "print('\\n'.join(m))\n" % ROOT)
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, out.stderr
    maps = out.stdout.split()
    hip = [m for m in maps if "libamdhip64" in m]
    hsa = [m for m in maps if "libhsa-runtime64" in m]
    assert len(hip) == 1 and len(hsa) == 1, maps
    import torch
    torch_lib = os.path.dirname(torch.__file__)
    assert hip[0].startswith(torch_lib) or not os.path.exists(os.path.join(torch_lib, "lib", "libamdhip64.so")), maps


def test_empty_buffer_may_have_no_memory(lib):
    """A buffer of capacity 0 may have a NULL base (a zero-size tensor has
    no memory); a buffer with capacity must have memory."""
    L = kvx.lib()
    pd = kvx.pool_desc(GOOD, FAKE)
    empty = kvx.buf_desc(BufSpec(GOOD.L, GOOD.C, GOOD.H, GOOD.D, GOOD.e, cap=0), 0)
    assert L.kvx_gather(ctypes.byref(pd), ctypes.byref(empty), FAKE, 1, FAKE, 0, None, None) == 0
    assert L.kvx_scatter(ctypes.byref(empty), ctypes.byref(pd), FAKE, 1, FAKE, 0, None, None) == 0
    full = kvx.buf_desc(BufSpec(GOOD.L, GOOD.C, GOOD.H, GOOD.D, GOOD.e, cap=1 << 10), 0)
    assert L.kvx_gather(ctypes.byref(pd), ctypes.byref(full), FAKE, 1, FAKE, 0, None, None) == -1
    assert "base is NULL" in kvx.kvx_last_error()


def _pages_reference(rows, T, side):
    """Pages a record touches on one side: the positions [start, start + n)
    of the record, page q // T for each position q, counted once."""
    total = 0
    for so, do, bo, s0, d0, n in rows:
        start = d0 if side else s0
        if n <= 0 or start < 0:
            continue
        total += len({q // T for q in range(start, start + n)})
    return total


@pytest.mark.parametrize("seed", range(6))
def test_plan_pages_matches_a_position_count(lib, seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(0, 40))
    rows = [[0, 0, 0, int(rng.integers(0, 300)), int(rng.integers(0, 300)), int(rng.integers(-2, 200))]
            for _ in range(n)]
    for T in (1, 3, 16, 64):
        for side in (0, 1):
            prefix, total, tokens = kvx.plan_pages(rows, T, side)
            per = [_pages_reference([r], T, side) for r in rows]
            assert total == sum(per)
            assert tokens == sum(max(r[5], 0) for r in rows)
            assert prefix.tolist() == [0] + np.cumsum(per, dtype=np.int64).tolist()


def test_plan_pages_counts_malformed_records_as_empty(lib):
    recs = kvx.pack_reqs([[0, 0, 0, 0, 0, 5], [0, 0, 0, 2**31 - 3, 0, 5], [0, 0, 0, 0, 0, 5]])
    recs["reserved"][2] = 1
    prefix = np.full(4, -7, np.int64)
    tokens = ctypes.c_int64(-7)
    assert lib.kvx_plan_pages(recs.ctypes.data, 3, 4, 0, prefix.ctypes.data, ctypes.byref(tokens)) == 2
    assert prefix.tolist() == [0, 2, 2, 2] and tokens.value == 5


def test_plan_pages_bad_arguments(lib):
    recs = kvx.pack_reqs([[0, 0, 0, 0, 0, 5]])
    c = lib.kvx_plan_pages
    assert c(recs.ctypes.data, 1, 0, 1, None, None) == -1          # no page size
    assert c(recs.ctypes.data, 1, 16, 2, None, None) == -1         # side not 0 or 1
    assert c(None, 1, 16, 1, None, None) == -1                     # records missing
    assert c(None, 0, 16, 1, None, None) == 0
    assert c(recs.ctypes.data, -1, 16, 1, None, None) == -1
    assert c(recs.ctypes.data, 1, 16, 1, None, None) == 1          # outputs optional


def _plan_reference(rows, Ts, Td):
    """The slots of a plan from the definition: for each destination page a
    record touches, in record order, the page's table index, the tokens it
    receives, and the table index and slot of the source position of its
    first token."""
    out = []
    for r, (so, do, _bo, s0, d0, n) in enumerate(rows):
        if n <= 0 or s0 < 0 or d0 < 0 or s0 + n >= 2**31 or d0 + n >= 2**31:
            continue
        for j in range(d0 // Td, (d0 + n - 1) // Td + 1):
            first, last = max(j * Td, d0), min((j + 1) * Td, d0 + n)
            pos = first - d0 + s0
            out.append([do + j, so + pos // Ts, first - j * Td, last - first, pos % Ts, r, 0, 0])
    return np.asarray(out, np.int64).reshape(-1, 8)


@pytest.mark.parametrize("seed", range(6))
def test_plan_fill_matches_the_definition(lib, seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(1, 30))
    rows = [[int(rng.integers(0, 50)), int(rng.integers(0, 50)), 0, int(rng.integers(0, 300)),
             int(rng.integers(0, 300)), int(rng.integers(-2, 150))] for _ in range(n)]
    for Ts, Td in ((1, 1), (3, 16), (16, 3), (64, 64), (7, 5)):
        buf, pages, tokens = kvx.host_plan(rows, Ts, Td)
        prefix, total, _ = kvx.plan_pages(rows, Td, 1)
        assert pages == total and buf.size * 8 == kvx.plan_bytes(n, pages)
        assert buf[:n + 1].tolist() == prefix.tolist()
        assert kvx.plan_slots(buf, n).tolist() == _plan_reference(rows, Ts, Td).tolist()


def test_plan_fill_clamps_table_indices(lib):
    rows = [[2**40, -2**40, 0, 0, 3, 3]]
    buf, pages, _ = kvx.host_plan(rows, 4, 4)
    assert pages == 2
    assert kvx.plan_slots(buf, 1)[:, :2].tolist() == [[-2**31, 2**31 - 1], [-2**31, 2**31 - 1]]


def test_plan_fill_bad_arguments(lib):
    recs = kvx.pack_reqs([[0, 0, 0, 0, 0, 5]])
    buf = np.zeros(kvx.plan_bytes(1, 1) // 8 + 1, np.int64)
    f = lib.kvx_plan_fill
    assert f(recs.ctypes.data, 1, 4, 8, 1, buf.ctypes.data) == 0
    assert f(recs.ctypes.data, 1, 4, 8, 2, buf.ctypes.data) == -5       # not the records' total
    assert f(recs.ctypes.data, 1, 0, 8, 1, buf.ctypes.data) == -5       # no page size
    assert f(recs.ctypes.data, -1, 4, 8, 1, buf.ctypes.data) == -5
    assert f(None, 1, 4, 8, 1, buf.ctypes.data) == -1
    assert f(recs.ctypes.data, 1, 4, 8, 1, None) == -1
    assert f(recs.ctypes.data, 1, 4, 8, 1, buf.ctypes.data + 4) == -3
    assert f(None, 0, 4, 8, 0, buf.ctypes.data) == 0


def test_planned_transfer_host_validation(lib):
    """The planned transfer checks its plan arguments and otherwise applies
    the plain transfer's host checks."""
    S = PoolSpec(1, 2, 1, 8, T=4, N=4, e=2, layout="LPCTHD")
    P = ctypes.byref(kvx.pool_desc(S, FAKE))
    call = lib.kvx_transfer_planned
    assert call(P, P, None, FAKE, 4, FAKE, 4, FAKE, 1, FAKE, -1, 4, None, None) == -5
    assert "plan_pages" in kvx.kvx_last_error()
    assert call(P, P, None, FAKE, 4, FAKE, 4, FAKE, 1, FAKE, 1, -4, None, None) == -5
    assert call(P, P, None, FAKE, 4, FAKE, 4, FAKE, 1, None, 3, 4, None, None) == -1
    assert "plan" in kvx.kvx_last_error()
    assert call(P, P, None, FAKE, 4, FAKE, 4, FAKE, 1, FAKE + 4, 3, 4, None, None) == -3
    assert call(None, P, None, FAKE, 4, FAKE, 4, FAKE, 1, FAKE, 3, 4, None, None) == -1
    assert call(P, P, None, FAKE, 4, FAKE, 4, FAKE, -1, FAKE, 3, 4, None, None) == -5
    bad = ctypes.byref(kvx.pool_desc(PoolSpec(1, 2, 1, 7, T=4, N=4, e=2), FAKE))
    assert call(bad, bad, None, FAKE, 4, FAKE, 4, FAKE, 1, FAKE, 3, 4, None, None) == -3
    assert call(P, P, None, FAKE, 4, FAKE, 4, FAKE, 0, None, 0, 0, None, None) == 0   # nothing to do


def test_layered_planned_transfer_host_validation(lib):
    """The layered planned transfer checks the group size and the plan
    arguments, then the plain layered transfer's rules."""
    S = PoolSpec(2, 2, 1, 8, T=4, N=4, e=2, layout="LPCTHD")
    P = ctypes.byref(kvx.pool_desc(S, FAKE))
    ev = (ctypes.c_void_p * 2)(FAKE, FAKE)
    call = lib.kvx_transfer_layered_planned
    assert call(P, P, None, FAKE, 4, FAKE, 4, FAKE, 1, 0, ev, 2, FAKE, 3, 4, None, None) == -5
    assert "layers_per_group" in kvx.kvx_last_error()
    assert call(P, P, None, FAKE, 4, FAKE, 4, FAKE, 1, 1, ev, 2, FAKE, -1, 4, None, None) == -5
    assert call(P, P, None, FAKE, 4, FAKE, 4, FAKE, 1, 1, ev, 2, None, 3, 4, None, None) == -1
    assert call(P, P, None, FAKE, 4, FAKE, 4, FAKE, 1, 1, ev, 2, FAKE + 4, 3, 4, None, None) == -3
    assert call(P, P, None, FAKE, 4, FAKE, 4, FAKE, 1, 1, ev, 1, FAKE, 3, 4, None, None) == -5
    assert "events" in kvx.kvx_last_error()


def test_test_build_exports_the_same_functions():
    out = subprocess.run(["nm", "-D", "--defined-only", build_lib.TEST_LIBRARY], capture_output=True,
                         text=True, check=True).stdout
    assert set(declared_functions()) <= set(re.findall(r"\b(kvx_\w+)$", out, flags=re.M))


def _header_defines(prefix):
    text = open(HEADER).read()
    return {m.group(1): int(m.group(2)) for m in re.finditer(rf"#define ({prefix}\w+) (-?\d+)", text)}


def test_launch_constants_match_the_header():
    choose, launch = _header_defines("KVX_CHOOSE_"), _header_defines("KVX_LAUNCH_")
    assert choose == {"KVX_CHOOSE_MEASURED": kvx.CHOOSE_MEASURED, "KVX_CHOOSE_SWEEP": kvx.CHOOSE_SWEEP,
                      "KVX_CHOOSE_GRID": kvx.CHOOSE_GRID}
    assert launch == {"KVX_LAUNCH_NONE": kvx.LAUNCH_NONE, "KVX_LAUNCH_GRID": kvx.LAUNCH_GRID,
                      "KVX_LAUNCH_SWEEP": kvx.LAUNCH_SWEEP}


def test_launch_choice_modes(lib):
    """The product library measures by default; every mode can be set, and
    anything else is refused without changing the mode."""
    assert kvx.kvx_launch_choice() == kvx.CHOOSE_MEASURED
    try:
        for mode in (kvx.CHOOSE_SWEEP, kvx.CHOOSE_GRID, kvx.CHOOSE_MEASURED):
            kvx.kvx_set_launch_choice(mode)
            assert kvx.kvx_launch_choice() == mode
        for bad in (-1, 3, 1 << 20):
            with pytest.raises(kvx.KvxError) as e:
                kvx.kvx_set_launch_choice(bad)
            assert e.value.status == -5 and "KVX_CHOOSE" in str(e.value)
            assert kvx.kvx_launch_choice() == kvx.CHOOSE_MEASURED
    finally:
        kvx.kvx_set_launch_choice(kvx.CHOOSE_MEASURED)


def test_test_build_starts_sweeping():
    test_lib = kvx.load(build_lib.TEST_LIBRARY)
    assert kvx.kvx_launch_choice(test_lib) == kvx.CHOOSE_SWEEP


def test_refused_call_reports_no_launch(lib):
    spec = PoolSpec(2, 2, 2, 64, T=16, N=4)
    pool = kvx.pool_desc(spec)
    status = lib.kvx_transfer(ctypes.byref(pool), None, None, 0, None, 0, None, 0, None, None)
    assert status == -1
    assert kvx.kvx_last_launch() == kvx.LAUNCH_NONE
