"""Plant plausible mistakes in the CPU oracle and check that its pins notice.

Each mutant is one textual edit of ``oracle/kvx_oracle.c`` (a dropped term, a
transposed operand, a wrong index, an off-by-one, a missing check).  The
mutant is compiled into a temporary directory and the whole pin suite runs
against it in a child process (a mutant may crash; that counts as caught).
The real oracle must pass the same suite.
"""
import os
import subprocess
import sys

import pytest

from oracle import kvx_oracle

HERE = os.path.dirname(os.path.abspath(__file__))
PINS = os.path.join(HERE, "oracle_pins.py")

T_LPCTHD = ("case ORA_LPCTHD:\n        return ((((l * P->N + p) * P->C + c) * P->T + s)"
            " * P->H + h) * P->D + d;")
T_LPCHTD = ("case ORA_LPCHTD:\n        return ((((l * P->N + p) * P->C + c) * P->H + h)"
            " * P->T + s) * P->D + d;")
T_PLCTHD = "case ORA_PLCTHD:\n        return ((((p * P->L + l) * P->C + c) * P->T + s) * P->H + h)"
T_PLCHTD = "case ORA_PLCHTD:\n        return ((((p * P->L + l)"
T_RESOLVE = ("            int bad = resolve(Dp, dst_pt, dst_pt_len, q[R_DST_PT], pd,\n"
             "                              ORA_ERR_DST_PAGE, &dp, &ds);\n"
             "            if (!bad)\n"
             "                bad = resolve(S, src_pt, src_pt_len, q[R_SRC_PT], ps,\n"
             "                              ORA_ERR_SRC_PAGE, &sp, &ss);")
T_XFER_H = ("for (int64_t h = 0; h < S->H; ++h)\n"
            "                        for (int64_t d = 0; d < S->D; ++d)\n"
            "                            copy_elem(dst + Dp->e * pool_index(Dp")

T_GS_POOL = ("src + S->e * pool_index(S, sl[0] + l, sl[3] + c,\n"
             "                                                              sp, ss, sl[6] + h, d)")
T_SS_POOL = ("copy_elem(dst + Dp->e * pool_index(Dp, sl[1] + l, sl[4] + c,\n"
             "                                                               dp, ds, sl[7] + h, d)")

MUTANTS = {
    "lpcthd_slot_head_swapped": (T_LPCTHD, T_LPCTHD.replace(
        "* P->T + s) * P->H + h)", "* P->H + h) * P->T + s)")),
    "lpcthd_kv_dropped": (T_LPCTHD, T_LPCTHD.replace("* P->C + c)", "* P->C)")),
    "lpchtd_dim_dropped": (T_LPCHTD, T_LPCHTD.replace("* P->D + d;", "* P->D;")),
    "plcthd_head_major": (T_PLCTHD, T_PLCTHD.replace(
        "* P->T + s) * P->H + h)", "* P->H + h) * P->T + s)")),
    "plchtd_layer_major": (T_PLCHTD, T_PLCHTD.replace("(p * P->L + l)", "(l * P->N + p)")),
    "buffer_layer_kv_swapped": ("return off + (((l * B->C + c) * n + i)",
                                "return off + (((c * B->L + l) * n + i)"),
    "buffer_head_major": ("(((l * B->C + c) * n + i) * B->H + h) * B->D + d",
                          "(((l * B->C + c) * B->H + h) * n + i) * B->D + d"),
    "slot_off_by_one": ("*slot = q % P->T;", "*slot = (q + 1) % P->T;"),
    "page_index_rounds_up": ("int64_t idx = pt_off + q / P->T;",
                             "int64_t idx = pt_off + (q + P->T - 1) / P->T;"),
    "source_position_from_dst_start": (
        "int64_t ps = q[R_SRC_START] + i, pd = q[R_DST_START] + i;",
        "int64_t ps = q[R_DST_START] + i, pd = q[R_DST_START] + i;"),
    "dst_position_from_src_start": (
        "int64_t ps = q[R_SRC_START] + i, pd = q[R_DST_START] + i;",
        "int64_t ps = q[R_SRC_START] + i, pd = q[R_SRC_START] + i;"),
    "element_last_byte_dropped": ("for (int64_t b = 0; b < e; ++b)",
                                  "for (int64_t b = 0; b + 1 < e; ++b)"),
    "transfer_one_head_short": (T_XFER_H, T_XFER_H.replace("h < S->H", "h + 1 < S->H")),
    "scatter_tokens_reversed": (
        "src + B->e * buf_index(B, q[R_BUF], n, l, c, i, h, d)",
        "src + B->e * buf_index(B, q[R_BUF], n, l, c, n - 1 - i, h, d)"),
    "block_may_not_reach_end": ("<= B->cap;", "< B->cap;"),
    "gather_ignores_dst_start": ("q[R_DST_START] != 0 ||", "0 ||"),
    "page_id_n_accepted": ("if (id < 0 || id >= P->N)", "if (id < 0 || id > P->N)"),
    "table_end_accepted": ("if (idx < 0 || idx >= pt_len)", "if (idx < 0 || idx > pt_len)"),
    "source_resolved_first": (T_RESOLVE, T_RESOLVE
                              .replace("resolve(Dp, dst_pt, dst_pt_len, q[R_DST_PT], pd,\n"
                                       "                              ORA_ERR_DST_PAGE, &dp, &ds)",
                                       "@@D@@")
                              .replace("resolve(S, src_pt, src_pt_len, q[R_SRC_PT], ps,\n"
                                       "                              ORA_ERR_SRC_PAGE, &sp, &ss)",
                                       "resolve(Dp, dst_pt, dst_pt_len, q[R_DST_PT], pd,\n"
                                       "                              ORA_ERR_DST_PAGE, &dp, &ds)")
                              .replace("@@D@@",
                                       "resolve(S, src_pt, src_pt_len, q[R_SRC_PT], ps,\n"
                                       "                              ORA_ERR_SRC_PAGE, &sp, &ss)")),
    "negative_start_accepted": ("return n >= 0 && start >= 0 &&", "return n >= 0 &&"),
    "int32_end_unchecked": ("&& start + n <= INT32_MAX;", ";"),
    "misaligned_block_accepted": ("if (off < 0 || (off * B->e) % 16 != 0)", "if (off < 0)"),
    "slice_dst_layer_from_src_offset": ("sl[1] + l", "sl[0] + l"),
    "slice_dst_head_from_src_offset": ("sl[7] + h", "sl[6] + h"),
    "slice_src_kv_offset_dropped": ("sl[3] + c", "c"),
    "slice_one_layer_short": ("l < sl[2]", "l + 1 < sl[2]"),
    "slice_heads_of_the_pool": (
        "h < sl[8]; ++h)\n                        for (int64_t d = 0; d < S->D; ++d)",
        "h < S->H; ++h)\n                        for (int64_t d = 0; d < S->D; ++d)"),
    "scatter_slice_heads_of_the_pool": (
        "h < sl[8]; ++h)\n                        for (int64_t d = 0; d < Dp->D; ++d)",
        "h < Dp->H; ++h)\n                        for (int64_t d = 0; d < Dp->D; ++d)"),
    "empty_slice_checked": ("    if (sl[2] == 0 || sl[5] == 0 || sl[8] == 0)\n        return 0;\n", ""),
    "gather_slice_layer_from_buffer_offset": (
        T_GS_POOL, T_GS_POOL.replace("sl[0] + l", "sl[1] + l")),
    "gather_slice_head_offset_dropped": (T_GS_POOL, T_GS_POOL.replace("sl[6] + h", "h")),
    "scatter_slice_kv_from_buffer_offset": (
        T_SS_POOL, T_SS_POOL.replace("sl[4] + c", "sl[3] + c")),
    "scatter_slice_one_layer_short": (
        T_SS_POOL, T_SS_POOL.replace("sl[1] + l", "sl[1] + l + (l > 0)")),
    "fnv1_instead_of_fnv1a": ("        h ^= p[i];\n        h *= FNV_PRIME;",
                              "        h *= FNV_PRIME;\n        h ^= p[i];"),
    "chain_pair_swapped": ("le64(pair, h);\n            le64(pair + 8, c);",
                           "le64(pair, c);\n            le64(pair + 8, h);"),
    "digest_continues_chain": ("count * rec_bytes, FNV_BASIS);", "count * rec_bytes, h);"),
    "seed_ignored": ("uint64_t h = (uint64_t)q[2];", "uint64_t h = 0;"),
    "last_page_padded": ("int64_t count = (n - first < T) ? n - first : T;", "int64_t count = T;"),
    "hash_out_shifted": ("out[out_off + j] = h;", "out[out_off + pages - 1 - j] = h;"),
    "hash_bounds_unchecked": ("off + n > payload_positions ||", "0 ||"),
}
# Sites that occur in more than one function: each occurrence is mutated on
# its own, in source order (ora_transfer, ora_gather, ora_scatter,
# ora_transfer_slice, ora_gather_slice, ora_scatter_slice).
OCCURRENCES = {"source_position_from_dst_start": 2, "dst_position_from_src_start": 2,
               "source_resolved_first": 2, "scatter_tokens_reversed": 2,
               "gather_ignores_dst_start": 2, "slice_dst_layer_from_src_offset": 2,
               "slice_dst_head_from_src_offset": 2, "slice_src_kv_offset_dropped": 2,
               "slice_one_layer_short": 3, "slice_heads_of_the_pool": 2,
               "empty_slice_checked": 3}
CASES = sorted((name, k) for name in MUTANTS for k in range(OCCURRENCES.get(name, 1)))


def _run_pins(lib):
    return subprocess.run([sys.executable, PINS, lib], capture_output=True, text=True,
                          timeout=300)


def test_real_oracle_passes_pins_in_child():
    kvx_oracle.build()
    r = _run_pins(kvx_oracle.LIBRARY)
    assert r.returncode == 0, r.stdout + r.stderr


@pytest.mark.parametrize("name,occurrence", CASES, ids=[f"{n}-{o}" for n, o in CASES])
def test_mutant_is_caught(name, occurrence, tmp_path):
    old, new = MUTANTS[name]
    text = open(kvx_oracle.SOURCE).read()
    want = OCCURRENCES.get(name, 1)
    assert text.count(old) == want, f"mutation site for {name} must occur {want} time(s)"
    assert old != new
    at = -1
    for _ in range(occurrence + 1):
        at = text.index(old, at + 1)
    src = tmp_path / "kvx_oracle_mutant.c"
    src.write_text(text[:at] + new + text[at + len(old):])
    lib = str(tmp_path / "libkvx_oracle_mutant.so")
    kvx_oracle.build(str(src), lib)
    r = _run_pins(lib)
    assert r.returncode != 0, f"mutant {name} survived every pin"
